"""GPU parity of the (deflated) polar factor against the CPU oracle.

Tolerances (relative Frobenius error of the output): 1e-4 for the float32
paths against the float64 oracle; 2e-2 for the bf16 paths, both against the
oracle's bf16 contract and against exact arithmetic on the bf16 input.
Deflation ranks must match exactly.
"""
import numpy as np
import pytest
import torch

import paper_2609_21102_amd as sd
import workloads
from oracle import filters
from oracle import muon as omuon
from oracle import rng as orng
from tests.gpu_util import dev_tensor, host64, rel_fro, say

pytestmark = pytest.mark.gpu

F32_TOL = 1e-4
BF16_TOL = 2e-2


def run_case(case, k=None, steps=None, **kw):
    k = case.k if k is None else k
    steps = case.steps if steps is None else steps
    x = dev_tensor(case.x, case.dtype)
    out, info = sd.msign(x, k, steps, case.coeffs[:steps], oversample=case.oversample,
                         power_iters=case.power_iters, gamma=case.gamma, info=True, **kw)
    torch.cuda.synchronize()
    return out, info


def oracle_case(case, k=None, steps=None, idx=None, mode=None, **kw):
    """The oracle on the case's input (the bf16 input's values for bf16
    cases): mode defaults to the bf16 contract for bf16 cases, else exact."""
    k = case.k if k is None else k
    steps = case.steps if steps is None else steps
    x64 = case.x64 if idx is None else case.x64[idx]
    if mode is None:
        mode = "bf16" if case.dtype == "bf16" else "exact"
    sketches = None
    if idx is not None and k > 0:
        # the oracle numbers matrices from 0; pass the sketches of the sampled ones
        s = min(case.x.shape[1:])
        r = kw["window"] if kw.get("tau", 0.0) > 0 and kw.get("window") else k
        rp = min(s, r + case.oversample)
        sketches = [orng.sketch(kw.get("seed", 0), int(b), s, rp) for b in idx]
    return omuon.msign_deflated(x64, k, case.coeffs[:steps], oversample=case.oversample,
                                power_iters=case.power_iters, gamma=case.gamma, mode=mode,
                                sketches=sketches, tau=kw.get("tau", 0.0), seed=kw.get("seed", 0),
                                window=kw.get("window"), restore=kw.get("restore", "padded"))


def check_bf16_sample(name, got, case, idx, **kw):
    """A bf16 output against the oracle's bf16 contract and against exact
    arithmetic on the same (bf16) input, both at the bf16 tolerance."""
    want_c, oinfo = oracle_case(case, idx=idx, **kw)
    want_e, _ = oracle_case(case, idx=idx, mode="exact", **kw)
    ec, ee = rel_fro(got, want_c[0]), rel_fro(got, want_e[0])
    say(f"{name}: rel err {ec:.3e} (bf16 contract), {ee:.3e} (exact on the bf16 input)")
    assert ec < BF16_TOL and ee < BF16_TOL
    return oinfo


def test_one_step_fp32():
    case = workloads.small_muon(1, 64, 200, k=0)
    say("one step fp32 64x200")
    out, _ = run_case(case, k=0, steps=1)
    want, _ = oracle_case(case, k=0, steps=1)
    assert rel_fro(host64(out), want) < 1e-5


SHAPES = [(1, 8, 17), (3, 17, 64), (2, 64, 17), (1, 130, 300), (2, 256, 129), (1, 300, 130), (2, 128, 384)]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("k", [0, 1, 4])
def test_fp32_shapes(shape, k):
    # Ragged, tall and wide shapes over several tiles, with config 1's bulk
    # down to 1e-3 under spikes up to 50 (s_1 / nu up to about 120: the
    # residual is formed in float64, so the head's rounding does not reach
    # R / nu).
    b, m, n = shape
    if k >= min(m, n):
        pytest.skip("k must be below min(m, n)")
    case = workloads.small_muon(b, m, n, k=max(k, 1), power_iters=1, bulk=(1e-3, 1.0))
    say(f"fp32 {shape} k={k}")
    out, info = run_case(case, k=k)
    want, oinfo = oracle_case(case, k=k)
    err = rel_fro(host64(out), want)
    say(f"  rel err {err:.3e}")
    assert err < F32_TOL
    assert info["k_eff"].cpu().tolist() == oinfo.k_eff


def test_config1_fp32():
    case = workloads.config1()
    for k in (0, case.k):
        say(f"config1 k={k}")
        out, info = run_case(case, k=k)
        want, oinfo = oracle_case(case, k=k)
        err = rel_fro(host64(out), want)
        say(f"  rel err {err:.3e}")
        assert err < F32_TOL
        assert info["k_eff"].cpu().tolist() == oinfo.k_eff
        np.testing.assert_allclose(info["nu"].cpu().numpy(), oinfo.nu, rtol=1e-4)
        if k:
            np.testing.assert_allclose(info["s"].cpu().numpy()[0], oinfo.s[0], rtol=1e-5)


@pytest.mark.parametrize("shape", [(2, 1, 37), (3, 45, 1)], ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_vector_inputs_closed_form(shape, dtype):
    # A 1 x n (or n x 1) input has one singular value; X0 = X / ||X||_F puts
    # it at 1, so the filter returns p^L(1) v / ||v|| with p^L the scalar
    # composition of the coefficient table (eq:general_ns_iteration). The
    # bf16 contract rounds every product operand (the 1 x 1 Gram is then
    # 1 + O(2^-8) and the error grows over the steps), so in bf16 only the
    # oracle's bf16 contract is the reference.
    case = workloads.small_muon(*shape, dtype=dtype, k=0, case_id=7)
    say(f"vector input {shape} {dtype}")
    out, _ = run_case(case, k=0)
    v = case.x64.reshape(shape[0], -1)
    scale = 1.0
    for row in case.coeffs:
        scale = sum(c * scale ** (2 * i + 1) for i, c in enumerate(row))
    want = scale * v / np.linalg.norm(v, axis=1, keepdims=True)
    got = host64(out).reshape(shape[0], -1)
    tol = F32_TOL if dtype == "f32" else BF16_TOL
    if dtype == "f32":
        for b in range(shape[0]):
            assert rel_fro(got[b], want[b]) < tol
    want_o, _ = oracle_case(case, k=0)
    assert rel_fro(host64(out), want_o) < tol


@pytest.mark.parametrize("shape", [(2, 2, 50), (2, 50, 3)], ids=lambda s: "x".join(map(str, s)))
def test_full_rank_sketch_fp32(shape):
    # r' = min(s, k + p) = s: the sketch spans the whole short side, so the
    # head is exact and only rounding is left in R (Sec. 2.2 exact deflation).
    # A moderate spike over the bulk: float32 resolves the residual's
    # singular values to about 1e-7 of the spike, so a spike 5000 times the
    # bulk leaves 5e-4 in R against the float64 oracle (measured), past the
    # 1e-4 contract; a ratio of at most 40 keeps that below 1e-5.
    case = workloads.small_muon(*shape, k=1, spikes=[4.0], bulk=(0.1, 1.0), case_id=8)
    say(f"full-rank sketch {shape}")
    out, info = run_case(case, k=1)
    want, oinfo = oracle_case(case, k=1)
    assert rel_fro(host64(out), want) < F32_TOL
    assert info["k_eff"].cpu().tolist() == oinfo.k_eff
    got_s = info["s"].cpu().numpy().reshape(shape[0], -1)
    for b in range(shape[0]):
        np.testing.assert_allclose(got_s[b][0], oinfo.s[b][0], rtol=1e-5)


@pytest.mark.parametrize("shape", [(2, 64, 200), (1, 96, 96), (3, 200, 70), (1, 128, 1000)],
                         ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("k", [0, 4])
def test_bf16_shapes(shape, k):
    b, m, n = shape
    case = workloads.small_muon(b, m, n, dtype="bf16", k=max(k, 1), bulk=(1e-3, 1.0))
    out, info = run_case(case, k=k)
    got = host64(out)
    for i in range(b):
        oinfo = check_bf16_sample(f"bf16 {shape} k={k} matrix {i}", got[i], case, [i], k=k)
        assert int(info["k_eff"][i]) == oinfo.k_eff[0]


def test_headline_768x3072_bf16_sampled():
    # The benchmark's launch: 24 matrices of 768 x 3072 in one call; the oracle
    # checks a sample of them.
    case = workloads.config2("768x3072")
    out, info = run_case(case)
    got = host64(out)
    for idx in ([0], [13], [23]):
        oinfo = check_bf16_sample(f"config2 768x3072 matrix {idx[0]}", got[idx[0]], case, idx)
        assert int(info["k_eff"][idx[0]]) == oinfo.k_eff[0]


@pytest.mark.parametrize("group", ["768x768", "768x2304"])
def test_config2_other_groups_sampled(group):
    case = workloads.config2(group)
    out, info = run_case(case)
    got = host64(out)
    for idx in ([0], [11]):
        check_bf16_sample(f"config2 {group} matrix {idx[0]}", got[idx[0]], case, idx)


@pytest.mark.parametrize("group,batch", [("768x3072", 4), ("768x768", 12), ("768x2304", 12)])
def test_config3_polar_express_table_sampled(group, batch):
    case = workloads.config3(group, batch=batch)
    out, _ = run_case(case)
    got = host64(out)
    for idx in ([0], [batch - 1]):
        check_bf16_sample(f"config3 {group} matrix {idx[0]}", got[idx[0]], case, idx)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_nonfinite_input_completes(dtype):
    """A NaN in one matrix of the batch: that matrix's output is not finite,
    the call completes (the singular values are ordered with NaN last under a
    total order, so the head's ordering stays a permutation), and the other
    matrix is unaffected."""
    case = workloads.small_muon(2, 96, 160, dtype=dtype, k=4, spikes=[50, 30, 20, 10])
    xs = case.x.copy()
    xs[0, 7, 11] = 0x7FC0 if dtype == "bf16" else np.nan   # bf16 quiet NaN bits / float32 NaN
    out = sd.msign(dev_tensor(xs, dtype), 4, 5)
    clean = sd.msign(dev_tensor(case.x, dtype), 4, 5)
    torch.cuda.synchronize()
    assert not torch.isfinite(out[0].float()).all()
    assert torch.isfinite(clean.float()).all()
    assert torch.equal(out[1], clean[1])


def test_gate_off_equals_baseline_bitwise():
    # Sec. 2.2: when the gate does not fire the method reduces exactly to Muon.
    case = workloads.small_muon(2, 96, 160, k=3, spikes=[2.0, 1.9, 1.8])
    x = dev_tensor(case.x, "f32")
    base = sd.msign(x, 0, 5)
    gated, info = sd.msign(x, 3, 5, tau=0.1, info=True)
    torch.cuda.synchronize()
    assert info["k_eff"].cpu().tolist() == [0, 0]
    assert torch.equal(base, gated)


def test_gate_fires_with_margin():
    case = workloads.small_muon(2, 96, 160, k=6, spikes=[50, 30, 20, 1.0, 0.9, 0.8], bulk=(1e-3, 0.5))
    x = dev_tensor(case.x, "f32")
    out, info = sd.msign(x, 6, 5, tau=0.1, info=True)
    torch.cuda.synchronize()
    want, oinfo = omuon.msign_deflated(case.x64, 6, case.coeffs, tau=0.1)
    assert info["k_eff"].cpu().tolist() == oinfo.k_eff == [3, 3]
    assert rel_fro(host64(out), want) < F32_TOL


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_gate_window_separate_from_k(dtype):
    # Alg. 1's gate over a window of r = 6 estimated values (r' = 14), capped
    # at k; deflation counts bit-exact against the oracle, on both paths.
    case = workloads.small_muon(2, 96, 160, dtype=dtype, k=6, spikes=[50, 30, 20, 1.0, 0.9, 0.8],
                                bulk=(1e-3, 0.5), case_id=45)
    for k, want_k in ((6, 3), (2, 2)):
        out, info = run_case(case, k=k, tau=0.1, window=6)
        got = host64(out)
        want, oinfo = oracle_case(case, k=k, tau=0.1, window=6)
        assert info["k_eff"].cpu().tolist() == oinfo.k_eff == [want_k, want_k]
        np.testing.assert_allclose(info["s"].cpu().numpy(), np.stack(oinfo.s), rtol=1e-5 if dtype == "f32" else 1e-4)
        if dtype == "f32":
            assert rel_fro(got, want) < F32_TOL
        else:
            for b in range(2):
                check_bf16_sample(f"gate window bf16 k={k} matrix {b}", got[b], case, [b], k=k, tau=0.1, window=6)


@pytest.mark.parametrize("m,n", [(100, 260), (96, 160)])
def test_deterministic_and_transpose_exact(m, n):
    # (96, 160): the tall transpose's short side is a multiple of 8, so its
    # canonical copy takes 16-byte accesses; (100, 260): element accesses
    case = workloads.small_muon(2, m, n, dtype="bf16", k=4)
    x = dev_tensor(case.x, "bf16")
    a = sd.msign(x, 4, 5)
    b = sd.msign(x, 4, 5)
    xt = x.transpose(1, 2).contiguous()
    c = sd.msign(xt, 4, 5)
    torch.cuda.synchronize()
    assert torch.equal(a, b)
    assert torch.equal(a, c.transpose(1, 2))


def test_batch_independent_across_store_policies():
    """A matrix's result does not depend on the rest of its batch, also where
    the batch size switches the Gram's epilogue between ordinary stores
    (outputs that fit in half of the last-level cache) and streaming stores:
    48 matrices of 768 x 1024 bf16 (170 MB of Gram copies per step, streamed)
    give for their first 24 bitwise the outputs, residual norms and singular
    values of those 24 alone (85 MB, ordinary stores)."""
    gen = torch.Generator(device="cuda")
    gen.manual_seed(11)
    x48 = torch.randn((48, 768, 1024), generator=gen, device="cuda", dtype=torch.float32).to(torch.bfloat16)
    x24 = x48[:24].contiguous()
    a, ia = sd.msign(x48, 8, 5, info=True)
    b, ib = sd.msign(x24, 8, 5, info=True)
    torch.cuda.synchronize()
    assert torch.equal(a[:24], b)
    assert torch.equal(ia["nu"][:24], ib["nu"])
    assert torch.equal(ia["s"][:24], ib["s"])
    assert int(ia["status"]) == 0 and int(ib["status"]) == 0


def test_device_sketch_matches_host_generator():
    for (b, s, rp, seed) in [(3, 80, 12, 5), (24, 768, 16, 0), (2, 17, 5, 2**40 + 7)]:
        dev = sd.sketch(b, s, rp, seed).cpu().numpy()
        host = sd.sketch_host(b, s, rp, seed)
        bad = np.count_nonzero(dev != host)
        say(f"sketch {b}x{s}x{rp}: {bad} mismatches, max diff {np.abs(dev - host).max():.3e}")
        assert bad == 0


def test_sketch_hook_matches_internal_generator():
    case = workloads.small_muon(3, 80, 150, k=4)
    x = dev_tensor(case.x, "f32")
    rp = min(80, 4 + 8)
    om = np.ascontiguousarray(np.stack([orng.sketch(5, b, 80, rp).T for b in range(3)]), dtype=np.float32)
    sk = torch.from_numpy(om).cuda()
    a = sd.msign(x, 4, 5, seed=5)
    b = sd.msign(x, 4, 5, seed=5, sketch=sk)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


def test_zero_matrix_and_in_place():
    z = torch.zeros(2, 40, 72, device="cuda")
    for k in (0, 3):
        assert torch.count_nonzero(sd.msign(z, k, 5)) == 0
    case = workloads.small_muon(1, 64, 128, k=2)
    x = dev_tensor(case.x, "f32")
    ref = sd.msign(x, 2, 5)
    sd.msign(x, 2, 5, out=x)
    torch.cuda.synchronize()
    assert torch.equal(ref, x)


def _closed_form_head(x, k, table, gamma=1.01):
    """p^L(1/gamma) U_k V_k^T from the input's SVD (float64), per matrix."""
    out = []
    scale = float(filters.scalar_compose(np.array([1.0 / gamma]), table)[0])
    for xb in x:
        u, s_, vt = np.linalg.svd(xb, full_matrices=False)
        out.append(scale * u[:, :k] @ vt[:k])
    return np.stack(out), scale


def test_rank_deficient_fp32_policy():
    # rank(X) = 2 <= k is outside Alg. 1's domain (k < rank(M)): the residual
    # is rounding of the head. The library drops a residual within 2^-20 of
    # ||X||_F (flag 4), so X0 = gamma^-1 U_k V_k^T and the output is the
    # closed form p^L(1/gamma) U_2 V_2^T of the input's SVD (explicit
    # restore: U_2 V_2^T). With k = 4 the two extra head directions are
    # rounding (pivot floor, flag 2): the output is finite and acts on the
    # input's range as p^L(1/gamma).
    import dataclasses
    base = workloads.small_muon(2, 64, 200, k=2, case_id=3)
    x = workloads.low_rank(2, 64, 200, 2, case_id=1)
    case = dataclasses.replace(base, x=x)
    table = case.coeffs
    want, scale = _closed_form_head(case.x64, 2, table)
    say("rank-deficient fp32 k=2")
    out, info = run_case(case)
    assert int(info["status"][0]) & 4
    assert rel_fro(host64(out), want) < F32_TOL
    out, info = run_case(case, restore="explicit")
    assert rel_fro(host64(out), want / scale) < F32_TOL
    say("rank-deficient fp32 k=4")
    out, info = run_case(case, k=4)
    assert int(info["status"][0]) & 6 == 6
    got = host64(out)
    assert np.isfinite(got).all()
    for b in range(2):
        u, _, vt = np.linalg.svd(case.x64[b], full_matrices=False)
        core = u[:, :2].T @ got[b] @ vt[:2].T
        np.testing.assert_allclose(core, scale * np.eye(2), atol=1e-4)
    say("full-rank fp32")
    out, info = run_case(workloads.small_muon(2, 64, 200, k=4, bulk=(1e-2, 1.0), case_id=2))
    assert int(info["status"][0]) == 0


def test_rank_deficient_bf16_input_is_full_rank():
    # bf16 rounding of a rank-2 matrix leaves a full-rank input whose tail is
    # its quantization (about 2^-9 of ||X||_F): Alg. 1 treats it as the
    # residual, as exact arithmetic on the bf16 input does; no flag is raised.
    # The output is then 62 filtered noise directions from small singular
    # values, where the filter's slope amplifies every bf16 operand rounding:
    # the oracle's own bf16 contract sits 2.3e-2 - 2.4e-2 from exact
    # arithmetic here, so the tolerance is twice that gap, measured on the
    # oracle in the test. The head is not noise: on the input's leading
    # singular vectors the output is p^L(1/gamma) I to the bf16 tolerance.
    import dataclasses
    base = workloads.small_muon(2, 64, 200, dtype="bf16", k=2, case_id=3)
    case = dataclasses.replace(base, x=workloads.to_bf16_bits(workloads.low_rank(2, 64, 200, 2, case_id=1)))
    out, info = run_case(case)
    assert int(info["status"][0]) == 0
    got = host64(out)
    scale = float(filters.scalar_compose(np.array([1.0 / case.gamma]), case.coeffs)[0])
    for b in range(2):
        want_c, _ = oracle_case(case, idx=[b])
        want_e, _ = oracle_case(case, idx=[b], mode="exact")
        gap = rel_fro(want_c[0], want_e[0])
        tol = max(BF16_TOL, 2 * gap)
        ec, ee = rel_fro(got[b], want_c[0]), rel_fro(got[b], want_e[0])
        u, _, vt = np.linalg.svd(case.x64[b], full_matrices=False)
        core = u[:, :2].T @ got[b] @ vt[:2].T
        say(f"bf16 rank-2 input matrix {b}: {ec:.3e} (contract), {ee:.3e} (exact), oracle gap {gap:.3e}; "
            f"head {np.abs(core - scale * np.eye(2)).max():.3e}")
        assert ec < tol and ee < tol
        np.testing.assert_allclose(core, scale * np.eye(2), atol=BF16_TOL * scale)


def test_tail_far_below_the_spike_fp32():
    # A full-rank input whose tail sits 1e-6 below the spike (64 x 200, spike
    # 1e6 over a tail in [1e-2, 1], k = 1, J = 2) keeps its tail: no residual
    # flag, full-rank output, and the error to polar(M) of Alg. 1 in exact
    # arithmetic. float32 resolves the tail's entries to about 2^-24 / 4e-6 =
    # 1.5e-2 of their size, which bounds the agreement with the float64 oracle.
    import dataclasses
    g = np.random.default_rng(5)
    m, n = 64, 200
    sig = np.concatenate([[1e6], np.sort(10 ** g.uniform(-2, 0, m - 1))[::-1]])
    x = ((workloads.haar_orthogonal(g, m, m) * sig) @ workloads.haar_orthogonal(g, n, m).T).astype(np.float32)
    case = dataclasses.replace(workloads.small_muon(1, m, n, k=1, power_iters=2, case_id=46), x=x[None])
    out, info = run_case(case)
    got = host64(out)[0]
    assert int(info["status"][0]) == 0
    target = omuon.polar_exact(case.x64)[0]
    want, _ = oracle_case(case)
    err_t, err_o = rel_fro(got, target), rel_fro(got, want[0])
    sv = np.linalg.svd(got, compute_uv=False)
    say(f"tail 1e-6 below the spike: to polar(M) {err_t:.3f} (oracle {rel_fro(want[0], target):.3f}), "
        f"to the oracle {err_o:.3e}, smallest singular value {sv.min():.3f}")
    assert sv.min() > 0.3
    assert err_t < 0.2


def test_caller_workspace():
    case = workloads.small_muon(2, 128, 256, dtype="bf16", k=4)
    x = dev_tensor(case.x, "bf16")
    nbytes = sd.msign_workspace_bytes(2, 128, 256, 4, sd.SD_DTYPE_BF16)
    ws = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    a = sd.msign(x, 4, 5)
    b = sd.msign(x, 4, 5, workspace=ws)
    torch.cuda.synchronize()
    assert torch.equal(a, b)
    with pytest.raises(sd.SdError):
        sd.msign(x, 4, 5, workspace=ws[: nbytes // 2])


def test_steps_zero_returns_start():
    case = workloads.small_muon(1, 64, 96, k=2)
    x = dev_tensor(case.x, "f32")
    out = sd.msign(x, 2, 0)
    torch.cuda.synchronize()
    want, _ = omuon.msign_deflated(case.x64, 2, np.zeros((0, 3)))
    assert rel_fro(host64(out), want) < 1e-5


def _group_args(case):
    return dict(x=dev_tensor(case.x, case.dtype), k=case.k, steps=case.steps, coeffs=case.coeffs,
                oversample=case.oversample, power_iters=case.power_iters, gamma=case.gamma)


@pytest.mark.parametrize("dtype,k,restore", [("bf16", 4, "padded"), ("f32", 4, "padded"), ("f32", 0, "padded"),
                                             ("bf16", 3, "explicit")])
def test_param_list_grouping_bitwise(dtype, k, restore):
    """sd_msign_params buckets a parameter list by shape with wide and tall
    sharing a group (polar(M^T) = polar(M)^T): every output equals, bit for
    bit, the batched call on its group stacked in list order with tall members
    transposed; also in place (outputs on the inputs)."""
    rng = np.random.default_rng([21102, 41, 0 if dtype == "bf16" else 1])
    shapes = [(64, 200), (200, 64), (96, 96), (64, 200), (128, 300), (300, 128), (96, 96), (33, 70), (70, 33)]
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    xs = [torch.from_numpy(rng.standard_normal(sh).astype(np.float32)).to(tdt).cuda().contiguous() for sh in shapes]
    say(f"param list {dtype} k={k} {restore}: {len(xs)} matrices")
    outs = sd.msign_params(xs, k, 5, restore=restore)
    torch.cuda.synchronize()
    groups = {}
    for i, x in enumerate(xs):
        groups.setdefault((min(x.shape), max(x.shape)), []).append(i)
    assert list(groups) == [(64, 200), (96, 96), (128, 300), (33, 70)]
    for key, idx in groups.items():
        stack = torch.stack([xs[i] if xs[i].shape[0] <= xs[i].shape[1] else xs[i].t() for i in idx]).contiguous()
        want = sd.msign(stack, k, 5, restore=restore)
        torch.cuda.synchronize()
        for b, i in enumerate(idx):
            w = want[b] if xs[i].shape[0] <= xs[i].shape[1] else want[b].t()
            assert torch.equal(outs[i], w), (key, i)
    copies = [x.clone() for x in xs]
    sd.msign_params(copies, k, 5, outs=copies, restore=restore)
    torch.cuda.synchronize()
    for a, b in zip(copies, outs):
        assert torch.equal(a, b)


def test_groups_match_single_calls_bitwise():
    """sd_msign_groups runs the groups concurrently on the library's streams;
    each group's result must be the single call's, bit for bit."""
    cases = [workloads.config2(g, batch=3) for g in ("768x768", "768x2304", "768x3072")]
    cases.append(workloads.small_muon(2, 300, 200, dtype="f32", k=4, case_id=31))
    groups = [_group_args(c) for c in cases]
    outs = sd.msign_groups(groups)
    outs2 = sd.msign_groups(groups)
    torch.cuda.synchronize()
    for g, c, o, o2 in zip(groups, cases, outs, outs2):
        ref = sd.msign(g["x"], c.k, c.steps, c.coeffs, oversample=c.oversample, power_iters=c.power_iters,
                       gamma=c.gamma)
        torch.cuda.synchronize()
        say(f"group {c.name}: equal {torch.equal(o, ref)}")
        assert torch.equal(o, ref)
        assert torch.equal(o, o2)


def test_groups_reject_bad_group_without_enqueueing():
    case = workloads.config2("768x768", batch=2)
    good = _group_args(case)
    out = torch.full_like(good["x"], 7.0)
    bad = dict(good, k=768)          # k >= min(m, n)
    with pytest.raises(sd.SdError):
        sd.msign_groups([dict(good, out=out), bad])
    torch.cuda.synchronize()
    assert bool((out == 7.0).all())  # nothing ran


@pytest.mark.slow
@pytest.mark.timeout(600)
def test_paper_scale_groups_sampled():
    """The paper's GPT-2 Large groups in one grouped call (144 x 1280 x 1280
    and 72 x 5120 x 1280, tall, k = 32, r' = 64); the oracle checks two
    batch positions of each group (each position draws its own sketch)."""
    cases = [workloads.paper_scale_group(g) for g in ("1280x1280", "5120x1280")]
    groups = [_group_args(c) for c in cases]
    outs = sd.msign_groups(groups)
    torch.cuda.synchronize()
    for c, o in zip(cases, outs):
        got = host64(o)
        for b in (1, c.x.shape[0] - 1):
            check_bf16_sample(f"{c.name} matrix {b}", got[b], c, [b])


@pytest.mark.parametrize("shape,dtype", [((2, 96, 200), "f32"), ((2, 200, 70), "f32"), ((1, 128, 256), "f32"),
                                         ((2, 64, 200), "bf16"), ((3, 200, 70), "bf16"), ((1, 128, 1024), "bf16")],
                         ids=lambda v: "x".join(map(str, v)) if isinstance(v, tuple) else v)
def test_explicit_restore(shape, dtype):
    """restore="explicit": X0 = R / nu and U_k V_k^T added to the filter
    output (eq:identities). Aligned wide inputs take the direct output path,
    tall or ragged ones the canonical buffer."""
    b, m, n = shape
    case = workloads.small_muon(b, m, n, dtype=dtype, k=4, case_id=41)
    out, info = run_case(case, restore="explicit")
    want, oinfo = omuon.msign_deflated(case.x64, case.k, case.coeffs, oversample=case.oversample,
                                       power_iters=case.power_iters, mode="bf16" if dtype == "bf16" else "exact",
                                       restore="explicit")
    err = rel_fro(host64(out), want)
    say(f"explicit restore {shape} {dtype}: rel err {err:.3e}")
    assert err < (BF16_TOL if dtype == "bf16" else F32_TOL)
    assert info["k_eff"].cpu().tolist() == oinfo.k_eff


def test_explicit_restore_headline_sampled():
    case = workloads.config2("768x3072", batch=6)
    out, _ = run_case(case, restore="explicit")
    got = host64(out)
    for idx in ([0], [5]):
        check_bf16_sample(f"explicit restore 768x3072 matrix {idx[0]}", got[idx[0]], case, idx, restore="explicit")


def test_explicit_restore_k0_is_baseline_bitwise():
    case = workloads.config2("768x768", batch=2)
    base, _ = run_case(case, k=0)
    expl, _ = run_case(case, k=0, restore="explicit")
    assert torch.equal(base, expl)
