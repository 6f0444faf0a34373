"""GPU parity of the (deflated) PSD projection against the CPU oracle.

Tolerance: relative Frobenius error 1e-4 (float32 path against the float64
oracle); deflated and positive counts must match exactly.
"""
import numpy as np
import pytest
import torch

import paper_2609_21102_amd as sd
import workloads
from oracle import psd as opsd
from tests.gpu_util import host64, rel_fro, say

pytestmark = pytest.mark.gpu

TOL = 1e-4


def gpu_psd(case, k=None, **kw):
    k = case.k if k is None else k
    z = torch.from_numpy(case.z).cuda()
    q = torch.from_numpy(np.ascontiguousarray(case.qwarm[:, :k])).cuda() if k > 0 else None
    out, info = sd.psd_project(z, k, case.steps, q, subspace_iters=case.subspace_iters, gamma=case.gamma,
                               info=True, **kw)
    torch.cuda.synchronize()
    return out, info, q


@pytest.mark.parametrize("n,k", [(100, 0), (100, 8), (256, 8), (300, 16), (129, 4)])
def test_small(n, k):
    case = workloads.small_psd(n, k=max(k, 1), case_id=n)
    say(f"psd n={n} k={k}")
    out, info, q = gpu_psd(case, k)
    z = case.z.astype(np.float64)
    if k > 0:
        want, vnext, oinfo = opsd.psd_project_deflated(z, case.qwarm[:, :k].astype(np.float64), steps=case.steps,
                                                       gamma=case.gamma, subspace_iters=case.subspace_iters)
        assert int(info["n_deflated"]) == oinfo.n_deflated
        assert int(info["n_positive"]) == oinfo.n_positive
        np.testing.assert_allclose(info["ritz"].cpu().numpy(), oinfo.ritz, rtol=1e-5, atol=1e-5)
        assert rel_fro(host64(q), vnext) < 1e-4
        theta = oinfo.theta
    else:
        want, theta = opsd.psd_project(z, steps=case.steps)
    err = rel_fro(host64(out), want)
    say(f"  rel err {err:.3e}  theta {float(info['theta']):.6g} vs {theta:.6g}")
    assert err < TOL
    assert abs(float(info["theta"]) - theta) <= 1e-5 * theta
    o = out.cpu().numpy()
    assert np.array_equal(o, o.T)


def test_gate_and_counts():
    case = workloads.small_psd(200, k=8, n_dom=3, dom=(100.0, 300.0), case_id=7)
    out, info, _ = gpu_psd(case, 8, tau=0.1, window=6)
    want, _, oinfo = opsd.psd_project_deflated(case.z.astype(np.float64), case.qwarm.astype(np.float64),
                                               steps=case.steps, gamma=case.gamma, tau=0.1, window=6,
                                               subspace_iters=case.subspace_iters)
    assert int(info["n_deflated"]) == oinfo.n_deflated == 3
    assert int(info["n_positive"]) == oinfo.n_positive
    assert rel_fro(host64(out), want) < TOL


def test_gate_off_is_baseline_bitwise():
    case = workloads.small_psd(160, k=6, n_dom=0, case_id=9)
    base, _, _ = gpu_psd(case, 0)
    gated, info, _ = gpu_psd(case, 6, tau=0.1, window=4)
    assert int(info["n_deflated"]) == 0
    assert torch.equal(base, gated)


def test_quintic_filter_table():
    case = workloads.small_psd(180, k=8, case_id=11)
    table = np.array([[1.875, -1.25, 0.375]] * case.steps, dtype=np.float32)
    out, info, _ = gpu_psd(case, 8, poly=table, poly_degree=5)
    want, _, _ = opsd.psd_project_deflated(case.z.astype(np.float64), case.qwarm.astype(np.float64),
                                           table=table.astype(np.float64), gamma=case.gamma,
                                           subspace_iters=case.subspace_iters)
    assert rel_fro(host64(out), want) < TOL


def test_zero_matrix():
    z = torch.zeros(64, 64, device="cuda")
    assert torch.count_nonzero(sd.psd_project(z, 0, 10)) == 0


@pytest.mark.slow
def test_config4_full():
    case = workloads.config4()
    say("config4 n=4096 k=16")
    out, info, q = gpu_psd(case)
    want, vnext, oinfo = opsd.psd_project_deflated(case.z.astype(np.float64), case.qwarm.astype(np.float64),
                                                   steps=case.steps, gamma=case.gamma,
                                                   subspace_iters=case.subspace_iters)
    err = rel_fro(host64(out), want)
    say(f"  rel err {err:.3e}")
    assert err < TOL
    assert int(info["n_deflated"]) == oinfo.n_deflated
    assert int(info["n_positive"]) == oinfo.n_positive
