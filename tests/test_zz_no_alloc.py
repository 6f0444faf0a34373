"""The allocation-free Muon entry point (sd_msign_deflated_noalloc) against
sd_msign_deflated_ex on the same inputs and options: two calls in a row, the
second with a smaller input, on both paths; oversize calls and a caller
workspace are rejected with nothing enqueued."""
import ctypes

import numpy as np
import pytest
import torch

import paper_2609_21102_amd as sd
import workloads
from tests.gpu_util import dev_tensor, say

pytestmark = pytest.mark.gpu


def _noalloc(x, k, steps, coeffs, out, opts=None):
    b, m, n = x.shape
    dtype = sd.SD_DTYPE_BF16 if x.dtype == torch.bfloat16 else sd.SD_DTYPE_F32
    table = np.ascontiguousarray(coeffs, dtype=np.float32)
    o = opts if opts is not None else sd.msign_opts()
    rc = sd.lib().sd_msign_deflated_noalloc(b, m, n, k, steps, table.ctypes.data_as(ctypes.c_void_p), dtype,
                                            ctypes.c_void_p(x.data_ptr()), ctypes.c_void_p(out.data_ptr()),
                                            ctypes.byref(o), ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    return rc


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_noalloc_matches_ex_two_calls(dtype):
    for shape, k, cid in (((3, 128, 256), 4, 61), ((1, 96, 160), 2, 62)):
        case = workloads.small_muon(*shape, dtype=dtype, k=k, case_id=cid)
        x = dev_tensor(case.x, dtype)
        want = sd.msign(x, k, case.steps, case.coeffs)
        got = torch.full_like(x, 7.0)
        rc = _noalloc(x, k, case.steps, case.coeffs, got)
        torch.cuda.synchronize()
        say(f"noalloc {dtype} {shape} k={k}: rc {rc}, equal {torch.equal(got, want)}")
        assert rc == 0
        assert torch.equal(got, want)


def test_noalloc_rejects_oversize_and_workspace():
    case = workloads.config2("768x3072", batch=4)   # about 150 MB of scratch at bf16
    x = dev_tensor(case.x, "bf16")
    out = torch.full_like(x, 7.0)
    assert sd.msign_workspace_bytes(4, 768, 3072, 8, sd.SD_DTYPE_BF16) > (64 << 20)
    rc = _noalloc(x, 8, 5, case.coeffs, out)
    torch.cuda.synchronize()
    assert rc == -5   # SD_ERR_WORKSPACE
    assert bool((out == 7.0).all())
    small = dev_tensor(workloads.small_muon(1, 64, 128, dtype="bf16", k=2, case_id=63).x, "bf16")
    ws = torch.empty(1 << 20, dtype=torch.uint8, device="cuda")
    o = sd.msign_opts(workspace=ws.data_ptr(), workspace_bytes=ws.numel())
    assert _noalloc(small, 2, 5, workloads.muon_coeff_table(5), torch.empty_like(small), opts=o) == -1
