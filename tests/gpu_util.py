"""Shared helpers of the GPU parity tests."""
import numpy as np
import torch

import workloads


def dev_tensor(case_x: np.ndarray, dtype: str):
    """Seeded host input -> device tensor with the same bits."""
    if dtype == "bf16":
        t = torch.from_numpy(case_x.view(np.int16).copy()).view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(case_x, dtype=np.float32))
    return t.cuda()


def host64(t) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def rel_fro(got: np.ndarray, want: np.ndarray) -> float:
    den = np.linalg.norm(want)
    return float(np.linalg.norm(got - want) / (den if den > 0 else 1.0))


def rel_fro_batched(got, want):
    return [rel_fro(g, w) for g, w in zip(got, want)]


def say(*a):
    print(*a, flush=True)


__all__ = ["dev_tensor", "host64", "rel_fro", "rel_fro_batched", "say", "workloads"]
