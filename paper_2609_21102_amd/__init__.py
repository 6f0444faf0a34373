"""Python binding of libsdeflate (the deflated polynomial matrix filters on
MI355X). Argument marshalling only: every step runs in the HIP library.

    msign(x, k, steps, coeffs=None, ...)        -> sd_msign_deflated_ex
    msign_groups([{x, k, steps, ...}, ...])      -> sd_msign_groups
    psd_project(X, k, steps, qwarm=None, ...)    -> sd_psd_project_deflated_ex
    admm_diag(C, b, iters, k, qwarm, ...)        -> sd_admm_diag

Tensors are torch CUDA (ROCm) tensors; torch provides device memory and the
current stream. The library must be built (paper_2609_21102_amd/build.py);
nothing here falls back to another implementation.
"""
from __future__ import annotations

import ctypes
import os
import re

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libsdeflate.so")
HEADER = os.path.join(os.path.dirname(HERE), "include", "sdeflate.h")

SD_OK = 0
SD_DTYPE_F32 = 0
SD_DTYPE_BF16 = 1
SD_RESTORE = {"padded": 0, "explicit": 1}
SD_PREC = {"f32": 0, "f16": 1}
SD_SCALE = {"lanczos": 0, "frobenius": 1}
MUON_QUINTIC = (3.4445, -4.7750, 2.0315)

_c_int_p = ctypes.POINTER(ctypes.c_int)
_c_float_p = ctypes.POINTER(ctypes.c_float)


class MsignOpts(ctypes.Structure):
    _fields_ = [
        ("oversample", ctypes.c_int),
        ("power_iters", ctypes.c_int),
        ("gamma", ctypes.c_float),
        ("tau", ctypes.c_float),
        ("seed", ctypes.c_uint64),
        ("sketch", ctypes.c_void_p),
        ("workspace", ctypes.c_void_p),
        ("workspace_bytes", ctypes.c_size_t),
        ("k_eff_out", ctypes.c_void_p),
        ("nu_out", ctypes.c_void_p),
        ("s_out", ctypes.c_void_p),
        ("status_dev", ctypes.c_void_p),
        ("restore", ctypes.c_int),
        ("window", ctypes.c_int),
    ]


class MsignGroup(ctypes.Structure):
    _fields_ = [
        ("batch", ctypes.c_int),
        ("m", ctypes.c_int),
        ("n", ctypes.c_int),
        ("k", ctypes.c_int),
        ("steps", ctypes.c_int),
        ("coeffs", ctypes.c_void_p),
        ("dtype", ctypes.c_int),
        ("input", ctypes.c_void_p),
        ("out", ctypes.c_void_p),
        ("opts", ctypes.POINTER(MsignOpts)),
    ]


class PsdOpts(ctypes.Structure):
    _fields_ = [
        ("subspace_iters", ctypes.c_int),
        ("lanczos_steps", ctypes.c_int),
        ("gamma", ctypes.c_float),
        ("tau", ctypes.c_float),
        ("window", ctypes.c_int),
        ("poly_degree", ctypes.c_int),
        ("poly", ctypes.c_void_p),
        ("seed", ctypes.c_uint64),
        ("workspace", ctypes.c_void_p),
        ("workspace_bytes", ctypes.c_size_t),
        ("n_deflated_out", ctypes.c_void_p),
        ("n_positive_out", ctypes.c_void_p),
        ("theta_out", ctypes.c_void_p),
        ("ritz_out", ctypes.c_void_p),
        ("status_dev", ctypes.c_void_p),
        ("precision", ctypes.c_int),
        ("scale_mode", ctypes.c_int),
    ]


_LIB = None


class MsignParam(ctypes.Structure):
    _fields_ = [
        ("input", ctypes.c_void_p),
        ("out", ctypes.c_void_p),
        ("m", ctypes.c_int),
        ("n", ctypes.c_int),
    ]


def _declare(lib):
    vp, i, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t
    sig = {
        "sd_msign": (i, [i, i, i, i, vp, vp, vp, vp]),
        "sd_msign_deflated": (i, [i, i, i, i, i, vp, vp, vp, vp]),
        "sd_msign_bf16": (i, [i, i, i, i, vp, vp, vp, vp]),
        "sd_msign_deflated_bf16": (i, [i, i, i, i, i, vp, vp, vp, vp]),
        "sd_msign_deflated_ex": (i, [i, i, i, i, i, vp, i, vp, vp, ctypes.POINTER(MsignOpts), vp]),
        "sd_msign_workspace_bytes": (sz, [i, i, i, i, i, ctypes.POINTER(MsignOpts)]),
        "sd_msign_deflated_noalloc": (i, [i, i, i, i, i, vp, i, vp, vp, ctypes.POINTER(MsignOpts), vp]),
        "sd_msign_groups": (i, [i, ctypes.POINTER(MsignGroup), vp]),
        "sd_msign_params": (i, [i, ctypes.POINTER(MsignParam), i, i, vp, i, ctypes.POINTER(MsignOpts), vp]),
        "sd_msign_opts_default": (None, [ctypes.POINTER(MsignOpts)]),
        "sd_psd_project": (i, [i, i, vp, vp, vp]),
        "sd_psd_project_deflated": (i, [i, i, i, vp, vp, vp, vp]),
        "sd_psd_project_deflated_ex": (i, [i, i, i, vp, vp, vp, ctypes.POINTER(PsdOpts), vp]),
        "sd_psd_workspace_bytes": (sz, [i, i, ctypes.POINTER(PsdOpts)]),
        "sd_admm_diag": (i, [i, i, i, ctypes.c_float, vp, vp, vp, vp, vp, i, vp, i, ctypes.POINTER(PsdOpts), vp, vp,
                             vp]),
        "sd_admm_workspace_bytes": (sz, [i, i, i, ctypes.POINTER(PsdOpts)]),
        "sd_psd_opts_default": (None, [ctypes.POINTER(PsdOpts)]),
        "sd_sketch": (i, [i, i, i, ctypes.c_uint64, vp, vp]),
        "sd_sketch_host": (i, [i, i, i, ctypes.c_uint64, vp]),
        "sd_status_string": (ctypes.c_char_p, [i]),
        "sd_profile_set": (None, [ctypes.c_uint]),
        "sd_profile_read": (i, [i, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_longlong)]),
        "sd_profile_reset": (None, []),
        "sd_version": (i, []),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args


def lib():
    """Load libsdeflate.so (raises if it has not been built)."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run python paper_2609_21102_amd/build.py")
        _LIB = ctypes.CDLL(LIB_PATH)
        _declare(_LIB)
    return _LIB


def header_functions() -> list[str]:
    """Names of the entry points declared in include/sdeflate.h."""
    with open(HEADER) as f:
        text = f.read()
    return sorted(set(re.findall(r"\b(sd_[a-z0-9_]+)\s*\(", text)))


class SdError(RuntimeError):
    def __init__(self, status: int, where: str):
        msg = lib().sd_status_string(status).decode()
        super().__init__(f"{where}: {msg} ({status})")
        self.status = status


def _check(rc: int, where: str):
    if rc != SD_OK:
        raise SdError(rc, where)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _host_table(coeffs, steps, width):
    if coeffs is None:
        return None, None
    arr = np.ascontiguousarray(np.asarray(coeffs, dtype=np.float32).reshape(steps, width))
    return arr, arr.ctypes.data_as(ctypes.c_void_p)


def msign_opts(**kw) -> MsignOpts:
    o = MsignOpts()
    lib().sd_msign_opts_default(ctypes.byref(o))
    for k, v in kw.items():
        setattr(o, k, v)
    return o


def psd_opts(**kw) -> PsdOpts:
    o = PsdOpts()
    lib().sd_psd_opts_default(ctypes.byref(o))
    for k, v in kw.items():
        setattr(o, k, v)
    return o


def msign(x, k: int = 0, steps: int = 5, coeffs=None, *, oversample: int = 8, power_iters: int = 1,
          gamma: float = 1.01, tau: float = 0.0, seed: int = 0, sketch=None, out=None, workspace=None,
          restore: str = "padded", window: int = 0, info: bool = False, stream=None):
    """(Deflated) polar factor of every matrix of x ([B, m, n] or [m, n], bf16 or
    float32, contiguous, on the GPU). k = 0 is the undeflated baseline.
    Returns out (same shape and dtype), and with info=True a dict of device
    tensors k_eff [B], nu [B], s [B, r] (r = window when tau > 0 and window > 0,
    else k) and status (int32 [1], the SD_FLAG_* bits the call raised).
    restore: "padded" (Alg. 1) or "explicit" (U_k V_k^T added after the
    filter). window: the gate's window r (tau > 0)."""
    import torch
    squeeze = x.dim() == 2
    xb = x.unsqueeze(0) if squeeze else x
    if xb.dim() != 3 or not xb.is_cuda or not xb.is_contiguous():
        raise ValueError("x must be a contiguous CUDA tensor of shape [B, m, n] or [m, n]")
    if xb.dtype == torch.bfloat16:
        dtype = SD_DTYPE_BF16
    elif xb.dtype == torch.float32:
        dtype = SD_DTYPE_F32
    else:
        raise TypeError("x must be bfloat16 or float32")
    b, m, n = xb.shape
    if out is None:
        out = torch.empty_like(xb)
    else:
        out = out.view(b, m, n)
    table, tptr = _host_table(coeffs, steps, 3)
    dev = xb.device
    keff = torch.empty(b, dtype=torch.int32, device=dev) if info else None
    nu = torch.empty(b, dtype=torch.float32, device=dev) if info else None
    kw = window if (tau > 0 and window > 0 and k > 0) else k
    sv = torch.empty((b, max(kw, 1)), dtype=torch.float32, device=dev) if info else None
    status = torch.zeros(1, dtype=torch.int32, device=dev) if info else None
    o = msign_opts(oversample=oversample, power_iters=power_iters, gamma=gamma, tau=tau, seed=seed,
                   restore=SD_RESTORE[restore], window=window)
    if sketch is not None:
        s_ = min(m, n)
        rp = min(s_, kw + oversample)
        if (not sketch.is_cuda or sketch.dtype != torch.float32 or not sketch.is_contiguous()
                or tuple(sketch.shape) != (b, rp, s_)):
            raise ValueError(f"sketch must be a contiguous float32 CUDA tensor of shape {(b, rp, s_)}")
        o.sketch = sketch.data_ptr()
    if workspace is not None:
        o.workspace = workspace.data_ptr()
        o.workspace_bytes = workspace.numel() * workspace.element_size()
    if info:
        o.k_eff_out, o.nu_out, o.s_out = keff.data_ptr(), nu.data_ptr(), sv.data_ptr()
        o.status_dev = status.data_ptr()
    rc = lib().sd_msign_deflated_ex(b, m, n, k, steps, tptr, dtype, _ptr(xb), _ptr(out), ctypes.byref(o),
                                    _stream(stream))
    _check(rc, "sd_msign_deflated_ex")
    del table
    res = out[0] if squeeze else out
    if info:
        return res, {"k_eff": keff, "nu": nu, "s": sv[:, :kw], "status": status}
    return res


def msign_groups(groups, *, stream=None):
    """One Muon step over several shape groups (sd_msign_groups): groups is a
    list of dicts with keys x ([B, m, n] bf16 or float32 CUDA tensor), k,
    steps, and optionally coeffs, out, oversample, power_iters, gamma, tau,
    seed, window, restore. The groups run concurrently inside the library; returns the list of
    outputs."""
    import torch
    n = len(groups)
    arr = (MsignGroup * n)()
    keep = []
    outs = []
    for i, g in enumerate(groups):
        x = g["x"]
        if x.dim() != 3 or not x.is_cuda or not x.is_contiguous():
            raise ValueError("every x must be a contiguous CUDA tensor [B, m, n]")
        if x.dtype == torch.bfloat16:
            dtype = SD_DTYPE_BF16
        elif x.dtype == torch.float32:
            dtype = SD_DTYPE_F32
        else:
            raise TypeError("x must be bfloat16 or float32")
        b, m, nn = x.shape
        steps = int(g.get("steps", 5))
        out = g.get("out")
        out = torch.empty_like(x) if out is None else out
        table, tptr = _host_table(g.get("coeffs"), steps, 3)
        o = msign_opts(**{key: g[key] for key in ("oversample", "power_iters", "gamma", "tau", "seed", "window")
                          if key in g})
        o.restore = SD_RESTORE[g.get("restore", "padded")]
        keep += [table, o]
        arr[i] = MsignGroup(b, m, nn, int(g.get("k", 0)), steps, tptr.value if tptr is not None else None, dtype,
                            x.data_ptr(), out.data_ptr(), ctypes.pointer(o))
        outs.append(out)
    _check(lib().sd_msign_groups(n, arr, _stream(stream)), "sd_msign_groups")
    del keep
    return outs


def msign_params(xs, k: int = 0, steps: int = 5, coeffs=None, *, outs=None, stream=None, **opts):
    """One Muon step over a parameter list (sd_msign_params): xs is a list of
    2-D CUDA tensors (all bfloat16 or all float32, contiguous), grouped by
    shape inside the library (m x n and n x m together); outs (optional) the
    output tensors, one per input (an output may be its own input). Options as
    in msign (oversample, power_iters, gamma, tau, seed, window, restore).
    Returns the outputs."""
    import torch
    if not xs:
        raise ValueError("empty parameter list")
    dt = xs[0].dtype
    if dt == torch.bfloat16:
        dtype = SD_DTYPE_BF16
    elif dt == torch.float32:
        dtype = SD_DTYPE_F32
    else:
        raise TypeError("parameters must be bfloat16 or float32")
    outs = [torch.empty_like(x) for x in xs] if outs is None else list(outs)
    arr = (MsignParam * len(xs))()
    for i, (x, y) in enumerate(zip(xs, outs)):
        if x.dim() != 2 or not x.is_cuda or not x.is_contiguous() or x.dtype != dt:
            raise ValueError("every parameter must be a contiguous 2-D CUDA tensor of one dtype")
        if y.shape != x.shape or y.dtype != dt or not y.is_contiguous():
            raise ValueError("every output must match its parameter's shape and dtype")
        arr[i] = MsignParam(x.data_ptr(), y.data_ptr(), x.shape[0], x.shape[1])
    table, tptr = _host_table(coeffs, steps, 3)
    o = msign_opts(**{key: v for key, v in opts.items() if key != "restore"})
    o.restore = SD_RESTORE[opts.get("restore", "padded")]
    _check(lib().sd_msign_params(len(xs), arr, k, steps, tptr, dtype, ctypes.byref(o), _stream(stream)),
           "sd_msign_params")
    del table
    return outs


def sketch_host(batch: int, s: int, rp: int, seed: int = 0) -> np.ndarray:
    """The library's Gaussian sketches computed on the host: [batch, rp, s]."""
    out = np.empty((batch, rp, s), dtype=np.float32)
    _check(lib().sd_sketch_host(batch, s, rp, seed, out.ctypes.data_as(ctypes.c_void_p)), "sd_sketch_host")
    return out


def sketch(batch: int, s: int, rp: int, seed: int = 0, stream=None):
    """The library's Gaussian sketches drawn on the GPU: [batch, rp, s] float32."""
    import torch
    out = torch.empty((batch, rp, s), dtype=torch.float32, device="cuda")
    _check(lib().sd_sketch(batch, s, rp, seed, _ptr(out), _stream(stream)), "sd_sketch")
    return out


def msign_workspace_bytes(batch, m, n, k, dtype=SD_DTYPE_BF16, **kw) -> int:
    o = msign_opts(**kw)
    return int(lib().sd_msign_workspace_bytes(batch, m, n, k, dtype, ctypes.byref(o)))


def psd_project(X, k: int = 0, steps: int = 10, qwarm=None, *, subspace_iters: int = 1,
                lanczos_steps: int = 20, gamma: float = 1.1, tau: float = 0.0, window: int = 1,
                poly=None, poly_degree: int = 3, seed: int = 0, precision: str = "f32", out=None,
                workspace=None, info: bool = False, scale: str = "lanczos", stream=None):
    """(Deflated) projection of the symmetric float32 X [n, n] onto the PSD cone.
    qwarm [n, k] (float32) is the warm-start basis and is overwritten with the
    next basis. precision: "f32", or "f16" (the sign filter's products take
    fp16 operands). scale: "lanczos" (App. E.1) or "frobenius" (theta =
    ||R||_F). Returns out, and with info=True a dict of device tensors
    n_deflated, n_positive, theta, ritz."""
    import torch
    if X.dim() != 2 or X.shape[0] != X.shape[1] or X.dtype != torch.float32 or not X.is_contiguous():
        raise ValueError("X must be a contiguous float32 [n, n] CUDA tensor")
    n = X.shape[0]
    if out is None:
        out = torch.empty_like(X)
    width = (poly_degree + 1) // 2
    table, tptr = _host_table(poly, steps, width)
    dev = X.device
    o = psd_opts(subspace_iters=subspace_iters, lanczos_steps=lanczos_steps, gamma=gamma, tau=tau,
                 window=window, poly_degree=poly_degree, seed=seed, precision=SD_PREC[precision],
                 scale_mode=SD_SCALE[scale])
    if tptr is not None:
        o.poly = tptr.value
    if workspace is not None:
        o.workspace = workspace.data_ptr()
        o.workspace_bytes = workspace.numel() * workspace.element_size()
    res = {}
    if info:
        res = {"n_deflated": torch.empty(1, dtype=torch.int32, device=dev),
               "n_positive": torch.empty(1, dtype=torch.int32, device=dev),
               "theta": torch.empty(1, dtype=torch.float32, device=dev),
               "ritz": torch.empty(max(k, 1), dtype=torch.float32, device=dev),
               "status": torch.zeros(1, dtype=torch.int32, device=dev)}
        o.n_deflated_out = res["n_deflated"].data_ptr()
        o.status_dev = res["status"].data_ptr()
        o.n_positive_out = res["n_positive"].data_ptr()
        o.theta_out = res["theta"].data_ptr()
        o.ritz_out = res["ritz"].data_ptr()
    if k > 0 and (qwarm is None or qwarm.shape != (n, k) or qwarm.dtype != torch.float32
                  or not qwarm.is_contiguous()):
        raise ValueError("qwarm must be a contiguous float32 [n, k] CUDA tensor")
    rc = lib().sd_psd_project_deflated_ex(n, k, steps, _ptr(X), _ptr(qwarm) if k > 0 else None, _ptr(out),
                                          ctypes.byref(o), _stream(stream))
    _check(rc, "sd_psd_project_deflated_ex")
    del table
    if info:
        res["ritz"] = res["ritz"][:k]
        return out, res
    return out


def admm_diag(C, b, iters: int, k: int = 0, qwarm=None, *, X=None, S=None, y=None, steps: int = 10,
              sigma: float = 1.0, warmup: int = 100, tau: float = 0.1, window: int = 1, gamma: float = 1.1,
              precision: str = "f32", seed: int = 0, poly=None, poly_degree: int = 3, stream=None):
    """`iters` ADMM iterations (sd_admm_diag) for min <C, X> s.t. diag(X) = b,
    X PSD, continuing from X, S, y (zeros when None; updated in place).
    qwarm [n, k] is the tracked basis (updated in place). Returns
    (X, S, y, eta [iters], n_deflated [iters]) as device tensors."""
    import torch
    n = C.shape[0]
    dev = C.device
    X = torch.zeros_like(C) if X is None else X
    S = torch.zeros_like(C) if S is None else S
    y = torch.zeros(n, dtype=torch.float32, device=dev) if y is None else y
    eta = torch.empty(max(iters, 1), dtype=torch.float32, device=dev)
    ndef = torch.empty(max(iters, 1), dtype=torch.int32, device=dev)
    # no tracked basis (k = 0): the undeflated projection, no gate
    o = psd_opts(gamma=gamma, tau=tau if k > 0 else 0.0, window=window, precision=SD_PREC[precision], seed=seed,
                 poly_degree=poly_degree)
    table, tptr = _host_table(poly, steps, (poly_degree + 1) // 2)
    if tptr is not None:
        o.poly = tptr.value
    rc = lib().sd_admm_diag(n, iters, steps, sigma, _ptr(C), _ptr(b), _ptr(X), _ptr(S), _ptr(y), k,
                            _ptr(qwarm) if k > 0 else None, warmup, ctypes.byref(o), _ptr(eta), _ptr(ndef),
                            _stream(stream))
    _check(rc, "sd_admm_diag")
    return X, S, y, eta[:iters], ndef[:iters]


STAGES = {"ns_gram": 0, "ns_poly": 1, "ns_update": 2, "sketch": 3, "cholqr": 4, "small": 5,
          "lowrank": 6, "lanczos": 7, "restore": 8}


def profile_set(*stages: str):
    """Bracket every launch of the named stages with HIP events."""
    mask = 0
    for s in stages:
        mask |= 1 << STAGES[s]
    lib().sd_profile_set(mask)


def profile_read(stage: str) -> tuple[float, int]:
    """(total milliseconds, launches) recorded for a stage (synchronizes)."""
    ms = ctypes.c_double()
    n = ctypes.c_longlong()
    _check(lib().sd_profile_read(STAGES[stage], ctypes.byref(ms), ctypes.byref(n)), "sd_profile_read")
    return ms.value, n.value


def profile_reset():
    lib().sd_profile_reset()


def psd_workspace_bytes(n, k, **kw) -> int:
    o = psd_opts(**kw)
    return int(lib().sd_psd_workspace_bytes(n, k, ctypes.byref(o)))
