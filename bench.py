#!/usr/bin/env python3
"""Benchmark of the deflated polar factor on one MI355X.

Workload (one "step" = one call that runs the whole path): 24 matrices of
768 x 3072 in bfloat16 (the largest group of a GPT-2-small-shaped Muon
batch), spectra with 8 spikes geometric from 50 down to 5 over a log-uniform
bulk in [1e-4, 1]; deflation rank k = 8, oversample 8, one power iteration,
5 steps of Muon's quintic (3.4445, -4.7750, 2.0315), gamma = 1.01. Inputs are
seeded and synthetic and are resident in HBM before the timed region.

Prints one JSON line: matrices/s (value), the achieved TFLOP/s against the
bf16 MFMA peak, a roofline entry for the dominant kernel (the iterate update
X <- a X + B X, timed with HIP events inside the timed region; its
arithmetic intensity, about 120 flop per byte, is below the bf16 ridge of
about 310, so it is priced against HBM) and the CPU oracle timed on a bounded
sample of the same workload.

--copy-calibration adds one plain device copy of 256 MiB before the timed
region, the reference kernel for scaling the FETCH_SIZE / WRITE_SIZE counters.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

MFMA_BF16_PEAK_TFLOPS = 2500.0
HBM_PEAK_GBS = 8000.0


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def ns_flops_per_matrix(s: int, l: int, steps: int) -> float:
    """Algorithmic flops of the filter for one s x l matrix: per step the Gram
    X X^T and A^2 counted once per symmetric entry, plus the 2 s^2 l update."""
    return steps * (s * (s + 1) * (l + s) + 2.0 * s * s * l)


def front_flops_per_matrix(s: int, l: int, k: int, rp: int, power_iters: int) -> float:
    """Sketch, power and projection products (2 s l r' each) plus the two
    rank-k passes (residual norm and start)."""
    return (2 + 2 * power_iters) * 2.0 * s * l * rp + 2 * 2.0 * s * l * k


def update_bytes_per_matrix(s: int, l: int, steps: int) -> float:
    """Algorithmic HBM bytes of the iterate updates of one s x l matrix,
    averaged over the call's launches. The bf16 iterate is stored as hi (bf16)
    plus an 8-bit residual. Every step reads B (bf16, s x s), the operand hi
    (s x l; the a X term takes hi from the same tiles) and the residuals; the
    first steps - 1 write the next hi and residuals, the last writes the bf16
    output."""
    inner = 2.0 * s * s + 2 * s * l + 1 * s * l + 3 * s * l
    last = 2.0 * s * s + 2 * s * l + 1 * s * l + 2 * s * l
    return ((steps - 1) * inner + last) / steps


KERNEL_SOURCES = ("gemm.hpp", "common.hpp", "msign.hip")


def kernel_hash() -> str:
    """Hash of the sources the update kernel is built from."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2609_21102_amd", "csrc")
    for name in KERNEL_SOURCES:
        with open(os.path.join(csrc, name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic():
    """HBM bytes per update launch from the committed counter summary, or
    None when the kernel sources changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", "ns_update_768x3072_bf16_traffic.txt")
    if not os.path.exists(path):
        return None
    vals = {}
    with open(path) as f:
        for line in f:
            if "=" in line and not line.startswith("#"):
                k, v = line.split("=", 1)
                vals[k.strip()] = v.strip()
    if vals.get("kernel_hash") != kernel_hash():
        return None
    try:
        return float(vals["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def cpu_baseline(case, seconds: float) -> dict:
    """The oracle (bf16-contract mode, float64) on whole matrices of the same
    workload, cycling through the batch until `seconds` have passed."""
    from threadpoolctl import threadpool_info
    from oracle import muon as omuon
    from oracle import rng as orng
    b = case.x.shape[0]
    s = min(case.x.shape[1:])
    rp = min(s, case.k + case.oversample)
    threads = max([d.get("num_threads", 1) for d in threadpool_info()] or [1])
    done, t0 = 0, time.perf_counter()
    while True:
        idx = done % b
        omuon.msign_deflated(case.x64[idx:idx + 1], case.k, case.coeffs, oversample=case.oversample,
                             power_iters=case.power_iters, gamma=case.gamma, mode="bf16",
                             sketches=[orng.sketch(0, idx, s, rp)])
        done += 1
        if time.perf_counter() - t0 >= seconds:
            break
    dt = time.perf_counter() - t0
    return {"value": done / dt, "unit": "matrices/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{done} matrices 768x3072 (cycling through the batch of {b}), float64 oracle in "
                      f"bf16-contract mode, {dt:.1f} s"}


def _timed(step, steps: int, warmup: int) -> float:
    """Milliseconds per step over `steps` timed calls after `warmup` calls."""
    import torch
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(steps):
        step()
    end.record()
    torch.cuda.synchronize()
    return start.elapsed_time(end) / steps


def _psd_update_roofline(sd, step, steps: int, n: int, precision: str) -> dict:
    """Roofline of the filter's update product X B (symmetric tiles: the
    n (n + 1) / 2 entries of the upper triangle, 2 n flops each, counted once)
    against the dense MFMA peak of its operand type."""
    ms, launches = _stage_time(sd, step, steps, "ns_update")
    n_pad = -(-n // 128) * 128
    flops = float(n_pad) * (n_pad + 1) * n_pad
    avg_ms = ms / max(launches, 1)
    tf = flops / (avg_ms / 1e3) / 1e12
    peak = 157.3 if precision == "f32" else MFMA_BF16_PEAK_TFLOPS   # fp16 dense = bf16 dense
    return {"bound": "mfma", "kernel": "filter update X <- a X + X B, symmetric tiles "
            + ("(gemm_dma_kernel, fp16 operands)" if precision == "f16" else "(gemm_kernel, fp32)"),
            "achieved": tf, "peak": peak, "unit": "TFLOP/s", "frac": tf / peak, "traffic": None,
            "flops_per_launch": flops, "avg_launch_us": avg_ms * 1e3, "launches": launches}


def _stage_time(sd, step, steps: int, stage: str) -> tuple[float, int]:
    """(milliseconds, launches) of one stage over `steps` further calls, each
    launch bracketed by HIP events on the library's stream."""
    import torch
    torch.cuda.synchronize()
    sd.profile_reset()
    sd.profile_set(stage)
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    sd.profile_set()
    return sd.profile_read(stage)


def _filter_table(args):
    """(steps, table, degree) of the PSD filter: 10 cubic Bjorck-Bowie steps,
    or (--poly quintic7) 7 steps of the degree-5 map (15/8, -5/4, 3/8), the
    shape of the paper's T = 7 degree-5 fp16 composite (whose own
    coefficients are not printed)."""
    if args.poly == "quintic7":
        return 7, [(1.875, -1.25, 0.375)] * 7, 5
    return 10, None, 3


def other_workload(args) -> int:
    """Throughput of the configurations other than the benchmark line, each
    with the roofline of its dominant kernel: the bf16 iterate update (HBM)
    for the Muon groups, the symmetric filter update (MFMA) for the PSD and
    ADMM workloads."""
    import torch
    import paper_2609_21102_amd as sd
    import workloads

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    def muon_groups(cases):
        groups = []
        for c in cases:
            x = torch.from_numpy(c.x.view(np.int16).copy()).view(torch.bfloat16).to(dev)
            groups.append(dict(x=x, out=torch.empty_like(x), k=c.k, steps=c.steps, coeffs=c.coeffs,
                               oversample=c.oversample, power_iters=c.power_iters, gamma=c.gamma))
        flops = 0.0
        for c in cases:
            b, m, n = c.x.shape
            s, l = min(m, n), max(m, n)
            rp = min(s, c.k + c.oversample)
            flops += b * (ns_flops_per_matrix(s, l, c.steps) + front_flops_per_matrix(s, l, c.k, rp, c.power_iters))
        return groups, flops

    if args.workload in ("c2-step", "paper-step", "c3"):
        if args.workload == "c2-step":
            cases = [workloads.config2(g) for g in ("768x768", "768x2304", "768x3072")]
        elif args.workload == "paper-step":
            cases = [workloads.paper_scale_group(g) for g in ("1280x1280", "5120x1280")]
        else:
            cases = [workloads.config3("768x3072")]
        groups, flops = muon_groups(cases)
        nmat = sum(c.x.shape[0] for c in cases)
        if args.sequential:
            def step():
                for g in groups:
                    sd.msign(g["x"], g["k"], g["steps"], g["coeffs"], oversample=g["oversample"],
                             power_iters=g["power_iters"], gamma=g["gamma"], out=g["out"])
        else:
            def step():
                sd.msign_groups(groups)
        ms = _timed(step, args.steps, args.warmup)
        # the update of every group, summed: bytes and flops over launch time
        # (grouped calls run groups concurrently, so launch times overlap)
        upd_ms, upd_n = _stage_time(sd, step, args.steps, "ns_update")
        upd_bytes = upd_flops = 0.0
        for c in cases:
            b_, s_, l_ = c.x.shape[0], min(c.x.shape[1:]), max(c.x.shape[1:])
            upd_bytes += b_ * update_bytes_per_matrix(s_, l_, c.steps) * c.steps * args.steps
            upd_flops += b_ * 2.0 * s_ * s_ * l_ * c.steps * args.steps
        sec = upd_ms / 1e3
        if upd_flops / upd_bytes > MFMA_BF16_PEAK_TFLOPS * 1e12 / (HBM_PEAK_GBS * 1e9):
            ach = upd_flops / sec / 1e12
            roof = {"bound": "mfma", "achieved": ach, "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                    "frac": ach / MFMA_BF16_PEAK_TFLOPS, "flops_per_launch": upd_flops / max(upd_n, 1)}
        else:
            ach = upd_bytes / sec / 1e9
            roof = {"bound": "hbm", "achieved": ach, "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": ach / HBM_PEAK_GBS,
                    "bytes_per_launch": upd_bytes / max(upd_n, 1)}
        roof.update({"kernel": "iterate update X <- a X + B X (gemm_dma_kernel, EpiUpdateHL), all groups",
                     "traffic": None, "avg_launch_us": upd_ms * 1e3 / max(upd_n, 1), "launches": upd_n,
                     "flop_per_byte": upd_flops / upd_bytes})
        desc = " + ".join(f"{c.x.shape[0]} x {c.x.shape[1]} x {c.x.shape[2]}" for c in cases)
        res = {"metric": f"deflated msign matrices/s ({args.workload}: {desc} bf16)", "value": nmat / (ms / 1e3),
               "unit": "matrices/s", "ms_per_step": ms, "tflops": flops / (ms / 1e3) / 1e12,
               "mfma_frac": flops / (ms / 1e3) / 1e12 / MFMA_BF16_PEAK_TFLOPS, "steps": args.steps,
               "warmup": args.warmup, "dtype": "bf16", "data": "synthetic",
               "config": {"workload": args.workload, "groups": desc,
                          "launch": "one call per group" if args.sequential else "sd_msign_groups",
                          "k": [c.k for c in cases], "filter_steps": [c.steps for c in cases]},
               "roofline": roof}
    elif args.workload == "admm":
        # ADMM on a max-cut relaxation of the size of the paper's n = 5000
        # instances (planted-bisection random graph), tracked basis K = 64
        # (the widest Rayleigh-Ritz block the library solves), r = 32, tau = 0.1;
        # one step = 10 iterations with the gate open, continuing the state.
        n, k, r, chunk = 5000, 64, 32, 10
        steps, table, degree = _filter_table(args)
        case = workloads.planted_maxcut(n, case_id=0)
        C = torch.from_numpy(case.c).to(dev)
        bvec = torch.from_numpy(case.b).to(dev)
        g = np.random.default_rng(11).standard_normal((n, k))
        q = torch.from_numpy(np.linalg.qr(g)[0].astype(np.float32)).to(dev)
        X, S, y = torch.zeros_like(C), torch.zeros_like(C), torch.zeros(n, dtype=torch.float32, device=dev)
        last = {}

        def call():
            _, _, _, eta, ndef = sd.admm_diag(C, bvec, chunk, k, q, X=X, S=S, y=y, steps=steps, warmup=0,
                                              tau=0.1, window=r, precision=args.precision, poly=table,
                                              poly_degree=degree)
            last.update(eta=eta, ndef=ndef)

        ms = _timed(call, args.steps, args.warmup)
        roof = _psd_update_roofline(sd, call, args.steps, n, args.precision)
        # per step: X^2 and the update (n^3 each, symmetric), plus A^2 for a quintic
        flops = chunk * ((2.0 if degree == 3 else 3.0) * n ** 3 * steps + 2.0 * n ** 3)
        peak = 157.3 if args.precision == "f32" else MFMA_BF16_PEAK_TFLOPS
        res = {"metric": f"ADMM iterations/s (max-cut SDP, n = {n}, K = {k}, {steps} degree-{degree} steps, "
                         f"{args.precision} filter products)",
               "value": chunk * 1e3 / ms, "unit": "iterations/s", "ms_per_step": ms,
               "tflops": flops / (ms / 1e3) / 1e12, "mfma_frac": flops / (ms / 1e3) / 1e12 / peak,
               "steps": args.steps, "warmup": args.warmup, "dtype": args.precision, "data": "synthetic",
               "config": {"workload": "admm", "n": n, "k": k, "window": r, "tau": 0.1, "filter_steps": steps,
                          "filter_degree": degree,
                          "iterations_per_step": chunk, "final_eta": float(last["eta"][-1]),
                          "final_n_deflated": int(last["ndef"][-1])},
               "roofline": roof}
    else:
        if args.workload == "c4":
            case = workloads.config4()
            z = torch.from_numpy(case.z).to(dev)
            lam, q0 = None, torch.from_numpy(np.ascontiguousarray(case.qwarm)).to(dev)
            n, k, steps, sub = case.z.shape[0], case.k, case.steps, case.subspace_iters
        else:
            z, lam, _, q0 = workloads.config5_device(16384)
            n, k, steps, sub = 16384, 32, 10, 1
        if args.poly != "cubic":
            steps, table, degree = _filter_table(args)
        else:
            table, degree = None, 3
        q = q0.clone()
        out = torch.empty_like(z)
        ws = torch.empty(sd.psd_workspace_bytes(n, k, precision=sd.SD_PREC[args.precision], poly_degree=degree),
                         dtype=torch.uint8, device=dev)

        def call():
            q.copy_(q0)   # every timed call starts from the same warm basis
            sd.psd_project(z, k, steps, q, subspace_iters=sub, gamma=1.1, out=out, workspace=ws,
                           precision=args.precision, poly=table, poly_degree=degree)

        ms = _timed(call, args.steps, args.warmup)
        roof = _psd_update_roofline(sd, call, args.steps, n, args.precision)
        # cubic filter: X^2 and X X^2 are both symmetric and computed on upper-triangle
        # tiles (n^3 each per step), a quintic adds A^2; the restore product R g is a full 2 n^3
        flops = (2.0 if degree == 3 else 3.0) * n ** 3 * steps + 2.0 * n ** 3
        peak = 157.3 if args.precision == "f32" else MFMA_BF16_PEAK_TFLOPS   # fp16 dense = bf16 dense
        res = {"metric": f"deflated PSD projections/s ({args.workload}: n = {n}, k = {k}, {steps} degree-{degree} "
                         f"steps, {args.precision} filter products)",
               "value": 1e3 / ms, "unit": "projections/s", "ms_per_step": ms,
               "tflops": flops / (ms / 1e3) / 1e12, "mfma_frac": flops / (ms / 1e3) / 1e12 / peak,
               "steps": args.steps, "warmup": args.warmup, "dtype": args.precision, "data": "synthetic",
               "config": {"workload": args.workload, "n": n, "k": k, "filter_steps": steps,
                          "filter_degree": degree, "subspace_iters": sub},
               "roofline": roof}
    r = res["roofline"]
    log(f"bench {args.workload}: {res['ms_per_step']:.3f} ms per call, {res['value']:.1f} {res['unit']}, "
        f"{res['tflops']:.1f} TFLOP/s; {r['kernel']}: {r['avg_launch_us']:.1f} us avg over {r['launches']} launches, "
        f"{r['achieved']:.0f} {r['unit']} ({100 * r['frac']:.1f}% of peak)")
    print(json.dumps(res), flush=True)
    return 0


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--baseline", action="store_true", help="time the undeflated filter (k = 0) instead")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run one plain 256 MiB device copy before timing (counter calibration)")
    ap.add_argument("--workload", default="headline",
                    choices=["headline", "c2-step", "c3", "paper-step", "c4", "c5", "admm"],
                    help="headline: the benchmark line; the others time further configurations "
                         "(one JSON line each, no roofline or CPU baseline)")
    ap.add_argument("--precision", default="f32", choices=["f32", "f16"],
                    help="c4 / c5 / admm: arithmetic of the sign filter's products")
    ap.add_argument("--poly", default="cubic", choices=["cubic", "quintic7"],
                    help="c4 / c5 / admm: the filter: 10 cubic steps, or 7 steps of the degree-5 map "
                         "(the shape of the paper's T = 7 fp16 composite)")
    ap.add_argument("--sequential", action="store_true",
                    help="c2-step / paper-step: one call per group on one stream instead of sd_msign_groups")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        log("bench.py: the library runs on a single GPU; --gpus must be 1 "
            "(sharding the batch by matrix across GPUs is not implemented)")
        return 2

    import torch
    import paper_2609_21102_amd as sd
    import workloads

    if args.workload != "headline":
        return other_workload(args)

    case = workloads.config2("768x3072")
    b, m, n = case.x.shape
    k = 0 if args.baseline else case.k
    s, l = min(m, n), max(m, n)
    rp = min(s, k + case.oversample) if k else 0
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    x = torch.from_numpy(case.x.view(np.int16).copy()).view(torch.bfloat16).to(dev)
    out = torch.empty_like(x)
    ws = torch.empty(sd.msign_workspace_bytes(b, m, n, k, sd.SD_DTYPE_BF16), dtype=torch.uint8, device=dev)
    coeffs = case.coeffs

    def step():
        sd.msign(x, k, case.steps, coeffs, oversample=case.oversample, power_iters=case.power_iters,
                 gamma=case.gamma, out=out, workspace=ws)

    log(f"bench: {b} x {m} x {n} bf16, k={k}, warmup {args.warmup}, steps {args.steps}")
    if args.copy_calibration:
        src = torch.ones(64 << 20, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    sd.profile_reset()
    sd.profile_set("ns_update")
    # an event after every step on the call's stream: the per-step spread
    marks = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    marks[0].record()
    for t in range(args.steps):
        step()
        marks[t + 1].record()
    torch.cuda.synchronize()
    sd.profile_set()
    ms_total = marks[0].elapsed_time(marks[-1])
    per_step = sorted(marks[t].elapsed_time(marks[t + 1]) for t in range(args.steps))
    pct = lambda q: per_step[min(len(per_step) - 1, int(round(q * (len(per_step) - 1))))]
    upd_ms, upd_n = sd.profile_read("ns_update")
    ms_per_step = ms_total / args.steps
    value = b * args.steps / (ms_total / 1e3)
    flops = b * (ns_flops_per_matrix(s, l, case.steps) + (front_flops_per_matrix(s, l, k, rp, case.power_iters)
                                                          if k else 0.0))
    tflops = flops / (ms_per_step / 1e3) / 1e12
    # totals over the timed calls, divided by the update launches they made
    # (one per filter step, or two when a call runs its batch in two halves)
    n_launch = max(upd_n, 1)
    upd_flops = 2.0 * s * s * l * b * case.steps * args.steps / n_launch
    upd_bytes = update_bytes_per_matrix(s, l, case.steps) * b * case.steps * args.steps / n_launch
    upd_avg_ms = upd_ms / n_launch
    upd_tflops = upd_flops / (upd_avg_ms / 1e3) / 1e12
    upd_gbs = upd_bytes / (upd_avg_ms / 1e3) / 1e9
    log(f"bench: {ms_per_step:.3f} ms/step, {value:.0f} matrices/s, {tflops:.1f} TFLOP/s; "
        f"update kernel {upd_avg_ms * 1e3:.1f} us avg over {upd_n} launches "
        f"({upd_gbs:.0f} GB/s algorithmic, {upd_tflops:.1f} TFLOP/s)")

    result = {
        "metric": "deflated msign matrices/s + TFLOP/s (% MFMA peak), batched 768x3072 bf16",
        "value": value,
        "unit": "matrices/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "ms_per_step_p10_p50_p90": [pct(0.1), pct(0.5), pct(0.9)],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"deflated msign, {b} x {m} x {n} bf16, k={k}, oversample {case.oversample}, "
                               f"{case.power_iters} power iteration, {case.steps} Muon quintic steps",
                   "batch": b, "m": m, "n": n, "k": k, "steps": case.steps, "parallelism": "single GPU"},
        "tflops": tflops,
        "mfma_frac": tflops / MFMA_BF16_PEAK_TFLOPS,
        "roofline": {"bound": "hbm", "kernel": "iterate update X <- a X + B X (gemm_dma_kernel, EpiUpdateHL)",
                     "achieved": upd_gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": upd_gbs / HBM_PEAK_GBS, "traffic": measured_traffic(),
                     "bytes_per_launch": upd_bytes, "avg_launch_us": upd_avg_ms * 1e3,
                     "launches": upd_n, "tflops": upd_tflops,
                     "mfma_frac": upd_tflops / MFMA_BF16_PEAK_TFLOPS, "kernel_hash": kernel_hash()},
    }
    if not args.no_cpu_baseline:
        log("bench: timing the CPU oracle on a sample")
        result["cpu_baseline"] = cpu_baseline(case, args.cpu_seconds)
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
