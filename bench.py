#!/usr/bin/env python3
"""Benchmark of the deflated polar factor on one MI355X.

Workload (one "step" = one call that runs the whole path): 24 matrices of
768 x 3072 in bfloat16 (the largest group of a GPT-2-small-shaped Muon
batch), spectra with 8 spikes geometric from 50 down to 5 over a log-uniform
bulk in [1e-4, 1]; deflation rank k = 8, oversample 8, one power iteration,
5 steps of Muon's quintic (3.4445, -4.7750, 2.0315), gamma = 1.01. Inputs are
seeded and synthetic and are resident in HBM before the timed region.

Prints one JSON line:
  value      matrices/s over the timed calls;
  roofline   the dominant kernel, the iterate update X <- a X + B X, priced
             against the bf16 dense MFMA peak with its algorithmic flops
             2 s^2 l per matrix, timed with HIP events around every launch
             inside the timed region; traffic = HBM bytes per launch measured
             by two rocprofv3 counter passes (FETCH_SIZE, WRITE_SIZE) run as
             child processes before the timed region and scaled by the same
             counters' reading of a plain 256 MiB copy, beside the algorithmic
             bytes (read X and B, write X, all bf16);
  stages     every stage of the call from HIP events around each launch (a
             second pass of the same calls): the filter's Gram, polynomial and
             update against the MFMA peak, the sketch products, the rank-k
             passes and the CholeskyQR panels against HBM, each with its
             algorithmic work, and the whole-call fraction sum_stage
             max(flops / MFMA peak, bytes / HBM peak) / call time;
  cpu_baseline  the CPU oracle on a bounded sample, at all cores and at one
             thread.
--workload selects further configurations (one JSON line each).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
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


def update_bytes_algorithmic(s: int, l: int) -> float:
    """Algorithmic HBM bytes of one update X <- a X + B X of an s x l matrix
    with a bf16 carry: read X and B, write X (2 bytes each)."""
    return 2.0 * s * l + 2.0 * s * s + 2.0 * s * l


def stage_work(s: int, l: int, k: int, rp: int, power_iters: int, steps: int) -> dict:
    """Algorithmic work per matrix of one call, by stage: (flops, bytes)."""
    return {
        # the chain's HBM bytes per step: X read by the Gram and the update and
        # written by the update (bf16), A written by the Gram and read by the
        # polynomial (fp32, the b A term), B written and read (bf16)
        "ns_gram": (steps * s * (s + 1.0) * l, steps * (2.0 * s * l + 4.0 * s * s)),
        "ns_poly": (steps * s * (s + 1.0) * s, steps * (4.0 * s * s + 2.0 * s * s)),
        "ns_update": (steps * 2.0 * s * s * l, steps * update_bytes_algorithmic(s, l)),
        # each pass over X reads it once (bf16); 2 s l r' flops
        "sketch": ((2 + 2 * power_iters) * 2.0 * s * l * rp, (2 + 2 * power_iters) * 2.0 * s * l),
        # residual norm: read X; padded start: read X, write X0 (bf16 carry)
        "lowrank": (2 * 2.0 * s * l * k, 2.0 * s * l + 4.0 * s * l),
        # two passes over an fp32 panel per CholeskyQR: the l-side panel
        # 1 + J times, the s-side J times
        "cholqr": (0.0, 2 * 4.0 * rp * ((1 + power_iters) * l + power_iters * s)),
        "small": (0.0, 0.0),
    }


STAGE_PEAKS = {"mfma_bf16_tflops": 2500.0, "hbm_gbs": 8000.0}


def stage_table(times_ms: dict, work: dict, batch: int, calls: int, call_ms: float) -> dict:
    """Per-stage achieved rates and roofline fractions, plus the whole-call
    fraction: sum over stages of max(flops / MFMA peak, bytes / HBM peak),
    divided by the call time."""
    out, ideal_ms = {}, 0.0
    for name, (ms_tot, launches) in times_ms.items():
        flops, nbytes = work[name]
        flops *= batch
        nbytes *= batch
        ms = ms_tot / calls
        t_mfma = flops / (STAGE_PEAKS["mfma_bf16_tflops"] * 1e12) * 1e3
        t_hbm = nbytes / (STAGE_PEAKS["hbm_gbs"] * 1e9) * 1e3
        bound = "mfma" if t_mfma >= t_hbm else "hbm"
        if flops == 0 and nbytes == 0:
            bound = "latency"
        ideal_ms += max(t_mfma, t_hbm)
        row = {"ms_per_call": ms, "launches_per_call": launches / calls, "bound": bound}
        if flops:
            row["tflops"] = flops / (ms / 1e3) / 1e12
        if nbytes:
            row["gbs"] = nbytes / (ms / 1e3) / 1e9
        if bound != "latency":
            row["frac"] = max(t_mfma, t_hbm) / ms
        out[name] = row
    chain = [n for n in ("ns_gram", "ns_poly", "ns_update") if n in out]
    if chain:
        fl = sum(work[n][0] for n in chain) * batch
        ms = sum(out[n]["ms_per_call"] for n in chain)
        out["ns_chain"] = {"ms_per_call": ms, "tflops": fl / (ms / 1e3) / 1e12, "bound": "mfma",
                           "frac": fl / (ms / 1e3) / 1e12 / STAGE_PEAKS["mfma_bf16_tflops"]}
    return {"stages": out, "whole_call_frac": ideal_ms / call_ms, "ideal_ms": ideal_ms, "call_ms": call_ms}


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


# ------------------------------------------------- live counter passes ----
COUNTERS = ("FETCH_SIZE", "WRITE_SIZE")
COPY_KIB = 262144.0   # the calibration copy moves 256 MiB each way


def counter_pass_child(args) -> int:
    """Child of a rocprofv3 --pmc run: one calibration copy of 256 MiB and a
    few calls of the workload (input from the parent's file)."""
    import torch
    import paper_2609_21102_amd as sd
    import workloads
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    case = workloads.config2("768x3072", batch=1)   # parameters only; the input comes from the file
    bits = np.load(args.counter_pass)
    b, m, n = bits.shape
    x = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(dev)
    out = torch.empty_like(x)
    src = torch.ones(64 << 20, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst
    for _ in range(3):
        sd.msign(x, case.k, case.steps, case.coeffs, oversample=case.oversample, power_iters=case.power_iters,
                 gamma=case.gamma, out=out)
    torch.cuda.synchronize()
    return 0


KERNEL_KEYS = {"ns_update": "EpiUpdateHL", "ns_gram": "EpiGramT", "ns_poly": "EpiPoly",
               "sketch": "EpiStoreRowsSplit", "lowrank": "lowrank_kernel"}


def counter_traffic(bits: np.ndarray, timeout_s: float = 180.0) -> dict:
    """HBM bytes per launch of the path's kernels from two rocprofv3 --pmc
    passes over child runs of this script (no GPU is used in this process
    before they end). Returns {"per_kernel": {stage: bytes per launch}, ...}
    or {"error": ...}."""
    import shutil
    import sqlite3
    import subprocess
    import tempfile
    exe = shutil.which("rocprofv3") or "/opt/rocm/bin/rocprofv3"
    if not os.path.exists(exe):
        return {"error": "rocprofv3 not found"}
    tmp = tempfile.mkdtemp(prefix="sdbench_", dir="/tmp")
    xpath = os.path.join(tmp, "x.npy")
    np.save(xpath, bits)
    env = dict(os.environ, TMPDIR="/tmp")
    readings = {}
    for ctr in COUNTERS:
        outdir = os.path.join(tmp, ctr)
        cmd = [exe, "--pmc", ctr, "-d", outdir, "-o", "run", "--", sys.executable, os.path.abspath(__file__),
               "--counter-pass", xpath]
        log(f"bench: counter pass {ctr}")
        proc = subprocess.Popen(cmd, cwd="/tmp", env=env, stdout=subprocess.DEVNULL, stderr=subprocess.PIPE,
                                start_new_session=True)
        try:
            _, err = proc.communicate(timeout=timeout_s)
        except subprocess.TimeoutExpired:
            os.killpg(proc.pid, 9)
            proc.wait()
            return {"error": f"counter pass {ctr} timed out"}
        dbs = [os.path.join(d, f) for d, _, fs in os.walk(outdir) for f in fs if f.endswith("_results.db")]
        if proc.returncode != 0 and not dbs:
            return {"error": f"counter pass {ctr} failed ({proc.returncode}): {err.decode()[-300:]}"}
        if not dbs:
            return {"error": f"counter pass {ctr}: no results database"}
        rows = []
        for db in dbs:
            con = sqlite3.connect(db)
            rows += con.execute("select kernel_name, dispatch_id, sum(value) from counters_collection "
                                "where counter_name = ? group by dispatch_id", (ctr,)).fetchall()
            con.close()
        readings[ctr] = rows
    shutil.rmtree(tmp, ignore_errors=True)

    def mean_kib(ctr, key):
        vals = [v for name, _, v in readings[ctr] if key in name]
        return (sum(vals) / len(vals), len(vals)) if vals else (None, 0)

    fetch_copy, _ = mean_kib("FETCH_SIZE", "copyBuffer")
    write_copy, _ = mean_kib("WRITE_SIZE", "copyBuffer")
    if not fetch_copy or not write_copy:
        return {"error": "calibration copy not found in the counter data"}
    ff, wf = COPY_KIB / fetch_copy, COPY_KIB / write_copy
    per = {}
    for stage, key in KERNEL_KEYS.items():
        f, nf = mean_kib("FETCH_SIZE", key)
        w, nw = mean_kib("WRITE_SIZE", key)
        if f is not None and w is not None:
            per[stage] = {"bytes_per_launch": 1024.0 * (f * ff + w * wf), "dispatches": nf}
    return {"per_kernel": per, "fetch_factor": ff, "write_factor": wf,
            "method": "rocprofv3 --pmc FETCH_SIZE, then WRITE_SIZE (KiB per dispatch), on child runs of "
                      "this script with 3 calls; scaled by the counters' reading of a 256 MiB device copy"}


def cpu_baseline(case, seconds: float) -> dict:
    """The oracle (bf16-contract mode, float64) on whole matrices of the same
    workload, cycling through the batch until `seconds` have passed: once
    with the BLAS threads it finds, once with one thread."""
    from threadpoolctl import threadpool_info, threadpool_limits
    from oracle import muon as omuon
    from oracle import rng as orng
    b = case.x.shape[0]
    s = min(case.x.shape[1:])
    rp = min(s, case.k + case.oversample)
    threads = max([d.get("num_threads", 1) for d in threadpool_info()] or [1])

    def run(sec):
        done, t0 = 0, time.perf_counter()
        while True:
            idx = done % b
            omuon.msign_deflated(case.x64[idx:idx + 1], case.k, case.coeffs, oversample=case.oversample,
                                 power_iters=case.power_iters, gamma=case.gamma, mode="bf16",
                                 sketches=[orng.sketch(0, idx, s, rp)])
            done += 1
            if time.perf_counter() - t0 >= sec:
                return done, time.perf_counter() - t0

    done, dt = run(seconds)
    with threadpool_limits(limits=1):
        done1, dt1 = run(seconds)
    return {"value": done / dt, "unit": "matrices/s", "cores": int(threads), "kind": "oracle",
            "value_1thread": done1 / dt1, "cpu_model": cpu_model(), "os_cpu_count": os.cpu_count(),
            "sample": f"{done} matrices 768x3072 at {threads} threads in {dt:.1f} s and {done1} at one thread "
                      f"in {dt1:.1f} s (cycling through the batch of {b}), float64 oracle in bf16-contract mode"}


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
        if args.param_list:
            # the same matrices as a parameter list (every other non-square
            # member as its transpose), grouped inside the library
            c0 = cases[0]
            if any((c.k, c.steps, c.oversample, c.power_iters, c.gamma) != (c0.k, c0.steps, c0.oversample,
                                                                          c0.power_iters, c0.gamma) or
                   not np.array_equal(c.coeffs, c0.coeffs) for c in cases):
                raise SystemExit("--param-list needs one k, filter and option set across the groups")
            xs = []
            for g in groups:
                for b_ in range(g["x"].shape[0]):
                    mat = g["x"][b_]
                    xs.append(mat.t().contiguous() if (b_ % 2 and mat.shape[0] != mat.shape[1]) else mat)
            outs = [torch.empty_like(x_) for x_ in xs]

            def step():
                sd.msign_params(xs, c0.k, c0.steps, c0.coeffs, outs=outs, oversample=c0.oversample,
                                power_iters=c0.power_iters, gamma=c0.gamma)
        elif args.sequential:
            def step():
                for g in groups:
                    sd.msign(g["x"], g["k"], g["steps"], g["coeffs"], oversample=g["oversample"],
                             power_iters=g["power_iters"], gamma=g["gamma"], out=g["out"])
        else:
            def step():
                sd.msign_groups(groups)
        ms = _timed(step, args.steps, args.warmup)
        # the update of every group, summed: flops over launch time (grouped
        # calls run groups concurrently, so launch times overlap), against the
        # bf16 MFMA peak
        upd_ms, upd_n = _stage_time(sd, step, args.steps, "ns_update")
        upd_bytes = upd_flops = 0.0
        for c in cases:
            b_, s_, l_ = c.x.shape[0], min(c.x.shape[1:]), max(c.x.shape[1:])
            upd_bytes += b_ * update_bytes_algorithmic(s_, l_) * c.steps * args.steps
            upd_flops += b_ * 2.0 * s_ * s_ * l_ * c.steps * args.steps
        ach = upd_flops / (upd_ms / 1e3) / 1e12
        roof = {"bound": "mfma", "achieved": ach, "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": ach / MFMA_BF16_PEAK_TFLOPS, "flops_per_launch": upd_flops / max(upd_n, 1),
                "algorithmic_bytes_per_launch": upd_bytes / max(upd_n, 1),
                "kernel": "iterate update X <- a X + B X (gemm_dma_kernel, EpiUpdateHL), all groups",
                "traffic": None, "avg_launch_us": upd_ms * 1e3 / max(upd_n, 1), "launches": upd_n,
                "flop_per_byte": upd_flops / upd_bytes}
        desc = " + ".join(f"{c.x.shape[0]} x {c.x.shape[1]} x {c.x.shape[2]}" for c in cases)
        res = {"metric": f"deflated msign matrices/s ({args.workload}: {desc} bf16)", "value": nmat / (ms / 1e3),
               "unit": "matrices/s", "ms_per_step": ms, "tflops": flops / (ms / 1e3) / 1e12,
               "mfma_frac": flops / (ms / 1e3) / 1e12 / MFMA_BF16_PEAK_TFLOPS, "steps": args.steps,
               "warmup": args.warmup, "dtype": "bf16", "data": "synthetic",
               "config": {"workload": args.workload, "groups": desc,
                          "launch": ("sd_msign_params (parameter list)" if args.param_list else
                                     "one call per group" if args.sequential else "sd_msign_groups"),
                          "k": [c.k for c in cases], "filter_steps": [c.steps for c in cases]},
               "roofline": roof}
    elif args.workload == "peaks":
        # re-measured roofline constants: dense bf16 MFMA rate, HBM copy and
        # read bandwidth (grid-stride and chunk-per-work-group streams, the
        # chunked read also with non-temporal loads), and the vendor batched GEMM (torch.bmm) on the
        # update's shape (24 x (768 x 768) x (768 x 3072) bf16) for scale
        import ctypes
        plib = ctypes.CDLL(os.path.join(ROOT, "paper_2609_21102_amd", "libsdpeaks.so"))
        vp = ctypes.c_void_p
        plib.sdp_mfma_bf16.argtypes = [ctypes.c_int, ctypes.c_int, vp, vp]
        plib.sdp_copy.argtypes = [vp, vp, ctypes.c_size_t, ctypes.c_int, vp]
        plib.sdp_read.argtypes = [vp, ctypes.c_size_t, ctypes.c_int, vp, vp]
        plib.sdp_copy_chunk.argtypes = [vp, vp, ctypes.c_size_t, vp]
        plib.sdp_read_chunk.argtypes = [vp, ctypes.c_size_t, ctypes.c_int, vp, vp]
        st = vp(torch.cuda.current_stream().cuda_stream)
        sink = torch.zeros(1 << 16, dtype=torch.float32, device=dev)
        csink = torch.zeros((1 << 30) // 16 // 1024, dtype=torch.float32, device=dev)   # one per chunk

        def timed_ms(fn, reps=5):
            fn()
            torch.cuda.synchronize()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            for _ in range(reps):
                fn()
            b.record()
            torch.cuda.synchronize()
            return a.elapsed_time(b) / reps

        blocks, iters = 4096, 256
        mf_ms = timed_ms(lambda: plib.sdp_mfma_bf16(blocks, iters, vp(sink.data_ptr()), st))
        mf_tf = blocks * 4 * 8 * iters * 32768.0 / (mf_ms / 1e3) / 1e12
        n4 = (1 << 30) // 16
        src = torch.ones(n4 * 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        cp_ms = timed_ms(lambda: plib.sdp_copy(vp(src.data_ptr()), vp(dst.data_ptr()), n4, 256 * 32, st))
        rd_ms = timed_ms(lambda: plib.sdp_read(vp(src.data_ptr()), n4, 256 * 32, vp(sink.data_ptr()), st))
        cpc_ms = timed_ms(lambda: plib.sdp_copy_chunk(vp(src.data_ptr()), vp(dst.data_ptr()), n4, st))
        rdc_ms = timed_ms(lambda: plib.sdp_read_chunk(vp(src.data_ptr()), n4, 0, vp(csink.data_ptr()), st))
        rdn_ms = timed_ms(lambda: plib.sdp_read_chunk(vp(src.data_ptr()), n4, 1, vp(csink.data_ptr()), st))
        del src, dst
        a16 = torch.randn(24, 768, 768, device=dev).to(torch.bfloat16)
        x16 = torch.randn(24, 768, 3072, device=dev).to(torch.bfloat16)
        bmm_ms = timed_ms(lambda: torch.bmm(a16, x16), reps=20)
        bmm_tf = 2.0 * 768 * 768 * 3072 * 24 / (bmm_ms / 1e3) / 1e12
        res = {"metric": "measured peaks (bf16 MFMA TFLOP/s, HBM GB/s)", "value": mf_tf, "unit": "TFLOP/s",
               "ms_per_step": mf_ms, "steps": 5, "warmup": 1, "dtype": "bf16", "data": "synthetic",
               "config": {"workload": "peaks"},
               "measured_peaks": {"mfma_bf16_tflops": mf_tf, "mfma_bf16_frac_of_2500": mf_tf / 2500.0,
                                  "hbm_copy_gbs": 2.0 * (1 << 30) / (cp_ms / 1e3) / 1e9,
                                  "hbm_read_gbs": 1.0 * (1 << 30) / (rd_ms / 1e3) / 1e9,
                                  "hbm_copy_chunk_gbs": 2.0 * (1 << 30) / (cpc_ms / 1e3) / 1e9,
                                  "hbm_read_chunk_gbs": 1.0 * (1 << 30) / (rdc_ms / 1e3) / 1e9,
                                  "hbm_read_chunk_nt_gbs": 1.0 * (1 << 30) / (rdn_ms / 1e3) / 1e9,
                                  "bmm_update_shape_us": bmm_ms * 1e3, "bmm_update_shape_tflops": bmm_tf},
               "roofline": {"bound": "mfma", "kernel": "sdp_mfma_bf16_kernel", "achieved": mf_tf, "peak": 2500.0,
                            "unit": "TFLOP/s", "frac": mf_tf / 2500.0, "traffic": None,
                            "avg_launch_us": mf_ms * 1e3, "launches": 5}}
        log(f"bench peaks: {json.dumps(res['measured_peaks'])}")
        print(json.dumps(res), flush=True)
        return 0
    elif args.workload == "c1":
        # config 1: one float32 256 x 256 matrix, k = 4, 2 power iterations, 5 steps;
        # a step is one call (latency-bound: every stage is one small launch)
        case = workloads.config1()
        x = torch.from_numpy(case.x.astype(np.float32)).to(dev)
        out = torch.empty_like(x)
        ws = torch.empty(sd.msign_workspace_bytes(1, 256, 256, case.k, sd.SD_DTYPE_F32, power_iters=case.power_iters),
                         dtype=torch.uint8, device=dev)

        def step():
            sd.msign(x, case.k, case.steps, case.coeffs, oversample=case.oversample,
                     power_iters=case.power_iters, gamma=case.gamma, out=out, workspace=ws)

        ms = _timed(step, args.steps, args.warmup)
        upd_ms, upd_n = _stage_time(sd, step, args.steps, "ns_update")
        s_ = l_ = 256
        fl = 2.0 * s_ * s_ * l_
        ach = fl / (upd_ms / max(upd_n, 1) / 1e3) / 1e12
        work = stage_work(s_, l_, case.k, min(s_, case.k + case.oversample), case.power_iters, case.steps)
        flops = sum(w[0] for w in work.values())
        res = {"metric": "deflated msign matrices/s (config 1: 1 x 256 x 256 float32, k = 4, J = 2, 5 steps)",
               "value": 1e3 / ms, "unit": "matrices/s", "ms_per_step": ms, "tflops": flops / (ms / 1e3) / 1e12,
               "steps": args.steps, "warmup": args.warmup, "dtype": "f32", "data": "synthetic",
               "config": {"workload": "c1", "m": 256, "n": 256, "k": case.k, "power_iters": case.power_iters,
                          "filter_steps": case.steps},
               "roofline": {"bound": "mfma", "kernel": "iterate update X <- a X + B X (gemm_kernel, fp32)",
                            "achieved": ach, "peak": 157.3, "unit": "TFLOP/s", "frac": ach / 157.3,
                            "traffic": None, "avg_launch_us": upd_ms * 1e3 / max(upd_n, 1), "launches": upd_n,
                            "flops_per_launch": fl}}
    elif args.workload == "admm":
        # ADMM on a max-cut relaxation of the size of the paper's n = 5000
        # instances (--admm-n: another size; planted-bisection random graph),
        # tracked basis of the paper's width K = ceil(0.05 n) with window
        # r = ceil(0.025 n) (--admm-k: another width, r = ceil(K / 2)),
        # tau = 0.1; one step = 10 iterations with the gate open, continuing
        # the state.
        n, chunk = args.admm_n, 10
        k = args.admm_k if args.admm_k else math.ceil(0.05 * n)
        r = math.ceil(0.025 * n) if not args.admm_k else max(1, (k + 1) // 2)
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
        stage_ms = {}
        for stg in ("ns_gram", "ns_poly", "ns_update", "restore", "sketch", "cholqr", "small", "lowrank", "lanczos"):
            t_ms, t_n = _stage_time(sd, call, args.steps, stg)
            if t_n:
                stage_ms[stg] = {"ms_per_iteration": t_ms / (args.steps * chunk), "launches_per_iteration":
                                 t_n / (args.steps * chunk)}
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
               "roofline": roof, "stages": stage_ms}
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
    ap.add_argument("--steps", type=int, default=None,
                    help="timed calls (default: 50 for the Muon workloads, 20 for the PSD and ADMM ones)")
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--baseline", action="store_true", help="time the undeflated filter (k = 0) instead")
    ap.add_argument("--no-counters", action="store_true", help="skip the rocprofv3 counter passes")
    ap.add_argument("--counter-pass", default=None, help=argparse.SUPPRESS)
    ap.add_argument("--workload", default="headline",
                    choices=["headline", "c1", "c2-step", "c3", "paper-step", "c4", "c5", "admm", "peaks"],
                    help="headline: the benchmark line; the others time further configurations "
                         "(one JSON line each, no roofline or CPU baseline)")
    ap.add_argument("--precision", default="f32", choices=["f32", "f16"],
                    help="c4 / c5 / admm: arithmetic of the sign filter's products")
    ap.add_argument("--poly", default="cubic", choices=["cubic", "quintic7"],
                    help="c4 / c5 / admm: the filter: 10 cubic steps, or 7 steps of the degree-5 map "
                         "(the shape of the paper's T = 7 fp16 composite)")
    ap.add_argument("--admm-n", type=int, default=5000, help="admm: order n of the SDP")
    ap.add_argument("--admm-k", type=int, default=0, help="admm: width K of the tracked basis (default ceil(0.05 n))")
    ap.add_argument("--param-list", action="store_true",
                    help="c2-step / paper-step: the matrices as a parameter list through sd_msign_params")
    ap.add_argument("--sequential", action="store_true",
                    help="c2-step / paper-step: one call per group on one stream instead of sd_msign_groups")
    args = ap.parse_args()
    if args.steps is None:
        args.steps = 50 if args.workload in ("headline", "c1", "c2-step", "c3", "paper-step") else 20
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        log("bench.py: the library runs on a single GPU; --gpus must be 1 "
            "(sharding the batch by matrix across GPUs is not implemented)")
        return 2

    if args.counter_pass:
        return counter_pass_child(args)

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
    # HBM traffic: two counter passes in child processes, before this
    # process uses the GPU
    traffic = None
    if not args.no_counters and not args.baseline:
        traffic = counter_traffic(case.x)
        if "error" in traffic:
            log(f"bench: counters unavailable: {traffic['error']}")
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
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # timed region: events around every update launch (on the library's
    # stream) and after every call
    sd.profile_reset()
    sd.profile_set("ns_update")
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
    work = stage_work(s, l, k, rp, case.power_iters, case.steps)
    flops = b * sum(w[0] for w in work.values()) if k else b * (work["ns_gram"][0] + work["ns_poly"][0] +
                                                                 work["ns_update"][0])
    tflops = flops / (ms_per_step / 1e3) / 1e12
    n_launch = max(upd_n, 1)
    upd_flops = b * work["ns_update"][0] * args.steps / n_launch
    upd_alg_bytes = b * work["ns_update"][1] * args.steps / n_launch
    upd_avg_ms = upd_ms / n_launch
    upd_tflops = upd_flops / (upd_avg_ms / 1e3) / 1e12

    # every stage, from events around each launch over the same number of calls
    names = ["ns_gram", "ns_poly", "ns_update"] + (["sketch", "cholqr", "small", "lowrank"] if k else ["lowrank"])
    sd.profile_reset()
    sd.profile_set(*names)
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    sd.profile_set()
    times = {nm: sd.profile_read(nm) for nm in names}
    table = stage_table(times, work, b, args.steps, ms_per_step)
    log(f"bench: {ms_per_step:.3f} ms/step, {value:.0f} matrices/s, {tflops:.1f} TFLOP/s; "
        f"update {upd_avg_ms * 1e3:.1f} us avg over {upd_n} launches ({upd_tflops:.1f} TFLOP/s, "
        f"{100 * upd_tflops / MFMA_BF16_PEAK_TFLOPS:.1f}% of bf16 MFMA); whole call "
        f"{100 * table['whole_call_frac']:.1f}% of its roofline")
    for nm, row in table["stages"].items():
        log(f"  {nm:10s} {row['ms_per_call'] * 1e3:8.1f} us/call  {row['bound']:7s} "
            + (f"{100 * row['frac']:5.1f}%" if "frac" in row else ""))

    tr = None
    if traffic and "per_kernel" in traffic and "ns_update" in traffic["per_kernel"]:
        tr = traffic["per_kernel"]["ns_update"]["bytes_per_launch"]
        for nm, row in traffic["per_kernel"].items():
            if nm in table["stages"]:
                table["stages"][nm]["traffic_bytes_per_launch"] = row["bytes_per_launch"]
    roofline = {"bound": "mfma", "kernel": "iterate update X <- a X + B X (gemm_dma_kernel, EpiUpdateHL)",
                "achieved": upd_tflops, "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": upd_tflops / MFMA_BF16_PEAK_TFLOPS, "traffic": tr,
                "flops_per_launch": upd_flops, "avg_launch_us": upd_avg_ms * 1e3, "launches": upd_n,
                "algorithmic_bytes_per_launch": upd_alg_bytes,
                "traffic_over_algorithmic": (tr / upd_alg_bytes) if tr else None,
                "traffic_method": (traffic or {}).get("method") if tr else (traffic or {}).get("error"),
                "counter_factors": [(traffic or {}).get("fetch_factor"), (traffic or {}).get("write_factor")]}
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
        "roofline": roofline,
        "stages": table["stages"],
        "whole_call_frac": table["whole_call_frac"],
    }
    if not args.no_cpu_baseline:
        log("bench: timing the CPU oracle on a sample")
        result["cpu_baseline"] = cpu_baseline(case, args.cpu_seconds)
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
