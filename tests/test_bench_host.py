"""Host-side checks of bench.py's roofline bookkeeping (no GPU): the
algorithmic work it prices each stage with, against the counts of the
Newton-Schulz chain (Sec. 2.1 iteration X <- a X + (b A + c A^2) X with
A = X X^T on the short side, symmetric products counted once)."""
import bench


def test_chain_work_per_step_768x3072():
    s, l, steps = 768, 3072, 5
    w = bench.stage_work(s, l, k=8, rp=16, power_iters=1, steps=steps)
    chain = ("ns_gram", "ns_poly", "ns_update")
    flops = sum(w[n][0] for n in chain) / steps
    nbytes = sum(w[n][1] for n in chain) / steps
    # s(s+1)(l+s) + 2 s^2 l flops per matrix and step: 5.892 GFLOP
    assert flops == s * (s + 1) * (l + s) + 2 * s * s * l
    assert abs(flops / 1e9 - 5.892) < 5e-4
    # X read twice and written once (bf16), A written and read (fp32),
    # B written and read (bf16): 21.23 MB per matrix and step
    assert nbytes == 3 * 2 * s * l + 2 * 4 * s * s + 2 * 2 * s * s
    assert abs(nbytes / 1e6 - 21.234) < 1e-3


def test_stage_table_takes_the_larger_bound():
    # a stage with 1 GFLOP and 1 GB in 1 ms: the HBM time (0.125 ms at 8 TB/s)
    # exceeds the MFMA time (0.0004 ms at 2.5 PFLOP/s)
    t = bench.stage_table({"x": (2.0, 4)}, {"x": (1e9 / 8, 1e9 / 8)}, batch=8, calls=2, call_ms=1.0)
    row = t["stages"]["x"]
    assert row["bound"] == "hbm"
    assert abs(row["frac"] - 0.125) < 1e-12
    assert abs(t["whole_call_frac"] - 0.125) < 1e-12
