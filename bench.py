#!/usr/bin/env python3
"""Throughput of the ECASQ hot path on one MI355X.

One step = the whole path on one synthetic vector already resident in HBM:
sort + histogram + exact prefix sums, the lambda search (one full dp_APX solve
per query), codebook recovery, three-colour refinement (5 rounds at most) and
the final Philox stochastic rounding with its empirical entropy.  By default
the library's own defaults run: DP schedule 1 (the column-block sweep, every
layer updated from each cell, codebook from the argmin traceback) with the
sequential chord search; --dp-schedule 0 runs the layer-by-layer O(d) path
with the search in passes of 8 multipliers and Hirschberg recovery.

Default workload (weights_256k): fp32, d = 2^18, 0.9 Normal(0, 0.01) +
0.1 Laplace(0, 0.1), s = 32, budget 2.0 bits/entry, seed 0.

Printed (one JSON line): DP cell-updates/s counted as s*d^2/2 per DP solve
(the nominal unit; one solve per multiplier), the roofline of the dominant DP
kernel measured with HIP events on its own stream, and the CPU oracle timed
on a bounded sample.

    python bench.py [--steps K] [--warmup W] [--workload NAME]
"""
import argparse
import json
import os
import sys
import time

# Algorithmic fp64 operations per DP cell in the canonical cell arithmetic.
# The DP is a min-plus recurrence bound by FP64 VALU issue, and its
# operations are not all flops (the min, the max of h, the compare), so the
# roofline counts algorithmic FP64 lane operations (add, mul, fma, min, max,
# compare, a division and a log2 each count 1) against the chip's FP64 lane
# issue rate: 256 CUs x 64 FP64 lanes x 2.4 GHz = 39.32 Tops/s (the rate at
# which the 78.6 TFLOP/s FMA peak is reached, an FMA counting 2 flops there).
# Per (k, j) pair, shared by every layer and multiplier (18): 4 range
# differences, tu, td, 2 for C, w*d, the division, yu, yd, 2 max, 2 log2,
# the mul and fma of Phi.  Per multiplier: the cost Q = fma(-lambda', P, C)
# (1); per (k, j, layer) cell: F_prev + Q and the min (2).
OPS_PAIR = 18
OPS_Q = 1
OPS_CELL = 2
LAMBDAS_PER_PASS = 8
ALU_PEAK_TOPS = 256 * 64 * 2.4e9 / 1e12
FP64_VECTOR_PEAK_TFLOPS = 78.6

# The roofline fraction proper: algorithmic FP64 flops per second against the
# published FP64 vector peak (256 CUs x 2.4 GHz x 128 flops per clock per CU).
# Flops per cell of the method: 23 with an FMA counting 2 (4 range
# differences, v_a + v_b, the Phi sum, the candidate's add; v_a v_b, g, u,
# w d and the two products of h; the FMAs of C (2), t_u, t_d and
# + lambda' Phi), plus the division and the two log2 at 1 flop each: 26.  The
# sweep forms everything but the candidate's add once per (k, j) pair and
# adds it once per (k, j, layer) cell: 25 per pair + 1 per cell (min and max
# count 0); a layer-2 column (its first interval's C and Phi) counts 25.
FLOPS_PAIR = 25
FLOPS_CELL = 1
FLOPS_LAYER2_COL = 25
# the + lambda' Phi FMA inside FLOPS_PAIR: the layer kernel forms it once per
# multiplier, so a (k, j) cell of its launch over nlam multipliers counts
# FLOPS_PAIR - FLOPS_Q + (FLOPS_Q + FLOPS_CELL) nlam (47 for 8)
FLOPS_Q = 2


def layer_flops_per_cell(nlam):
    """Algorithmic FP64 flops of one (k, j) cell of the layer kernel with
    nlam multipliers per launch."""
    return FLOPS_PAIR - FLOPS_Q + (FLOPS_Q + FLOPS_CELL) * nlam


def flops_per_cell(nlam):
    """Algorithmic ops of one (k, j) cell of the layer kernel with nlam
    multipliers per launch."""
    return OPS_PAIR + (OPS_Q + OPS_CELL) * nlam


# HBM bytes per launch of the pass kernel (k_dp_layer, 8 multipliers) from
# rocprofv3 FETCH_SIZE / WRITE_SIZE runs of this bench on weights_256k
# (profiles/k_dp_layer_pass8_weights_256k.md), scaled by a plain copy's
# readings (FETCH x2.0, WRITE x1.0).  Valid only for the kernel sources they
# were taken on: reported as null once those sources change.
TRAFFIC_BYTES_PER_LAUNCH = 2.489e9
TRAFFIC_SOURCES_SHA = "4d97e06384505869"
KERNEL_SOURCES = ("dp.hip", "device.hpp", "launch.hpp", "log2_table.inc")
# the same, averaged over the k_sweep_step launches of the default workload
# (profiles/k_sweep_step_weights_256k.md)
SWEEP_TRAFFIC_BYTES_PER_LAUNCH = 1.412e8
SWEEP_TRAFFIC_SHA = "cf524e0f9632736c"
# hardware counters of the same profile: SQ_INSTS_VALU_FLOPS_FP64 per solve over
# the seconds per solve, and the share of VALU issue slots used
SWEEP_COUNTER_FP64_TFLOPS = 22.7
SWEEP_COUNTER_VALU_BUSY = 0.759
# VALU wave instructions per solve of the same profile (SQ_INSTS_VALU): at
# one instruction per SIMD every 4 cycles they bound the solve from below,
# and with it the flop fraction this instruction stream can reach
SWEEP_COUNTER_VALU_INSTS_PER_SOLVE = 5.982e10
SWEEP_SOURCES = ("sweep.hip", "device.hpp", "launch.hpp", "log2_table.inc")
# the (workload, s) both traffic figures were measured on; null for others
TRAFFIC_WORKLOAD = ("weights_256k", 32)


def kernel_sources_sha(files=None):
    import hashlib
    h = hashlib.sha256()
    here = os.path.join(os.path.dirname(os.path.abspath(__file__)), "paper_2608_18147_amd", "csrc")
    for f in files or KERNEL_SOURCES:
        with open(os.path.join(here, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def log(*a):
    print(*a, file=sys.stderr, flush=True)


# diagonal blocks k_sweep_step makes final per launch (the last launch: the rest)
SWEEP_STEP_BLOCKS = 16


def sweep_launches(p, s):
    """k_sweep_step launches of one sweep solve (the library's step schedule:
    blocks of 64 columns, SWEEP_STEP_BLOCKS per launch)."""
    nblk = (p + 63) // 64
    return (nblk + SWEEP_STEP_BLOCKS - 1) // SWEEP_STEP_BLOCKS


def sweep_issue_bound_frac(flops):
    """The flop fraction at which the profiled instruction stream would run
    with every SIMD issuing a VALU instruction every 4 cycles (1024 SIMDs x
    2.4 GHz): the ceiling of `frac` for this kernel's instruction mix."""
    t_min = SWEEP_COUNTER_VALU_INSTS_PER_SOLVE * 4.0 / (1024 * 2.4e9)
    return flops / t_min / 1e12 / FP64_VECTOR_PEAK_TFLOPS


def sweep_roofline(p, s, ms, solves, cells, measured=True):
    """Roofline of DP schedule 1: all k_sweep_step launches of one solve timed
    as one unit.  achieved = algorithmic FP64 flops per solve (FLOPS_PAIR per
    (k, j) pair, FLOPS_CELL per (k, j, layer) cell of layers 3..I,
    FLOPS_LAYER2_COL per layer-2 column) / seconds per solve, against the
    78.6 TFLOP/s FP64 vector peak.  Also reported, under their own names: the
    algorithmic FP64 lane operations per second against the lane issue rate
    (19 per pair with the cost Q, 2 per cell, 20 per layer-2 column; every
    add, mul, fma, min, max, division and log2 counting 1), and the
    hardware-counted FP64 rate and VALU busy share of the committed profile
    (for the kernel sources it was taken on)."""
    I = min(s, p)
    pairs = p * (p - 1) / 2.0
    layer_cells = sum((p - i + 1) * (p - i + 2) / 2.0 for i in range(3, I + 1))
    flops = FLOPS_PAIR * pairs + FLOPS_CELL * layer_cells + FLOPS_LAYER2_COL * (p - 1)
    ops = (OPS_PAIR + OPS_Q) * pairs + OPS_CELL * layer_cells + 20.0 * (p - 1)
    per_ms = ms / max(solves, 1)
    achieved = flops / (per_ms * 1e-3) / 1e12 if ms > 0 else 0.0
    lane = ops / (per_ms * 1e-3) / 1e12 if ms > 0 else 0.0
    steps = sweep_launches(p, s)
    current = measured and kernel_sources_sha(SWEEP_SOURCES) == SWEEP_TRAFFIC_SHA
    return {
        "bound": "alu",
        "kernel": "k_sweep_step (fp64 VALU); one DP solve = %d launches" % steps,
        "achieved": achieved,
        "peak": FP64_VECTOR_PEAK_TFLOPS,
        "unit": "TFLOP/s",
        "frac": achieved / FP64_VECTOR_PEAK_TFLOPS,
        "traffic": SWEEP_TRAFFIC_BYTES_PER_LAUNCH if current else None,
        "traffic_unit": "bytes/launch",
        "flops_per_solve": flops,
        "flops_accounting": ("%d per (k, j) pair + %d per (k, j, layer) cell + %d per layer-2 "
                             "column; FMA = 2, division and log2 = 1 each, min/max = 0"
                             % (FLOPS_PAIR, FLOPS_CELL, FLOPS_LAYER2_COL)),
        "lane_ops": {"achieved_tops": lane, "peak_tops": ALU_PEAK_TOPS,
                     "frac": lane / ALU_PEAK_TOPS, "ops_per_solve": ops},
        "counters": ({"fp64_tflops": SWEEP_COUNTER_FP64_TFLOPS,
                      "frac_of_fp64_peak": SWEEP_COUNTER_FP64_TFLOPS / FP64_VECTOR_PEAK_TFLOPS,
                      "valu_busy": SWEEP_COUNTER_VALU_BUSY,
                      "frac_at_full_valu_issue": sweep_issue_bound_frac(flops)}
                     if current else None),
        "avg_launch_ms": per_ms / steps,
        "launches": solves * steps,
        "ms_per_solve": per_ms,
        "solves": solves,
        "cells_per_s": cells / (ms * 1e-3) if ms > 0 else None,
    }


def _omp():
    """The OpenMP runtime the oracle library uses (to set its thread count)."""
    import ctypes
    import ctypes.util
    name = ctypes.util.find_library("gomp") or "libgomp.so.1"
    return ctypes.CDLL(name)


def cpu_baseline(x, s, lam, sample_d, sample_d1=None):
    """The oracle's forward DP on the sample_d smallest entries of the same
    input (exact cell arithmetic, OpenMP over columns) with all threads, and
    on the sample_d1 smallest with one thread."""
    import numpy as np

    from oracle import pipeline

    omp = _omp()
    threads = int(omp.omp_get_max_threads())

    def run(n):
        H = pipeline.prepare(np.sort(x)[:n])
        t0 = time.perf_counter()
        r = pipeline.dp_forward(H, s, lam * H.s2tot)
        return r, time.perf_counter() - t0

    r, dt = run(sample_d)
    nominal = s * sample_d * sample_d / 2.0
    out = {
        "value": nominal / dt,
        "unit": "cell-updates/s",
        "cores": threads,
        "kind": "oracle",
        "sample": (f"one forward dp_APX solve (s={s}, lambda={lam}) on the {sample_d} smallest "
                   f"entries of the same input: {r['cells']} cells evaluated in {dt:.2f} s "
                   f"on {threads} threads; value counts s*d^2/2 with d={sample_d}"),
        "exact_cells_per_s": r["cells"] / dt,
    }
    n1 = sample_d1 or max(1024, sample_d // 4)
    omp.omp_set_num_threads(1)
    try:
        r1, dt1 = run(n1)
    finally:
        omp.omp_set_num_threads(threads)
    out["one_thread"] = {
        "value": s * n1 * n1 / 2.0 / dt1, "unit": "cell-updates/s", "cores": 1,
        "exact_cells_per_s": r1["cells"] / dt1,
        "sample": (f"the same solve on the {n1} smallest entries, one thread: "
                   f"{r1['cells']} cells in {dt1:.2f} s"),
    }
    return out


def batched_rate(torch, ecasq, inputs, reps=10):
    """Solves/s of the batched path: 4096 KV-cache-like fp16 rows of d = 128,
    s = 16, budget 3.0 bits/entry, one solve per row (no refinement), all rows
    in one launch.  ms_per_launch is the kernel, from HIP events recorded
    around each launch; ms_per_call adds the binding's output tensors and the
    call's wait for the stream."""
    rows = inputs.make("kv_rows", seed=0)
    xd = torch.from_numpy(rows).to("cuda")
    opts = ecasq.ecasq_default_options(refine_rounds=0)
    ecasq.ecasq_solve_batched(xd, 16, 3.0, options=opts)  # warm-up
    torch.cuda.synchronize()
    ecasq.ecasq_timing_read(ecasq.TIMING_BATCHED, reset=True)
    ecasq.ecasq_timing_enable(True)
    try:
        t0 = time.perf_counter()
        for _ in range(reps):
            cbs, tt, infos = ecasq.ecasq_solve_batched(xd, 16, 3.0, options=opts)
        torch.cuda.synchronize()
        dt_call = (time.perf_counter() - t0) / reps
    finally:
        ecasq.ecasq_timing_enable(False)
    kms, kn, _ = ecasq.ecasq_timing_read(ecasq.TIMING_BATCHED, reset=True)
    dt = kms / kn / 1e3  # the kernel, from HIP events around each launch
    inf = ecasq.infos_to_dicts(infos)
    cells = sum(i["cells"] for i in inf)
    solves = sum(i["dp_solves"] for i in inf)
    n, d = rows.shape
    log(f"batched: {dt * 1e3:.2f} ms per {n}-row launch ({dt_call * 1e3:.2f} ms per call)")
    return {
        "workload": "kv_rows", "rows": n, "d": d, "s": 16, "budget_bits": 3.0,
        "refine_rounds": 0, "ms_per_launch": dt * 1e3, "ms_per_call": dt_call * 1e3,
        "launches_timed": kn, "solves_per_s": n / dt,
        "dp_solves_per_row": solves / n, "cells_per_s": cells / dt,
        "nominal_cell_updates_per_s": solves * 16 * d * d / 2.0 / dt,
    }


def alphabet_rate(torch, ecasq, xd, s, b, opts, full_info, grids=(("uniform", 4096),
                                                                   ("quantile", 4096))):
    """The same solve on permissible grids of m points (App. D with P != X):
    time per solve step and the objective against the solve over all distinct
    values (full_info)."""
    res = []
    for kind, m in grids:
        o = ecasq.ecasq_options()
        ctypes_copy = {f: getattr(opts, f) for f, _ in opts._fields_}
        for f, v in ctypes_copy.items():
            setattr(o, f, v)
        o.alphabet = 1 if kind == "uniform" else 2
        o.alphabet_size = m
        ecasq.ecasq_solve(xd, s, b, options=o)  # warm-up
        torch.cuda.synchronize()
        reps = 3
        t0 = time.perf_counter()
        for _ in range(reps):
            cb, rk, info = ecasq.ecasq_solve(xd, s, b, options=o)
        torch.cuda.synchronize()
        ms = (time.perf_counter() - t0) / reps * 1e3
        res.append({"grid": kind, "m": m, "p": info["p"], "ms_per_solve_step": ms,
                    "dp_solves": info["dp_solves"], "t": info["t"], "vnmse": info["vnmse"],
                    "entropy": info["entropy"], "objective": info["objective"],
                    "vnmse_vs_all_values": info["vnmse"] / full_info["vnmse"]})
    return res


# y = yu + yd, max, log2, the mul m log2(m), the candidate's fma, the min
OPT_OPS_PER_CANDIDATE = 6
# the same as flops: the add, the log2 (1), the mul, the fma (2); max and min 0
OPT_FLOPS_PER_CANDIDATE = 5


def optimal_rate(torch, ecasq, inputs, reps=3):
    """Optimal lambda-ECASQ (Sec. 4) on the weight-like 2^18 vector in bf16
    (a few thousand permissible values), s = 64, lambda = 0.1: time per solve
    with the monotone-bracket scan and with the full scan, and the full scan's
    layer kernel against the FP64 vector peak."""
    x = torch.from_numpy(inputs.make("weights_256k", seed=0)).to(torch.bfloat16).to("cuda")
    s, lam = 64, 0.1
    out = {"workload": "weights_256k as bf16", "s": s, "lambda": lam}
    for name, scan in (("monotone", 0), ("full", 1)):
        o = ecasq.ecasq_default_options(optimal_scan=scan)
        ecasq.ecasq_solve_optimal(x, s, lam, options=o)  # warm-up
        torch.cuda.synchronize()
        ecasq.ecasq_timing_enable(True)
        ecasq.ecasq_timing_read(ecasq.TIMING_OPT, reset=True)
        t0 = time.perf_counter()
        for _ in range(reps):
            cb, rk, info = ecasq.ecasq_solve_optimal(x, s, lam, options=o)
        torch.cuda.synchronize()
        ms = (time.perf_counter() - t0) / reps * 1e3
        kms, launches, cands = ecasq.ecasq_timing_read(ecasq.TIMING_OPT)
        ecasq.ecasq_timing_enable(False)
        r = {"ms_per_solve": ms, "p": info["p"], "t": info["t"], "objective": info["objective"],
             "vnmse": info["vnmse"], "entropy": info["entropy"],
             "layer_ms_per_solve": kms / reps, "layer_launches": launches // reps}
        if scan == 1 and kms > 0:
            rate = cands / (kms * 1e-3)
            achieved = OPT_FLOPS_PER_CANDIDATE * rate / 1e12
            tops = OPT_OPS_PER_CANDIDATE * rate / 1e12
            r["roofline"] = {"bound": "alu", "kernel": "k_opt_layer<full> (fp64 VALU)",
                             "achieved": achieved, "peak": FP64_VECTOR_PEAK_TFLOPS,
                             "unit": "TFLOP/s", "frac": achieved / FP64_VECTOR_PEAK_TFLOPS,
                             "flops_per_candidate": OPT_FLOPS_PER_CANDIDATE,
                             "lane_ops": {"achieved_tops": tops, "peak_tops": ALU_PEAK_TOPS,
                                          "frac": tops / ALU_PEAK_TOPS,
                                          "ops_per_candidate": OPT_OPS_PER_CANDIDATE},
                             "candidates_per_s": rate,
                             "avg_launch_ms": kms / max(launches, 1)}
        out[name] = r
    out["speedup_monotone"] = out["full"]["ms_per_solve"] / out["monotone"]["ms_per_solve"]
    return out


# the paper's mean runtimes at its runtime setting (its CPU implementation,
# BF16 inputs, d = 2^18, s = 64, lambda = 0.1): context, not a target
PAPER_RUNTIME_S = {"approx": 0.26, "refined": 0.33, "optimal": 6.39}


def paper_setting_rate(torch, ecasq, inputs, seeds=5):
    """The paper's runtime setting: d = 2^18 vectors of its four synthetic
    distributions (Normal, Lognormal, Student-t, sparse outliers) cast to
    bf16, s = 64, lambda = 0.1, five seeds each.  Time of one whole solve
    (sort, histogram, DP, recovery, metrics), without refinement, with five
    refinement rounds, and of the optimal DP (monotone brackets); like the
    paper, the mean of the four distributions' means."""
    d, s, lam = 1 << 18, 64, 0.1
    gens = (("normal", inputs.normal), ("lognormal", inputs.lognormal_signed),
            ("student_t", inputs.student_t), ("sparse_outlier", inputs.sparse_outlier))
    opts = {"approx": ecasq.ecasq_default_options(refine_rounds=0),
            "refined": ecasq.ecasq_default_options(refine_rounds=5),
            "optimal": ecasq.ecasq_default_options()}
    per = {v: [] for v in opts}
    ps = []
    for _, gen in gens:
        ms = {v: [] for v in opts}
        for seed in range(seeds):
            x = torch.from_numpy(gen(d, seed)).to(torch.bfloat16).to("cuda")
            for v, o in opts.items():
                run = ((lambda: ecasq.ecasq_solve_optimal(x, s, lam, options=o)) if v == "optimal"
                       else (lambda: ecasq.ecasq_solve_lagrangian(x, s, lam, options=o)))
                run()  # warm-up
                torch.cuda.synchronize()
                t0 = time.perf_counter()
                info = run()[2]
                torch.cuda.synchronize()
                ms[v].append((time.perf_counter() - t0) * 1e3)
            ps.append(info["p"])
        for v in opts:
            per[v].append(sum(ms[v]) / len(ms[v]))
    out = {"workload": "normal, lognormal, student_t, sparse_outlier; d = 2^18 as bf16",
           "s": s, "lambda": lam, "seeds": seeds, "p_range": [min(ps), max(ps)]}
    for v in opts:
        mean = sum(per[v]) / len(per[v])
        out[v] = {"ms_per_solve": mean, "per_distribution_ms": per[v],
                  "paper_cpu_s_other_machine": PAPER_RUNTIME_S[v]}
    return out


def rounding_rate(torch, ecasq, d=1 << 26, t=32, reps=5):
    """The final stochastic rounding (k_quantize: 4 B in, 1 B out per entry)
    and its time-shared form (k_quantize_ts: 4 B in, 1 + 1 B out) on 2^26
    standard normal fp32 entries with t = 32 evenly spaced values over
    [min, max] (alpha = 0.4 and a second codebook of 31 for the time-shared
    form), timed with HIP events on the stream the library launches on,
    against the 8 TB/s HBM peak."""
    g = torch.Generator(device="cuda")
    g.manual_seed(0)
    x = torch.randn(d, generator=g, device="cuda", dtype=torch.float32)
    lo, hi = float(x.min()), float(x.max())
    c0 = torch.linspace(lo, hi, t, dtype=torch.float64, device="cuda")
    c1 = torch.linspace(lo, hi, t - 1, dtype=torch.float64, device="cuda")
    out = {"d": d, "t": t}
    for name, run, per in (
            ("quantize", lambda: ecasq.ecasq_quantize(x, c0, 7), 5),
            ("quantize_timeshare", lambda: ecasq.ecasq_quantize_timeshare(x, c0, c1, 0.4, 7), 6)):
        run()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            run()
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / reps
        gbs = per * d / (ms * 1e-3) / 1e9
        out[name] = {"ms": ms, "bytes_per_entry": per, "achieved_GBs": gbs, "frac_of_8TBs": gbs / 8000.0,
                     "bound": "valu (Philox4x32-10's 32x32->64 products at a quarter of the issue rate)"}
    return out


def coding_rate(torch, ecasq, sym, t, info, reps=5):
    """rANS coding of the final symbols: coded bits per entry (payload,
    16-bit frequency descriptors, segment table, and a 16-bit value per
    codebook entry as App. F.1 charges) against H(Xhat) + 32 t / d, and the
    encode / decode times."""
    d = sym.numel()
    data = ecasq.ecasq_encode(sym, t)
    back = ecasq.ecasq_decode(data, d, t)
    assert torch.equal(back, sym)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(reps):
        data = ecasq.ecasq_encode(sym, t)
    torch.cuda.synchronize()
    enc_ms = (time.perf_counter() - t0) / reps * 1e3
    t0 = time.perf_counter()
    for _ in range(reps):
        back = ecasq.ecasq_decode(data, d, t)
    torch.cuda.synchronize()
    dec_ms = (time.perf_counter() - t0) / reps * 1e3
    return {"t": t, "d": d, "stream_bytes": int(data.numel()),
            "coded_bits_per_entry": (8.0 * data.numel() + 16.0 * t) / d,
            "ideal_rate_total": info["rate_total"], "entropy": info["entropy"],
            "encode_ms": enc_ms, "decode_ms": dec_ms}


def refined_search_rate(torch, ecasq, xd, s, b):
    """The refinement-aware search (dp_objective 2) on the same input and
    budget: time per solve step and the codebook's quality."""
    o = ecasq.ecasq_default_options(dp_objective=2)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    cb, rk, info = ecasq.ecasq_solve(xd, s, b, options=o)
    torch.cuda.synchronize()
    return {"ms_per_solve_step": (time.perf_counter() - t0) * 1e3, "dp_solves": info["dp_solves"],
            "t": info["t"], "vnmse": info["vnmse"], "entropy": info["entropy"],
            "entropy_surrogate": info["entropy_surrogate"], "objective": info["objective"]}


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawTextHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=2)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="weights_256k")
    ap.add_argument("--budget", type=float, default=None,
                    help="one budget (default: the workload's first; with --all-budgets\n"
                         "every budget of the workload is solved per step with shared solves)")
    ap.add_argument("--all-budgets", action="store_true")
    ap.add_argument("--progress", action="store_true",
                    help="print a line per DP solve (stderr)")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--cpu-sample", type=int, default=32768)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-batched", action="store_true")
    ap.add_argument("--no-optimal", action="store_true",
                    help="skip the optimal-DP solves (bf16 weights, s = 64, lambda = 0.1)")
    ap.add_argument("--optimal-only", action="store_true",
                    help="only run the optimal-DP measurement and print it")
    ap.add_argument("--rounding-only", action="store_true",
                    help="only run the final-rounding measurement (2^26 fp32 entries, t = 32)\n"
                         "and print it")
    ap.add_argument("--batched-only", action="store_true",
                    help="only run the batched-rows measurement (4096 fp16 rows of 128) and\n"
                         "print it")
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the side measurements (grids, optimal DP, refinement-aware\n"
                         "search, entropy coding, batched rows, the paper's runtime setting,\n"
                         "the stochastic rounding at 2^26 entries)")
    ap.add_argument("--no-alphabet", action="store_true",
                    help="skip the permissible-grid solves (uniform / quantile, 4096 points)")
    ap.add_argument("--dp-schedule", type=int, default=None, choices=(0, 1),
                    help="0: layer by layer (passes of 8, Hirschberg); 1: column-block sweep\n"
                         "(default: the library's defaults)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run one plain device copy of 2^28 bytes (the reference kernel\n"
                         "that scales rocprofv3 FETCH_SIZE / WRITE_SIZE readings) and exit")
    args = ap.parse_args()

    if args.copy_calibration:
        import torch
        n = 1 << 28
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        torch.cuda.synchronize()
        dst = src.clone()
        torch.cuda.synchronize()
        log(f"copied {dst.numel()} bytes")
        return

    if args.gpus != 1:
        print("bench.py measures one GPU only: the single-vector path runs on one GPU and "
              "is not sharded across GPUs", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2608_18147_amd import ecasq, inputs

    if args.optimal_only:
        print(json.dumps(optimal_rate(torch, ecasq, inputs)), flush=True)
        return
    if args.batched_only:
        print(json.dumps(batched_rate(torch, ecasq, inputs)), flush=True)
        return
    if args.rounding_only:
        print(json.dumps(rounding_rate(torch, ecasq)), flush=True)
        return

    w = inputs.WORKLOADS[args.workload]
    if "rows" in w:
        raise SystemExit("use a single-vector workload")
    d, s = w["d"], w["s"]
    b = args.budget if args.budget is not None else w["budgets"][0]
    x = inputs.make(args.workload, seed=args.seed)
    xd = torch.from_numpy(x).to("cuda")
    torch.cuda.synchronize()

    if args.dp_schedule == 0:
        opts = ecasq.ecasq_default_options(dp_schedule=0, search_width=8)
    elif args.dp_schedule == 1:
        opts = ecasq.ecasq_default_options(dp_schedule=1, search_width=1)
    else:
        opts = ecasq.ecasq_default_options()
    sweep = opts.dp_schedule == 1

    budgets = list(w["budgets"]) if args.all_budgets else [b]

    last = {}

    def step():
        if len(budgets) == 1:
            cb, rk, info = ecasq.ecasq_solve(xd, s, b, options=opts)
            sym, ent, hist = ecasq.ecasq_quantize(xd, cb, args.seed)
            last["sym"], last["t"] = sym, info["t"]
            return info, ent
        res = ecasq.ecasq_solve_budgets(xd, s, budgets, options=opts)
        agg = dict(res[-1][2])
        agg["dp_solves"] = sum(r[2]["dp_solves"] for r in res)
        agg["cells"] = sum(r[2]["cells"] for r in res)
        agg["search_passes"] = sum(r[2]["search_passes"] for r in res)
        agg["per_budget"] = []
        for bb, (cb, rk, info) in zip(budgets, res):
            sym, ent, hist = ecasq.ecasq_quantize(xd, cb, args.seed)
            agg["per_budget"].append({"budget": bb, "t": info["t"], "vnmse": info["vnmse"],
                                      "entropy": info["entropy"], "dp_solves": info["dp_solves"],
                                      "empirical_entropy": float(ent)})
        return agg, ent

    # long steps (the 2^20 budget sweep) print a line per DP solve
    ecasq.ecasq_timing_enable(args.progress, verbose=args.progress)
    for i in range(args.warmup):
        t0 = time.perf_counter()
        info, ent = step()
        torch.cuda.synchronize()
        log(f"warmup {i + 1}/{args.warmup}: {time.perf_counter() - t0:.2f} s, "
            f"{info['dp_solves']} DP solves, t={info['t']}")

    ecasq.ecasq_timing_enable(True, verbose=args.progress)
    for v in (ecasq.TIMING_SINGLE, ecasq.TIMING_PASS, ecasq.TIMING_SWEEP):
        ecasq.ecasq_timing_read(v, reset=True)
    infos = []
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for i in range(args.steps):
        t0 = time.perf_counter()
        info, ent = step()
        infos.append((info, ent))
        log(f"step {i + 1}/{args.steps}: {time.perf_counter() - t0:.2f} s")
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start
    ms, launches, cells = ecasq.ecasq_timing_read(ecasq.TIMING_PASS)
    ms1, launches1, cells1 = ecasq.ecasq_timing_read(ecasq.TIMING_SINGLE)
    msw, nsw, cellsw = ecasq.ecasq_timing_read(ecasq.TIMING_SWEEP)
    ecasq.ecasq_timing_enable(False)

    nominal = sum(inf["dp_solves"] * s * d * d / 2.0 for inf, _ in infos)
    exact = sum(inf["cells"] for inf, _ in infos)
    value = nominal / elapsed
    info, ent = infos[-1]
    p = info["p"]
    measured = (args.workload, s) == TRAFFIC_WORKLOAD
    if sweep:
        roofline = sweep_roofline(p, s, msw, nsw, cellsw, measured)
    else:
        avg_ms = ms / max(launches, 1)
        fpc = flops_per_cell(LAMBDAS_PER_PASS)
        flc = layer_flops_per_cell(LAMBDAS_PER_PASS)
        rate = (cells / max(launches, 1)) / (avg_ms * 1e-3) if ms > 0 else 0.0
        achieved = flc * rate / 1e12
        tops = fpc * rate / 1e12
        roofline = {
            "bound": "alu",
            "kernel": "k_dp_layer, 8 multipliers per launch (fp64 VALU)",
            "achieved": achieved,
            "peak": FP64_VECTOR_PEAK_TFLOPS,
            "unit": "TFLOP/s",
            "frac": achieved / FP64_VECTOR_PEAK_TFLOPS,
            "traffic": (TRAFFIC_BYTES_PER_LAUNCH
                        if measured and kernel_sources_sha() == TRAFFIC_SOURCES_SHA else None),
            "traffic_unit": "bytes/launch",
            "flops_per_cell": flc,
            "flops_accounting": ("per (k, j) cell of a launch: %d for C and Phi, then %d per "
                                 "multiplier (the + lambda' Phi FMA and the candidate's add); "
                                 "FMA = 2, division and log2 = 1 each, min/max/compare = 0"
                                 % (FLOPS_PAIR - FLOPS_Q, FLOPS_Q + FLOPS_CELL)),
            "lane_ops": {"achieved_tops": tops, "peak_tops": ALU_PEAK_TOPS,
                         "frac": tops / ALU_PEAK_TOPS, "ops_per_cell": fpc},
            "avg_launch_ms": avg_ms,
            "launches": launches,
            "cells_per_s": cells / (ms * 1e-3) if ms > 0 else None,
            "lambda_cells_per_s": LAMBDAS_PER_PASS * cells / (ms * 1e-3) if ms > 0 else None,
        }
    out = {
        "metric": "DP cell-updates/s (s*d^2/2 per solve)",
        "value": value,
        "unit": "cell-updates/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": elapsed / args.steps * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64",
        "data": "synthetic",
        "config": {
            "workload": args.workload, "d": d, "s": s,
            "budget_bits": budgets if len(budgets) > 1 else b, "seed": args.seed,
            "refine_rounds": 5, "input_dtype": "f32", "dp_schedule": opts.dp_schedule,
            "search_width": opts.search_width,
            "recovery": "argmin traceback" if sweep else "hirschberg",
        },
        "roofline": roofline,
        "single_multiplier_layers": {
            "launches": launches1, "ms": ms1,
            "cells_per_s": cells1 / (ms1 * 1e-3) if ms1 > 0 else None,
            "achieved_tops": (flops_per_cell(1) * cells1 / (ms1 * 1e-3) / 1e12
                                if ms1 > 0 else None),
        },
        "exact_cells_per_s": exact / elapsed,
        "dp_solves_per_step": info["dp_solves"],
        **({"per_budget": info["per_budget"]} if "per_budget" in info else {}),
        "search_passes_per_step": info["search_passes"],
        "solution": {
            "t": info["t"], "p": info["p"], "lambda": info["lambda"], "vnmse": info["vnmse"],
            "entropy": info["entropy"], "entropy_surrogate": info["entropy_surrogate"],
            "empirical_entropy": float(ent), "refine_rounds_run": info["refine_rounds_run"],
        },
    }
    if args.no_extras:
        args.no_alphabet = args.no_optimal = args.no_batched = True
    if not args.no_extras and len(budgets) == 1:
        out["entropy_coding"] = coding_rate(torch, ecasq, last["sym"], last["t"], info)
        r = refined_search_rate(torch, ecasq, xd, s, b)
        r["vnmse_vs_default"] = r["vnmse"] / info["vnmse"]
        out["refined_search"] = r
    if not args.no_alphabet and len(budgets) == 1:
        out["alphabet"] = alphabet_rate(torch, ecasq, xd, s, b, opts, info)
        for r in out["alphabet"]:
            r["speedup"] = out["ms_per_step"] / r["ms_per_solve_step"]
    if not args.no_optimal:
        out["optimal"] = optimal_rate(torch, ecasq, inputs)
    if not args.no_extras:
        out["paper_setting"] = paper_setting_rate(torch, ecasq, inputs)
        out["rounding"] = rounding_rate(torch, ecasq)
    if not args.no_batched:
        out["batched"] = batched_rate(torch, ecasq, inputs)
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle) ...")
        out["cpu_baseline"] = cpu_baseline(x, s, 0.1, args.cpu_sample)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
