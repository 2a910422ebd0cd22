#!/usr/bin/env python3
"""Benchmark of MKOR's per-step hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config 3]

A step is one full pass of the hot path (stabiliser + SM update of both
factors of every layer, preconditioning, rescale) over the whole grouped layer
list, launched through the C ABI (mkor_step).  The default workload is the
BERT-Large-shaped set: 24 blocks x {4 x 1024x1024, 1024x4096, 4096x1024},
fp32 factors, bf16 gradients, preconditioned on the layers' default GEMM path
(the exact three-way bf16 split on the bf16 matrix cores for these shapes;
the fp32 MFMA path is measured beside it, "fp32_mfma_path").  Inputs are
synthetic, seeded, and resident in HBM before the timed region starts.

Prints one JSON line: layer-updates/s, per-kernel times measured with HIP
events on the launch stream, the roofline of the dominant kernel, and the
float64 CPU oracle timed on a bounded sample of the same workload.  The same
workload with half-precision (bf16) factors is measured beside it
("half_factors"; skip with --no-half, or time it as the main line with
--factor-dtype bf16).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import statistics
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "layer-updates/sec (SM update + precondition), BERT-Large set; % HBM / % MFMA peak"
HBM_PEAK_GBS = 8000.0       # MI355X HBM3E
FP32_MFMA_PEAK_TF = 157.3   # MI355X dense fp32 matrix
BF16_MFMA_PEAK_TF = 2500.0  # MI355X dense bf16 matrix


REPEATS = 5                 # timed windows per measurement; the median is reported


def timed_windows(run, stream, steps, repeats):
    """ms per step of `repeats` windows of `steps` calls of run(), each window
    bracketed by HIP events on `stream` with the device idle before it."""
    import torch
    out = []
    for _ in range(repeats):
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(steps):
            run()
        e1.record(stream)
        torch.cuda.synchronize()
        out.append(e0.elapsed_time(e1) / steps)
    return out


PROFILE_TRAFFIC = {False: os.path.join(ROOT, "profiles", "traffic_bert_large_144.md"),
                   True: os.path.join(ROOT, "profiles", "traffic_bert_large_144_bf16.md")}


def library_source_sha256() -> str:
    """SHA-256 over the library sources (csrc/ and include/), path and bytes of
    each file in sorted order: identifies the kernels a profile was taken with."""
    h = hashlib.sha256()
    for sub in ("paper_2306_01685_amd/csrc", "include"):
        d = os.path.join(ROOT, sub)
        for f in sorted(os.listdir(d)):
            if f.endswith((".hip", ".cpp", ".h")):
                h.update(f"{sub}/{f}".encode())
                with open(os.path.join(d, f), "rb") as fh:
                    h.update(fh.read())
    return h.hexdigest()


def profiled_traffic(kernel: str, config: int, half: bool = False):
    """HBM bytes per launch of `kernel` from the committed rocprofv3 counter
    summary (FETCH_SIZE and WRITE_SIZE, copy-calibrated) of the fp32- or
    bf16-factor run, or None if there is no record for this workload or the
    library changed since it was taken."""
    path = PROFILE_TRAFFIC[half]
    if config != 3 or not os.path.exists(path):
        return None
    for line in open(path):
        if line.startswith("traffic-record:"):
            rec = json.loads(line.split(":", 1)[1])
            if rec.get("source_sha256") != library_source_sha256() or kernel not in rec["bytes"]:
                return None
            rd, wr = rec["bytes"][kernel]
            return dict(read_bytes=rd, write_bytes=wr, total_bytes=rd + wr,
                        source=os.path.relpath(path, ROOT))
    return None


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", type=int, default=3)
    ap.add_argument("--eps", type=float, default=100.0)
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-stage-timing", action="store_true")
    ap.add_argument("--rows", type=int, default=0,
                    help="form a and g inside each step from this many bf16 token rows per layer "
                         "(Algorithm 1's rank-1 means); 0 (default): a and g are given, as in the "
                         "headline metric")
    ap.add_argument("--no-schedule", action="store_true",
                    help="skip the update-every-10-steps measurement")
    ap.add_argument("--mode", choices=["step", "copy", "power"], default="step",
                    help="copy: time a plain device-to-device copy of --copy-mib MiB (the reference "
                         "kernel whose FETCH_SIZE / WRITE_SIZE counters calibrate the traffic figures); "
                         "power: run the step and single GEMM stages back to back, --power-seconds "
                         "each, while sampling board power and clocks with amd-smi")
    ap.add_argument("--power-seconds", type=float, default=6.0)
    ap.add_argument("--no-power", action="store_true",
                    help="skip the board power / clock sample taken while the dominant GEMM runs "
                         "(roofline.power)")
    ap.add_argument("--copy-mib", type=int, default=1024)
    ap.add_argument("--factor-dtype", choices=["fp32", "bf16"], default="fp32",
                    help="storage type of the inverse factors of the timed run (bf16: the "
                         "half-precision factors, bf16 MFMA preconditioning)")
    ap.add_argument("--rank", type=int, default=1,
                    help="vectors per factor update (the rank-r extension; fp32 factors)")
    ap.add_argument("--no-opt", action="store_true",
                    help="skip the measurement of the step with the fused LAMB optimizer")
    ap.add_argument("--no-half", action="store_true",
                    help="skip the extra measurement with bf16 factors")
    ap.add_argument("--gemm-path", choices=["auto", "fp32", "split"], default="auto",
                    help="preconditioning GEMMs of fp32 factors (auto: the split where the shape allows)")
    ap.add_argument("--no-fp32-path", action="store_true",
                    help="skip the extra measurement on the fp32 MFMA GEMM path")
    ap.add_argument("--no-stabilised", action="store_true",
                    help="skip the extra window with the stabiliser firing on every step (eps = 0)")
    ap.add_argument("--no-references", action="store_true",
                    help="skip the copy-kernel and torch.matmul reference measurements")
    ap.add_argument("--graph", action="store_true",
                    help="also time the step captured once in a HIP graph and replayed K times "
                         "(saves the launch gaps of launch-bound workloads)")
    return ap.parse_args()


def copy_measure(mib, steps, warmup):
    """A plain device-to-device copy of `mib` MiB (torch's copy kernel): the
    achievable-bandwidth reference for read + write traffic."""
    import torch
    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    stream = torch.cuda.current_stream()
    for _ in range(warmup):
        dst.copy_(src)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(steps):
        dst.copy_(src)
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    nbytes = 2 * n * 4
    del src, dst
    torch.cuda.empty_cache()
    return {"bytes_read": n * 4, "bytes_written": n * 4, "ms": ms,
            "gbs": nbytes / (ms / 1e3) / 1e9, "frac_hbm": nbytes / (ms / 1e3) / 1e9 / HBM_PEAK_GBS}


def copy_reference(args):
    """--mode copy: the copy kernel alone (its FETCH_SIZE / WRITE_SIZE
    counters calibrate the traffic figures)."""
    print(json.dumps({"mode": "copy", **copy_measure(args.copy_mib, args.steps, args.warmup)}), flush=True)


def torch_matmul_reference(w, reps=3):
    """torch.matmul in fp32 (the vendor GEMM library) on the workload's two
    preconditioning products per layer, Linv @ G then X @ Rinv, one pair per
    distinct shape timed and weighted by its count: an out-of-product
    reference for the preconditioning GEMMs."""
    import torch
    counts = {}
    for s in w.shapes:
        counts[s] = counts.get(s, 0) + 1
    stream = torch.cuda.current_stream()
    total_ms, flops = 0.0, 0
    for (d_in, d_out), c in counts.items():
        L = torch.randn(d_in, d_in, device="cuda")
        R = torch.randn(d_out, d_out, device="cuda")
        G = torch.randn(d_in, d_out, device="cuda")
        for _ in range(2):
            torch.matmul(torch.matmul(L, G), R)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            torch.matmul(torch.matmul(L, G), R)
        e1.record(stream)
        torch.cuda.synchronize()
        total_ms += c * e0.elapsed_time(e1) / reps
        flops += c * 2 * d_in * d_out * (d_in + d_out)
        del L, R, G
    torch.cuda.empty_cache()
    return {"ms": total_ms, "tflops": flops / (total_ms / 1e3) / 1e12,
            "frac_fp32_mfma_peak": flops / (total_ms / 1e3) / 1e12 / FP32_MFMA_PEAK_TF,
            "allow_tf32": bool(torch.backends.cuda.matmul.allow_tf32),
            "note": "torch.matmul fp32, Linv @ G @ Rinv per layer, shapes timed one pair at a time"}


def torch_matmul_bf16_reference(n=8192, settle_s=1.5, reps=200, sample_power=True, power_seconds=3.0):
    """torch.matmul in bf16 (the vendor GEMM library) on one n x n x n
    product, run back to back for settle_s before a timed window of reps so
    that the clock has settled under load as it has in the bench's windows:
    the bf16 matrix-core rate the library sustains on this part, a measured
    ceiling for GEMMs that feed the bf16 MFMAs."""
    import torch
    a = torch.randn(n, n, device="cuda", dtype=torch.bfloat16)
    b = torch.randn(n, n, device="cuda", dtype=torch.bfloat16)
    stream = torch.cuda.current_stream()
    torch.cuda.synchronize()
    t0 = time.time()
    while time.time() - t0 < settle_s:
        for _ in range(10):
            torch.matmul(a, b)
        torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        torch.matmul(a, b)
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    pw = clock_during(lambda: torch.matmul(a, b), power_seconds) if sample_power else None
    del a, b
    torch.cuda.empty_cache()
    return {"n": n, "ms": ms, "tflops": 2 * n ** 3 / (ms / 1e3) / 1e12,
            "frac_bf16_peak": 2 * n ** 3 / (ms / 1e3) / 1e12 / BF16_MFMA_PEAK_TF, "power": pw,
            "note": f"torch.matmul bf16, {n}^3, timed after {settle_s} s back to back"}


def workload_desc(w, factor_dtype="fp32"):
    counts = {}
    for s in w.block_shapes:
        counts[s] = counts.get(s, 0) + 1
    inner = ", ".join(f"{c}x {i}x{o}" if c > 1 else f"{i}x{o}" for (i, o), c in counts.items())
    return f"{w.name}: {w.blocks} x {{{inner}}}, {factor_dtype} factors, {w.grad_dtype} G"


def split_eligible(w, gemm_path):
    """True when every layer of the workload runs on the split GEMMs."""
    if gemm_path == "fp32":
        return False
    return all(i % 64 == 0 and o % 64 == 0 for i, o in w.shapes)


def fill_rows(layers, seed=2307):
    """Seeded bf16 token rows on the GPU: activations N(0, 1), output gradients
    N(0, 1e-6), the distributions of the workload's rows."""
    import torch
    gen = torch.Generator(device="cuda")
    gen.manual_seed(seed)
    for L in layers:
        for k, std in (("A", 1.0), ("Gout", 1e-3)):
            if k in L:
                for r0 in range(0, L[k].shape[0], 4096):   # bounded temporaries
                    blk = L[k][r0:r0 + 4096]
                    tmp = torch.empty(blk.shape, dtype=torch.float32, device="cuda")
                    tmp.normal_(0.0, std, generator=gen)
                    blk.copy_(tmp)
                    del tmp


def fill_inputs(layers, w, seed=2306):
    """Seeded synthetic inputs drawn on the GPU with the workload's distributions:
    a ~ N(0, v/rows) (v = 1, or 2 for Student-t(4) rows), g ~ N(0, 1e-6/rows),
    G ~ N(0, 1e-6) (bf16-rounded for bf16 workloads)."""
    import torch
    gen = torch.Generator(device="cuda")
    gen.manual_seed(seed)
    va = 2.0 if w.act_dist == "student_t4" else 1.0
    for L in layers:
        L["a"].normal_(0.0, math.sqrt(va / w.rows), generator=gen)
        L["g"].normal_(0.0, w.grad_row_std / math.sqrt(w.rows), generator=gen)
        if L["G"].dtype == torch.float32:
            L["G"].normal_(0.0, w.G_std, generator=gen)
        else:
            tmp = torch.empty(L["G"].shape, dtype=torch.float32, device="cuda")
            tmp.normal_(0.0, w.G_std, generator=gen)
            L["G"].copy_(tmp)
            del tmp


def cpu_baseline(w, budget_s):
    """The float64 oracle (as is) on a bounded sample: the first block of the
    workload (one layer of each shape), full steps from the initial factors,
    repeated until the time budget is used."""
    import numpy as np

    import oracle as O
    import workloads as W
    affinity = len(os.sched_getaffinity(0))
    try:
        from threadpoolctl import threadpool_info
        threads = max([d.get("num_threads", 1) for d in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = affinity
    nb = len(w.block_shapes)
    inputs = []
    for i in range(nb):
        a, g = W.rank1_vectors(w, i, 0)
        G = W.gradient(w, i, 0)
        L0, R0 = W.initial_factors(w, i)
        inputs.append(dict(Linv=L0.astype(np.float64), Rinv=R0.astype(np.float64), a=a, g=g, G=G))
    p = O.Params(gamma=w.gamma, eps=100.0)
    steps, t0 = 0, time.perf_counter()
    while True:
        out = O.oracle_step(inputs, p)
        for L, o in zip(inputs, out):
            L["Linv"], L["Rinv"] = o["Linv"], o["Rinv"]
        steps += 1
        el = time.perf_counter() - t0
        if el >= budget_s:
            break
    # cores: the threads the oracle ran on (its GEMMs on the BLAS pool; its
    # rank-1 updates are single-threaded NumPy elementwise work)
    return dict(value=nb * steps / el, unit="layer-updates/s", cores=int(threads), kind="oracle",
                blas_threads=int(threads), affinity_cpus=affinity,
                sample=f"first block of the workload ({nb} layers, one of each shape), {steps} full "
                       f"float64 steps in {el:.1f} s")


def stage_times(plan, params, stream, steps):
    """Average ms of each kernel of a step (MKOR_STAGE_*), over `steps` steps
    launched stage by stage with HIP events between consecutive kernels on the
    launch stream."""
    import torch

    from paper_2306_01685_amd import NUM_STAGES
    acc = [0.0] * NUM_STAGES
    for _ in range(steps):
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(NUM_STAGES + 1)]
        ev[0].record(stream)
        for s in range(NUM_STAGES):
            plan.run_stage(params, s)
            ev[s + 1].record(stream)
        torch.cuda.synchronize()
        for s in range(NUM_STAGES):
            acc[s] += ev[s].elapsed_time(ev[s + 1])
    return [a / steps for a in acc]


NOMINAL_GFX_MHZ = 2400.0   # MI355X peak engine clock, the clock the MFMA peaks are quoted at


def clock_during(fn, seconds):
    """Median board power (W) and graphics clock (MHz) from amd-smi (read-only,
    a background thread) while fn runs back to back for `seconds`; the first
    1.5 s are left out.  None if amd-smi gives nothing."""
    import threading

    import torch
    samples, stop = [], threading.Event()

    def sampler():
        while not stop.is_set():
            t, v = time.time(), _smi_sample()
            if v is not None:
                samples.append((t, *v))
            time.sleep(0.1)

    th = threading.Thread(target=sampler, daemon=True)
    th.start()
    torch.cuda.synchronize()
    t0 = time.time()
    while time.time() - t0 < seconds:
        for _ in range(5):
            fn()
        torch.cuda.synchronize()
    stop.set()
    th.join(timeout=30)
    xs = [x for x in samples if x[0] >= t0 + 1.5]
    if not xs:
        return None
    return dict(board_w=statistics.median(x[1] for x in xs), gfx_mhz=statistics.median(x[2] for x in xs),
                samples=len(xs))


def measure(w, args, factor_dtype, gemm_path="auto", sample_power=False):
    """Times mkor_step over the workload with the given factor storage type
    (and, for fp32 factors, GEMM path).  Returns (ms_per_step, kernels,
    roofline, schedule)."""
    import torch

    from paper_2306_01685_amd import NUM_STAGES, STAGE_NAMES, Params, harness as H

    half = factor_dtype == "bf16"
    rank = args.rank if not half else 1
    split = not half and split_eligible(w, gemm_path)
    layers = H.allocate_layers(w.shapes, w.grad_dtype, stats=False, rows=args.rows, act_dtype="bf16",
                               factor_dtype=factor_dtype, rank=rank,
                               gemm_path=None if half else gemm_path)
    if w.init != "identity":
        for i, L in enumerate(layers):
            H.set_factors(L, *initial_factors_stored(w, i, half))
    fill_inputs(layers, w)
    if args.rows:
        fill_rows(layers)
    plan = H.make_plan(layers)
    params = Params(gamma=w.gamma, zeta=0.5, eps=args.eps)
    stream = torch.cuda.current_stream()
    torch.cuda.synchronize()

    for _ in range(args.warmup):
        plan.step(params)
    torch.cuda.synchronize()
    # the paper's protocol: the median of REPEATS timed windows, each of
    # exactly args.steps steps
    windows = timed_windows(lambda: plan.step(params), stream, args.steps, REPEATS)
    ms_step = statistics.median(windows)

    # per-kernel times: the same steps launched stage by stage with HIP events
    # between consecutive kernels on the launch stream
    kernels, roof = {}, None
    esz = 2 if half else 4                                  # factor element bytes
    mfma_peak = BF16_MFMA_PEAK_TF if half else FP32_MFMA_PEAK_TF
    if not args.no_stage_timing:
        ms = stage_times(plan, params, stream, args.steps)
        sq = w.factor_elems
        # stage 1 contracts over d_in (fp32 MFMA: Linv G; split with a bf16 G
        # and d_in > d_out: Linv G) or d_out (G Rinv)
        def k1(i, o):
            if half:
                return o
            if split:
                return i if (w.grad_dtype == "bf16" and i > o) else o
            return i
        f1 = sum(2 * i * o * k1(i, o) for i, o in w.shapes)
        f2 = sum(2 * i * o * (i + o - k1(i, o)) for i, o in w.shapes)
        # bf16 MFMA products per fp32 product on the split: 3 (bf16 G) or 6
        terms = ((3 if w.grad_dtype == "bf16" else 6), 6) if split else (1, 1)
        nel = sum(i * o for i, o in w.shapes)
        gb = 1e-9
        sd = sum(i + o for i, o in w.shapes)
        means_ms, ms = ms[0], ms[1:]   # stage 0: rank-1 means (no work when a and g are given)
        prep_ms, ms = ms[2], ms[:2] + ms[3:]   # operand preparation of the bf16 MFMA paths
        g1, g2 = ("gemm_gr", "gemm_ly") if half else ("sgemm_gr", "sgemm_ly") if split else ("gemm_xt", "gemm_dw")
        # steady state, rank 1: every factor has a pending term, so the pass reads
        # and writes each element once, and the finalize moves O(sum d) (partials,
        # u_raw and x read, w written).  Rank r > 1: the pass only reads (the
        # previous update is already in the factor) and the finalize stage also
        # writes the new update into the factor (a read and a write).
        # the factor of a split layer's first GEMM is written back every other
        # step (two pending terms), so its pass moves 6 B per element on average
        lazy_sq = sum((i * i if (w.grad_dtype == "bf16" and i > o) else o * o) for i, o in w.shapes) if split else 0
        pass_b = (2 * esz * sq - 2 * lazy_sq) if rank == 1 else esz * sq
        fin_b = 12 * sd if rank == 1 else 2 * esz * sq + 12 * rank * sd
        # preparation bytes: the bf16 copy of an fp32 G (bf16 factors), G^T of the
        # split layers with d_in > d_out, the split's row pass over its first
        # GEMM's Q (G or G^T, bf16, min(d_in, d_out) rows of max(d_in, d_out))
        # and w, with (Q w) written per row
        if half:
            prep_b = 6 * nel if w.grad_dtype == "fp32" else 0
        elif split and w.grad_dtype == "bf16":
            prep_b = (sum(4 * i * o for i, o in w.shapes if i > o) + 2 * nel
                      + sum(4 * (i + o) for i, o in w.shapes))
        else:
            prep_b = 0
        kernels = {
            "gemm_prep": dict(ms=prep_ms, alg_bytes=prep_b, gbs=prep_b * gb / (prep_ms / 1e3) if prep_ms > 0 else 0.0),
            "sm_pass": dict(ms=ms[0], alg_bytes=pass_b, gbs=pass_b * gb / (ms[0] / 1e3)),
            "sm_finalize": dict(ms=ms[1], alg_bytes=fin_b, gbs=fin_b * gb / (ms[1] / 1e3)),
            g1: dict(ms=ms[2], flops=f1, tflops=f1 / (ms[2] / 1e3) / 1e12),
            g2: dict(ms=ms[3], flops=f2, tflops=f2 / (ms[3] / 1e3) / 1e12),
            "rescale": dict(ms=ms[4], alg_bytes=8 * nel, gbs=8 * nel * gb / (ms[4] / 1e3)),
        }
        if args.rows:
            mb = args.rows * sd * 2   # every bf16 token row read once
            kernels["means"] = dict(ms=means_ms, alg_bytes=mb, gbs=mb * gb / (means_ms / 1e3),
                                    frac_hbm=mb * gb / (means_ms / 1e3) / HBM_PEAK_GBS,
                                    rows=args.rows)
        sm_ms = ms[0] + ms[1]
        sm_b = pass_b + fin_b
        kernels["sm_total"] = dict(ms=sm_ms, alg_bytes=sm_b, gbs=sm_b * gb / (sm_ms / 1e3),
                                   frac_hbm=sm_b * gb / (sm_ms / 1e3) / HBM_PEAK_GBS)
        pre_ms = ms[2] + ms[3]
        # the split's peak in fp32 products: the bf16 MFMA peak over the bf16
        # products each one takes
        peaks = (BF16_MFMA_PEAK_TF / terms[0], BF16_MFMA_PEAK_TF / terms[1]) if split else (mfma_peak, mfma_peak)
        mfma_ms = (f1 / peaks[0] + f2 / peaks[1]) / 1e12 * 1e3   # both GEMMs at their peaks
        kernels["gemm_total"] = dict(ms=pre_ms, flops=f1 + f2,
                                     tflops=(f1 + f2) / (pre_ms / 1e3) / 1e12,
                                     frac_mfma=mfma_ms / pre_ms,
                                     frac_of_fp32_mfma_peak=(f1 + f2) / (pre_ms / 1e3) / 1e12 / FP32_MFMA_PEAK_TF)
        for k in ("sm_pass", "sm_finalize", "rescale"):
            kernels[k]["frac_hbm"] = kernels[k]["gbs"] / HBM_PEAK_GBS
        # the SM update's algorithmic bytes per step (read every factor element
        # once, write it once), whatever the write-back cadence actually moves
        alg_sm = 2 * esz * sq
        kernels["sm_pass"]["alg_basis_bytes"] = alg_sm
        kernels["sm_pass"]["gbs_alg"] = alg_sm * gb / (ms[0] / 1e3)
        kernels["sm_pass"]["frac_alg"] = kernels["sm_pass"]["gbs_alg"] / HBM_PEAK_GBS
        for k, pk, tm in ((g1, peaks[0], terms[0]), (g2, peaks[1], terms[1])):
            kernels[k]["peak"] = pk
            kernels[k]["frac_mfma"] = kernels[k]["tflops"] / pk
            if split:
                kernels[k]["bf16_mfma_terms"] = tm
                kernels[k]["bf16_mfma_tflops"] = kernels[k]["tflops"] * tm
                # fp32 products per second against the raw bf16 peak (no credit
                # for the split's extra bf16 products)
                kernels[k]["frac_of_bf16_peak"] = kernels[k]["tflops"] / BF16_MFMA_PEAK_TF
        names = ["sm_pass", "sm_finalize", g1, g2, "rescale"]
        dom = max(range(len(names)), key=lambda s: ms[s])
        name = names[dom]
        k = kernels[name]
        traffic = profiled_traffic(name, args.config, half)
        if "flops" in k:
            roof = dict(kernel=name, bound="mfma", achieved=k["tflops"], peak=k["peak"],
                        unit="TFLOP/s", frac=k["frac_mfma"],
                        traffic=None if traffic is None else traffic["total_bytes"],
                        per_launch=f"{k['flops']:.4e} flop (sum of 2*M*N*K over the layers)")
            if split:
                roof["peak_basis"] = (f"fp32 products on the three-way bf16 split: the {BF16_MFMA_PEAK_TF:.0f} "
                                      f"TFLOP/s bf16 MFMA peak / {k['bf16_mfma_terms']} bf16 products each")
                roof["frac_of_fp32_mfma_peak"] = k["tflops"] / FP32_MFMA_PEAK_TF
                roof["frac_of_bf16_peak"] = k["tflops"] / BF16_MFMA_PEAK_TF
                roof["bf16_mfma_tflops"] = k["bf16_mfma_tflops"]
        else:
            roof = dict(kernel=name, bound="hbm", achieved=k["gbs"], peak=HBM_PEAK_GBS, unit="GB/s",
                        frac=k["gbs"] / HBM_PEAK_GBS,
                        traffic=None if traffic is None else traffic["total_bytes"],
                        per_launch=f"{k['alg_bytes']:.4e} B")
        roof["traffic_detail"] = traffic
        if sample_power and roof["bound"] == "mfma" and not getattr(args, "no_power", False):
            # the clock the dominant GEMM runs at: at the board's power limit it
            # is below the nominal clock its peak assumes
            stage = [1, 2, 4, 5, 6][dom]
            pw = clock_during(lambda: plan.run_stage(params, stage), args.power_seconds)
            if pw is not None:
                peak_clk = roof["peak"] * pw["gfx_mhz"] / NOMINAL_GFX_MHZ
                pw.update(nominal_mhz=NOMINAL_GFX_MHZ, peak_at_clock=peak_clk,
                          frac_at_clock=roof["achieved"] / peak_clk,
                          note="amd-smi while this kernel's stage runs back to back after the timed windows")
            roof["power"] = pw
        # the SM update, the step's bandwidth-bound half: its roofline beside (its
        # traffic differs with the GEMM path: only the split path writes some
        # factors every other step)
        k = kernels["sm_pass"]
        t = profiled_traffic("sm_pass" if (half or split) else "sm_pass_fp32", args.config, half)
        roof["sm_update"] = dict(kernel="sm_pass", bound="hbm", achieved=k["gbs"], peak=HBM_PEAK_GBS,
                                 unit="GB/s", frac=k["gbs"] / HBM_PEAK_GBS,
                                 traffic=None if t is None else t["total_bytes"],
                                 per_launch=f"{k['alg_bytes']:.4e} B",
                                 achieved_alg=k["gbs_alg"], frac_alg=k["frac_alg"],
                                 per_launch_alg=f"{k['alg_basis_bytes']:.4e} B (8 B per fp32 factor "
                                                f"element: one read, one write)")

    # The same step captured in a HIP graph (kernel launches only) and replayed.
    graph = None
    if getattr(args, "graph", False):
        side = torch.cuda.Stream()
        side.wait_stream(stream)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.stream(side):
            with torch.cuda.graph(g, stream=side):
                plan.step(params)
        stream.wait_stream(side)
        torch.cuda.synchronize()
        for _ in range(args.warmup):
            g.replay()
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(args.steps):
            g.replay()
        e1.record(stream)
        torch.cuda.synchronize()
        g_ms = e0.elapsed_time(e1) / args.steps
        graph = dict(ms_per_step=g_ms, value=w.n_layers / (g_ms / 1e3), unit="layer-updates/s",
                     note="one mkor_step captured in a HIP graph, replayed")
        del g

    # The paper's schedule: factors updated every 10 iterations (stale factors
    # precondition the other nine); per-step rate averaged over whole cycles.
    schedule = None
    if not args.no_schedule:
        cycles = max(1, args.steps // 10)
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(cycles):
            plan.step(params)
            for _ in range(9):
                plan.precondition(params)
        e1.record(stream)
        torch.cuda.synchronize()
        f_ms = e0.elapsed_time(e1) / (10 * cycles)
        schedule = dict(update_every=10, steps=10 * cycles, ms_per_step=f_ms,
                        value=w.n_layers / (f_ms / 1e3), unit="layer-updates/s")
    # A window in which the stabiliser fires: eps = 0 blends every factor on
    # every step, so the GEMMs run their variants with the diagonal shift
    # (c2 != 0), which the eps = 100 windows above never reach.
    stabilised = None
    if not args.no_stabilised:
        p0 = Params(gamma=w.gamma, zeta=0.5, eps=0.0)
        for _ in range(2):
            plan.step(p0)
        sw = timed_windows(lambda: plan.step(p0), stream, args.steps, REPEATS)
        s_ms = statistics.median(sw)
        stabilised = dict(eps=0.0, ms_per_step=s_ms, value=w.n_layers / (s_ms / 1e3), unit="layer-updates/s",
                          windows_ms_per_step=sw,
                          note="stabiliser fires on every factor at every step (eps = 0)")
        if not args.no_stage_timing:
            st = stage_times(plan, p0, stream, args.steps)
            stabilised["gemm_ms"] = [st[4], st[5]]
    del plan, layers
    torch.cuda.empty_cache()
    if graph is not None:
        kernels["graph_replay"] = graph
    extra = dict(windows_ms_per_step=windows, stabilised_step=stabilised)
    return ms_step, kernels, roof, schedule, extra


def measure_opt(w, args):
    """The same workload stepped with mkor_step_opt (backend LAMB fused into the
    rescale, weights and moments of every layer in HBM) against mkor_step."""
    import torch

    from paper_2306_01685_amd import OPT_LAMB, OptParams, Params, harness as H

    layers = H.allocate_layers(w.shapes, w.grad_dtype, stats=False, optimizer="lamb")
    fill_inputs(layers, w)
    for L in layers:
        L["W"].normal_(0.0, 0.02)
    plan = H.make_plan(layers)
    params = Params(gamma=w.gamma, zeta=0.5, eps=args.eps)
    stream = torch.cuda.current_stream()
    res = {}
    for name in ("step", "step_opt"):
        for t in range(args.warmup):
            if name == "step":
                plan.step(params)
            else:
                plan.step_opt(params, OptParams(kind=OPT_LAMB, step=t + 1, lr=1e-3))
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for t in range(args.steps):
            if name == "step":
                plan.step(params)
            else:
                plan.step_opt(params, OptParams(kind=OPT_LAMB, step=args.warmup + t + 1, lr=1e-3))
        e1.record(stream)
        torch.cuda.synchronize()
        res[name] = e0.elapsed_time(e1) / args.steps
    nel = sum(i * o for i, o in w.shapes)
    del plan, layers
    torch.cuda.empty_cache()
    # LAMB pass A reads dW_hat, W, m, v and writes m, v; pass B reads m, v, W and writes W
    extra_ms = res["step_opt"] - res["step"]
    return dict(kind="lamb", ms_per_step=res["step_opt"], ms_per_step_without=res["step"],
                value=w.n_layers / (res["step_opt"] / 1e3), unit="layer-updates/s",
                optimizer_bytes=40 * nel, extra_ms=extra_ms,
                note="step with LAMB fused into the rescale (weights, m, v in HBM) vs the step that only "
                     "writes dW; the optimizer itself moves 40 B per weight (rescale pass 24 + 12 read/4 "
                     "write of the second pass) in place of the rescale's 8")


def initial_factors_stored(w, i, half):
    """The workload's initial factors, rounded to bf16 for bf16 storage."""
    import workloads as W
    L0, R0 = W.initial_factors(w, i)
    if half:
        L0, R0 = W.round_to_bf16(L0), W.round_to_bf16(R0)
    return L0, R0


def _smi_sample():
    """One reading of socket power (W) and the mean graphics clock of the XCDs
    (MHz) from `amd-smi metric` (read-only), or None."""
    import subprocess
    try:
        r = subprocess.run(["amd-smi", "metric", "-g", "0", "-p", "-c", "--json"],
                           capture_output=True, text=True, timeout=15)
        g = json.loads(r.stdout)["gpu_data"][0]
        clks = [v["clk"]["value"] for k, v in g["clock"].items()
                if k.startswith("gfx_") and isinstance(v, dict) and isinstance(v["clk"]["value"], (int, float))]
        return float(g["power"]["socket_power"]["value"]), statistics.mean(clks)
    except Exception:  # noqa: BLE001  (tool missing, or a field not reported)
        return None


def power_profile(args):
    """--mode power: the step and its GEMM stages (split, bf16 factors, fp32
    MFMA) and the rescale, each launched back to back for --power-seconds,
    with board power and graphics clock sampled by a background thread.  The
    first 1.5 s of each phase are left out (the clock settles)."""
    import threading

    import torch

    import workloads as W
    from paper_2306_01685_amd import STAGE_NAMES, Params, harness as H

    w = W.WORKLOADS[args.config]
    samples, stop = [], threading.Event()

    def sampler():
        while not stop.is_set():
            t, v = time.time(), _smi_sample()
            if v is not None:
                samples.append((t, *v))
            time.sleep(0.1)

    def make(factor_dtype, gemm_path):
        layers = H.allocate_layers(w.shapes, w.grad_dtype, stats=False, factor_dtype=factor_dtype,
                                   gemm_path=None if factor_dtype == "bf16" else gemm_path)
        fill_inputs(layers, w)
        plan = H.make_plan(layers)
        p = Params(gamma=w.gamma, zeta=0.5, eps=args.eps)
        for _ in range(3):
            plan.step(p)
        torch.cuda.synchronize()
        return layers, plan, p

    phases = []

    def phase(name, fn):
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0, n = time.time(), 0
        e0.record()
        while time.time() - t0 < args.power_seconds:
            for _ in range(5):
                fn()
            n += 5
            torch.cuda.synchronize()
        e1.record()
        torch.cuda.synchronize()
        phases.append(dict(name=name, t0=t0, t1=time.time(), calls=n, ms_per_call=e0.elapsed_time(e1) / n))

    th = threading.Thread(target=sampler, daemon=True)
    th.start()
    t_idle = time.time()
    time.sleep(3.0)
    phases.append(dict(name="idle", t0=t_idle - 1.5, t1=time.time(), calls=0, ms_per_call=0.0))
    stage = {n: i for i, n in enumerate(STAGE_NAMES)}
    if split_eligible(w, "auto"):
        runs = [("fp32", "auto", "split"), ("bf16", None, "bf16_factors"), ("fp32", "fp32", "fp32_mfma")]
    else:
        runs = [("fp32", "fp32", "fp32_mfma"), ("bf16", None, "bf16_factors")]
    for fdt, path, tag in runs:
        layers, plan, p = make(fdt, path)
        phase(f"{tag}: step", lambda: plan.step(p))
        phase(f"{tag}: first GEMM", lambda: plan.run_stage(p, stage["gemm_xt"]))
        phase(f"{tag}: second GEMM", lambda: plan.run_stage(p, stage["gemm_dw"]))
        if tag == "split":
            phase("rescale", lambda: plan.run_stage(p, stage["rescale"]))
        del plan, layers
        torch.cuda.empty_cache()
    stop.set()
    th.join(timeout=30)
    out = []
    for ph in phases:
        xs = [x for x in samples if ph["t0"] + 1.5 <= x[0] <= ph["t1"]]
        out.append(dict(name=ph["name"], ms_per_call=ph["ms_per_call"], samples=len(xs),
                        power_w=statistics.median([x[1] for x in xs]) if xs else None,
                        gfx_mhz=statistics.median([x[2] for x in xs]) if xs else None))
    print(json.dumps({"mode": "power", "workload": workload_desc(w), "phases": out,
                      "note": "board (socket) power and mean graphics clock of the 8 XCDs, medians"}), flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only: --gpus {args.gpus} is not supported "
              "(the hot path runs on a single MI355X)", file=sys.stderr)
        sys.exit(2)

    if args.mode == "copy":
        copy_reference(args)
        return
    if args.mode == "power":
        power_profile(args)
        return

    import torch

    import workloads as W

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    w = W.WORKLOADS[args.config]
    ms_step, kernels, roof, schedule, extra = measure(w, args, args.factor_dtype, args.gemm_path, sample_power=True)
    value = w.n_layers / (ms_step / 1e3)
    fp32_path = None
    if (args.factor_dtype == "fp32" and not args.no_fp32_path and args.rank == 1
            and split_eligible(w, args.gemm_path)):
        # the same workload on the fp32 MFMA GEMMs, reported beside
        f_ms, f_k, f_roof, _, _ = measure(w, argparse.Namespace(**{**vars(args), "no_schedule": True,
                                                                   "no_stabilised": True}), "fp32", "fp32")
        fp32_path = dict(value=w.n_layers / (f_ms / 1e3), unit="layer-updates/s", ms_per_step=f_ms,
                         gemm="fp32 MFMA (v_mfma_f32_32x32x2_f32)", roofline=f_roof, kernels=f_k)
    half = None
    if args.factor_dtype == "fp32" and not args.no_half and args.rank == 1:
        # the same workload with half-precision (bf16) factors, reported beside
        h_ms, h_k, h_roof, h_sched, _ = measure(w, argparse.Namespace(**{**vars(args), "no_stabilised": True}),
                                                "bf16", sample_power=True)
        half = dict(value=w.n_layers / (h_ms / 1e3), unit="layer-updates/s", ms_per_step=h_ms,
                    dtype="bf16 factors, bf16 MFMA (fp32 accumulation)", roofline=h_roof,
                    schedule_f10=h_sched, kernels=h_k)

    opt = None
    if args.factor_dtype == "fp32" and not args.no_opt and args.rank == 1:
        opt = measure_opt(w, args)
    refs = None
    if not args.no_references:
        refs = dict(copy_kernel=copy_measure(args.copy_mib, args.steps, args.warmup),
                    torch_matmul_fp32=torch_matmul_reference(w),
                    torch_matmul_bf16=torch_matmul_bf16_reference(sample_power=not args.no_power))
        bf = roof.get("bf16_mfma_tflops")
        if bf is not None:
            # the dominant split GEMM's bf16 matrix-core rate beside the rate
            # the library's own bf16 GEMM sustains on this part
            lib = refs["torch_matmul_bf16"]["tflops"]
            roof["vs_library_bf16"] = dict(kernel_bf16_mfma_tflops=bf, library_bf16_tflops=lib, ratio=bf / lib)
        if half is not None and half["roofline"]["bound"] == "mfma":
            hr, lib = half["roofline"], refs["torch_matmul_bf16"]["tflops"]
            hr["vs_library_bf16"] = dict(kernel_bf16_mfma_tflops=hr["achieved"], library_bf16_tflops=lib,
                                         ratio=hr["achieved"] / lib)

    out = {
        "metric": METRIC, "value": value, "unit": "layer-updates/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32" if args.factor_dtype == "fp32" else "bf16",
        "data": "synthetic (seeded; layer shapes only)",
        "config": {"workload": workload_desc(w, args.factor_dtype), "n_layers": w.n_layers,
                   "factor_elems": w.factor_elems, "precond_flops": w.precond_flops,
                   "gamma": w.gamma, "zeta": 0.5, "eps": args.eps, "grad_dtype": w.grad_dtype,
                   "factor_dtype": args.factor_dtype, "token_rows": args.rows, "rank": args.rank,
                   "gemm": ("bf16 factors, bf16 MFMA" if args.factor_dtype == "bf16" else
                            "fp32 operands as exact three-way bf16 splits on bf16 MFMA, fp32 accumulation"
                            if split_eligible(w, args.gemm_path) else "fp32 MFMA")},
        "roofline": roof,
        "timing": {"repeats": REPEATS, "windows_ms_per_step": extra["windows_ms_per_step"],
                   "statistic": "median of the windows (the paper's median of 5 runs)"},
        "stabilised_step": extra["stabilised_step"],
        "references": refs,
        "schedule_f10": schedule,
        "kernels": kernels,
        "fp32_mfma_path": fp32_path,
        "half_factors": half,
        "fused_optimizer": opt,
        "device": torch.cuda.get_device_name(0),
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, args.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
