#!/usr/bin/env python3
"""Benchmark of the MI355X SiLU Gated MLP, Y = (silu(X Wg) * (X Wu)) Wd.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
                    [--variant silu|swiglu|glu|rmsnorm|rmsnorm_swiglu]

One step is one full pass of the hot path (a gate/up kernel and a down
kernel: split-K GEMVs for T <= 8, MFMA GEMMs above) over one batch of
synthetic inputs already resident in HBM.  W untimed steps,
then exactly K steps timed with HIP events on the library's stream,
bracketed by device synchronisation (the paper times 100 runs after 20
warm-ups, Section 6.1; those are the defaults here).

Memory-bound workloads rotate through several device copies of the weights
(over 1 GB in total), so that each step streams its weights from HBM rather
than from the 256 MB Infinity Cache.

By default (--workload suite) prints ONE JSON line: the T=1 decode workload
(the HBM half of the metric) as the line's value, and under "configs" the
other four Gated MLP workloads measured in the same run (tiny, small_batch,
prefill and large_prefill: the MFMA half of the metric at T >= 2048), each
with its own step time, value, roofline and CPU baseline.  --workload NAME
prints one line for that workload alone (all: one line per workload).
Each record has:
  value      whole-job throughput: GB/s of algorithmic bytes 2(3DF + 2TD)
             for memory-bound shapes, TFLOP/s of 6TDF for compute-bound ones;
  roofline   the dominant kernel (the gate/up kernel; with --path fused
             the one kernel, i.e. the step) launched on its own and timed
             with HIP events on the library's stream: its algorithmic bytes
             or flops per launch over its average duration, against the
             MI355X peak (8 TB/s HBM, 2.5 PFLOP/s dense bf16);
  cpu_baseline  the CPU fp64 oracle on this host's cores, on a bounded
             sample of the same workload, scaled to the same unit.
--variant selects a member of the Gated MLP family (default: the SiLU Gated
MLP): swiglu = swish gate with beta 1.702, glu = sigmoid gate, rmsnorm =
RMSNorm of X in front (eps 1e-6), rmsnorm_swiglu = both.
--workload softmax_matmul (M = K = N = 8192) or softmax_matmul_tiny benches
the second workload, Z = softmax(X) Y computed as (exp(X - rowmax) Y) / rowsum
(one exp/row-sum kernel, then the matmul with the divide in its epilogue):
value in TFLOP/s of 2MKN, the matmul kernel as the dominant one.
--path picks the kernel path (auto, gemv, mfma, or fused: the one-kernel
decode path); --graph adds the step's time when captured in a HIP graph and
replayed; --vendor-gemm adds the vendor library's time for the same matmul
shapes (context).  The default run also times, after the workloads, loops of
MFMAs on register operands (paper_2606_26344_amd/mfma_ceiling, 32x32x16 and
16x16x32, random and all-zero data): under the board's power limit the
random-data rate of an instruction is the ceiling of any GEMM on random data
that issues it, reported beside the MFMA-bound records as
roofline.power_capped_mfma, with the fraction of the dominant kernel's own
instruction (--mfma-ceiling prints the ceilings alone).  Only one GPU is
used: --gpus above 1 exits with a message.
"""
from __future__ import annotations

import argparse
import ctypes
import json
import math
import os
import subprocess
import sys
import time

METRIC = ("Gated-MLP TFLOP/s & % bf16 MFMA peak (prefill); "
          "GB/s & % HBM peak (decode)")
SMM_METRIC = "Softmax+MatMul TFLOP/s & % bf16 MFMA peak"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, published
BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 MFMA, published (no sparsity)
RIDGE = BF16_PEAK_TFLOPS * 1e12 / (HBM_PEAK_GBS * 1e9)  # ~312 FLOP/B
MALL_DEFEAT_BYTES = 1.1e9      # rotate weights over at least this many bytes
COPY_BYTES = 256 << 20         # size of the calibration copy
HERE = os.path.dirname(os.path.abspath(__file__))
# Members of the Gated MLP family: oracle/binding keyword arguments.
VARIANTS = {
    "silu": {},
    "swiglu": {"activation": "swish", "beta": 1.702},
    "glu": {"activation": "sigmoid"},
    "rmsnorm": {"rmsnorm": True, "eps": 1e-6},
    "rmsnorm_swiglu": {"activation": "swish", "beta": 1.702, "rmsnorm": True, "eps": 1e-6},
}
PROFILES = os.path.join(HERE, "profiles")
CSRC = os.path.join(HERE, "paper_2606_26344_amd", "csrc")


def kernel_source_sha256():
    """Hash of the HIP sources without their comments and whitespace: a
    traffic record is only valid for the kernels it was measured on."""
    import hashlib
    import re

    h = hashlib.sha256()
    for name in sorted(os.listdir(CSRC)):
        if name.endswith((".hip", ".hpp")):
            with open(os.path.join(CSRC, name)) as fh:
                code = fh.read()
            code = re.sub(r"/\*.*?\*/", " ", code, flags=re.S)
            code = re.sub(r"//[^\n]*", " ", code)
            code = " ".join(code.split())
            h.update(name.encode() + b"\0" + code.encode())
    return h.hexdigest()


def committed_traffic(workload, kernel):
    """HBM bytes per launch of `kernel` from the committed rocprofv3 record
    for this workload, or None if absent or measured on other sources."""
    path = os.path.join(PROFILES, "traffic_%s.json" % workload)
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        rec = json.load(fh)
    if rec.get("source_sha256") != kernel_source_sha256():
        return None
    k = rec.get("kernels", {}).get(kernel)
    return None if k is None else k.get("traffic_bytes_per_launch")


def parse_args(argv=None):
    p = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=100)
    p.add_argument("--warmup", type=int, default=20)
    p.add_argument("--workload", default="suite",
                   help="suite (default: the decode line, with the other four Gated MLP "
                        "workloads as nested records) | decode | tiny | small_batch | prefill | "
                        "large_prefill | softmax_matmul | softmax_matmul_tiny | all")
    p.add_argument("--variant", default="silu", choices=sorted(VARIANTS),
                   help="member of the Gated MLP family (default: the SiLU Gated MLP)")
    p.add_argument("--path", default="auto", choices=["auto", "gemv", "mfma", "fused", "fused_mfma"],
                   help="kernel path of the Gated MLP step (fused: both GEMV steps in one kernel, "
                        "T <= 8; fused_mfma: both MFMA steps in one kernel, T <= 64)")
    p.add_argument("--graph", action="store_true",
                   help="also time the step captured in a HIP graph (one step per weight copy, "
                        "replayed; context for launch overhead)")
    p.add_argument("--copies", type=int, default=0,
                   help="weight copies to rotate through (0: enough to exceed 1.1 GB "
                        "for memory-bound shapes, 1 otherwise)")
    p.add_argument("--cpu-seconds", type=float, default=12.0,
                   help="approximate CPU time budget of the oracle baseline")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--copy-calibration", action="store_true",
                   help="after the timed region, run plain device copies of %d MiB (a known "
                        "number of bytes) for calibrating rocprofv3 FETCH_SIZE / WRITE_SIZE"
                        % (COPY_BYTES >> 20))
    p.add_argument("--power", type=float, default=0.0, metavar="SECONDS",
                   help="after the measurement, run steps back to back for SECONDS while sampling "
                        "the board's socket power and shader clocks with amd-smi (context for the "
                        "MFMA roofline: the board's power cap sets the clock)")
    p.add_argument("--sweep-tokens", metavar="T,T,...",
                   help="instead of the benchmark line: the step time at each token count T "
                        "(D and F of --workload, weights rotated as for the workload's decode "
                        "shape), one JSON line per T and path; with --path auto also the GEMV, "
                        "MFMA and fused paths for T <= 8 and the MFMA and fused MFMA paths up "
                        "to T = 64")
    p.add_argument("--mfma-ceiling", action="store_true",
                   help="print the board's sustained bf16 MFMA rate on random and zero operands "
                        "(the power-limited ceiling of the MFMA-bound steps) and exit")
    p.add_argument("--vendor-gemm", action="store_true",
                   help="also time torch.matmul (the vendor GEMM library) on the same two "
                        "matmul shapes, for context (X [T,D] x [Wg|Wu] [D,2F], H [T,F] x Wd)")
    p.add_argument("--summarize-profile", metavar="DIR", nargs="+",
                   help="print per-kernel averages from rocprofv3 CSV output directories "
                        "and exit (no GPU work)")
    p.add_argument("--write-traffic", metavar="JSON",
                   help="with --summarize-profile: FETCH_SIZE and WRITE_SIZE runs of "
                        "--copy-calibration benches -> traffic record for the roofline")
    return p.parse_args(argv)


def algorithmic(T, D, F):
    """Bytes any method must move (X, three weights, Y) and FLOPs (6TDF)."""
    return 2.0 * (3.0 * D * F + 2.0 * T * D), 6.0 * T * D * F


def gate_up_algorithmic(T, D, F):
    """Per launch of the gate/up kernel: reads X, Wg, Wu, writes H."""
    return 2.0 * (2.0 * D * F + T * D + T * F), 4.0 * T * D * F


def cpu_baseline(w, X, Wg, Wu, Wd, bound, budget_s, variant=None):
    import numpy as np

    import oracle

    orc = oracle.default_oracle()
    T, D, F = w.T, w.D, w.F
    nbytes, flops = algorithmic(T, D, F)
    threads = orc.max_threads()
    # Calibrate on a few rows (as many as the threads, which work on whole
    # rows), then size the sample to fill the time budget.
    variant = variant or {}
    c = min(T, 2 * threads)
    t0 = time.perf_counter()
    orc.gated_mlp_rows(X, Wg, Wu, Wd, rows=np.arange(c), **variant)
    t_row = max((time.perf_counter() - t0) / c, 1e-6)
    n = int(max(1, min(T, budget_s // t_row)))
    rows = np.linspace(0, T - 1, n).round().astype(np.int64) if n < T else None
    reps = 1 if n < T else int(max(1, min(100000, budget_s // (t_row * T))))
    t0 = time.perf_counter()
    for _ in range(reps):
        orc.gated_mlp_rows(X, Wg, Wu, Wd, rows=rows, **variant)
    t_total = time.perf_counter() - t0
    rows_done = (T if rows is None else n)
    t_full = (t_total / reps) * T / rows_done  # seconds per full step
    if bound == "hbm":
        value, unit = nbytes / t_full / 1e9, "GB/s"
    else:
        value, unit = flops / t_full / 1e12, "TFLOP/s"
    if rows is None:
        sample = "all %d rows, %d repetitions (%.1f s)" % (T, reps, t_total)
    else:
        sample = ("%d of %d rows (evenly spaced), %d repetition(s) in %.1f s, "
                  "time extrapolated x%.1f to the full step" % (n, T, reps, t_total, T / n))
    return {"value": round(value, 6), "unit": unit, "cores": threads, "kind": "oracle",
            "sample": sample, "seconds_per_step": t_full}


def run_workload(name, args):
    import torch

    from paper_2606_26344_amd import gmlp
    from paper_2606_26344_amd import inputs as I

    w = I.WORKLOADS[name]
    T, D, F = w.T, w.D, w.F
    nbytes, flops = algorithmic(T, D, F)
    bound = "hbm" if flops / nbytes < RIDGE else "mfma"
    lib = gmlp.library()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    t_gen = time.perf_counter()
    X, Wg, Wu, Wd = I.generate(T, D, F, seed=w.seed, unit_rms_rows=w.unit_rms_rows)
    t_gen = time.perf_counter() - t_gen

    weight_bytes = 2.0 * 3 * D * F
    # Rotating copies keeps the weights out of the 256 MB Infinity Cache for
    # memory-bound shapes; weights of a few MB stay in the L2 caches whatever
    # is rotated (the tiny workload is bound by latency), so they get one copy.
    big = weight_bytes >= 64e6
    copies = args.copies or (max(3, math.ceil(MALL_DEFEAT_BYTES / weight_bytes))
                             if bound == "hbm" and big else 1)
    x = gmlp.from_bf16_bits(X, dev)
    wsets = [tuple(gmlp.from_bf16_bits(a, dev) for a in (Wg, Wu, Wd))]
    for _ in range(copies - 1):
        wsets.append(tuple(t.clone() for t in wsets[0]))
    y = torch.empty((T, D), dtype=torch.bfloat16, device=dev)
    h = torch.empty((T, F), dtype=torch.bfloat16, device=dev)
    ws = gmlp.Workspace(T, D, F, device=dev)
    stream = torch.cuda.current_stream(dev)
    st = ctypes.c_void_p(stream.cuda_stream)
    P = ctypes.c_void_p
    xp, yp, hp, wsp = P(x.data_ptr()), P(y.data_ptr()), P(h.data_ptr()), P(ws.buffer.data_ptr())
    wp = [tuple(P(t.data_ptr()) for t in s) for s in wsets]
    path_id = gmlp._PATHS[args.path]
    variant = VARIANTS[args.variant]
    vargs = gmlp._variant(variant.get("activation", "silu"), variant.get("beta", 1.0),
                          variant.get("rmsnorm", False), variant.get("eps", 0.0))

    def step(i, stream_ptr=st):
        g, u, d = wp[i % copies]
        if not variant:
            return lib.gmlp_forward_ex(xp, g, u, d, yp, T, D, F, path_id, wsp, ws.nbytes, stream_ptr)
        return lib.gmlp_forward_variant(xp, g, u, d, yp, T, D, F, *vargs, path_id, wsp, ws.nbytes,
                                        stream_ptr)

    # The steps alone run on the step's own path (the fused path has no
    # single-step form: its steps alone are the GEMV kernels it fuses).
    step_path = {"fused": gmlp.PATH_GEMV, "fused_mfma": gmlp.PATH_MFMA}.get(args.path, path_id)

    def gate_up_only(i):
        g, u, _ = wp[i % copies]
        if not variant:
            return lib.gmlp_gate_up_ws(xp, g, u, hp, T, D, F, step_path, wsp, ws.nbytes, st)
        return lib.gmlp_gate_up_variant(xp, g, u, hp, T, D, F, *vargs, step_path, wsp, ws.nbytes, st)

    def down_only(i):
        _, _, d = wp[i % copies]
        return lib.gmlp_down_ws(hp, d, yp, T, F, D, step_path, wsp, ws.nbytes, st)

    def timed(fn, k):
        """Average ms per call over k calls on the library stream (HIP events)."""
        start = torch.cuda.Event(enable_timing=True)
        end = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        start.record(stream)
        for i in range(k):
            rc = fn(i)
            if rc:
                raise gmlp.GmlpError(rc, gmlp.last_error())
        end.record(stream)
        torch.cuda.synchronize()
        return start.elapsed_time(end) / k

    # Warm-up, then the timed region: exactly K steps.
    for i in range(args.warmup):
        if step(i):
            raise gmlp.GmlpError(1, gmlp.last_error())
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    ms_per_step = timed(step, args.steps)
    wall = time.perf_counter() - wall0

    # The gate/up and down kernels, each launched and timed alone.
    k_kernel = max(args.steps, 20)
    gate_up_ms = timed(gate_up_only, k_kernel)
    down_ms = timed(down_only, k_kernel)
    plan = gmlp.describe(T, D, F, args.path)
    stats = per_step_stats(step, k_kernel, stream)
    # Context only: every step on the same weight copy, which the 256 MB
    # Infinity Cache may then serve in part.
    unrotated_ms = timed(lambda i: step(0), k_kernel) if copies > 1 else None
    graph_ms = graph_step_ms(step, copies, args.steps, dev) if args.graph else None

    sec = ms_per_step / 1e3
    if bound == "hbm":
        value, unit = nbytes / sec / 1e9, "GB/s"
    else:
        value, unit = flops / sec / 1e12, "TFLOP/s"
    if len(plan) == 1:
        # One kernel is the whole step: its launches are the timed steps.
        dom_kernel, dom_ms = plan[0][0], ms_per_step
        dom_bytes, dom_flops = nbytes, flops
    else:
        dom_kernel, dom_ms = plan[0][0], gate_up_ms
        dom_bytes, dom_flops = gate_up_algorithmic(T, D, F)
    if bound == "hbm":
        achieved, peak, r_unit = dom_bytes / (dom_ms / 1e3) / 1e9, HBM_PEAK_GBS, "GB/s"
    else:
        achieved, peak, r_unit = dom_flops / (dom_ms / 1e3) / 1e12, BF16_PEAK_TFLOPS, "TFLOP/s"
    path = args.path if args.path != "auto" else ("gemv" if plan[0][0].startswith("gemv") else "mfma")
    props = torch.cuda.get_device_properties(dev)
    result = {
        "metric": METRIC,
        "value": round(value, 3),
        "unit": unit,
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": "%s%s: T=%d, D=%d, F=%d%s" % (
                name, "" if args.variant == "silu" else " (%s Gated MLP)" % args.variant, T, D, F,
                ", X rows at unit RMS" if w.unit_rms_rows else ""),
            "variant": dict({"name": args.variant}, **variant),
            "T": T, "D": D, "F": F,
            "path": path,
            "kernels": [{"name": k, "grid": g, "block": b, "k_splits": sp} for k, g, b, sp in plan],
            "weight_copies_rotated": copies,
            "parallelism": "single GPU",
        },
        "roofline": {
            "bound": bound,
            "achieved": round(achieved, 3),
            "peak": peak,
            "unit": r_unit,
            "frac": round(achieved / peak, 4),
            "traffic": committed_traffic(name, dom_kernel),
            "kernel": dom_kernel,
            "per_launch": ("%.4g bytes" % dom_bytes) if bound == "hbm" else ("%.4g flop" % dom_flops),
            "avg_launch_us": round(dom_ms * 1e3, 3),
        },
        "step": {
            "gbs": round(nbytes / sec / 1e9, 3),
            "tflops": round(flops / sec / 1e12, 3),
            "frac_hbm_peak": round(nbytes / sec / 1e9 / HBM_PEAK_GBS, 4),
            "frac_bf16_peak": round(flops / sec / 1e12 / BF16_PEAK_TFLOPS, 4),
            "gate_up_alone_us": round(gate_up_ms * 1e3, 3),
            "down_alone_us": round(down_ms * 1e3, 3),
            "wall_s": round(wall, 4),
            "single_steps": stats,
            "unrotated_weights_us": None if unrotated_ms is None else round(unrotated_ms * 1e3, 3),
            "graph_replay_us": None if graph_ms is None else round(graph_ms * 1e3, 3),
        },
        "device": {"name": props.name, "cus": props.multi_processor_count,
                   "arch": getattr(props, "gcnArchName", "")},
        "input_generation_s": round(t_gen, 2),
    }
    if args.copy_calibration:
        # A plain elementwise pass reading and writing COPY_BYTES (the only
        # elementwise kernel this script launches).
        src = torch.empty(COPY_BYTES, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.mul(src, 1, out=dst)
        torch.cuda.synchronize()
        result["copy_calibration_bytes"] = COPY_BYTES
        del src, dst
    if args.vendor_gemm:
        result["vendor_gemm"] = vendor_gemm(T, D, F, args, wsets, x, stream)
    if args.power > 0:
        result["power"] = power_samples(step, args.power, stream)
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(w, X, Wg, Wu, Wd, bound, args.cpu_seconds, variant)
    del wsets, x, y, h, ws
    torch.cuda.empty_cache()
    return result


def parse_smi_csv(text):
    """(socket power in W, [shader clock of every XCD in MHz]) from the CSV
    that `amd-smi metric -p -c --csv` prints, or None if a field is missing."""
    import csv
    import io
    import re

    try:
        row = next(csv.DictReader(io.StringIO(text)))
        clocks = [float(row[k]) for k in sorted(row, key=lambda k: k or "")
                  if re.fullmatch(r"gfx_\d+_clk", k or "")]
        return float(row["socket_power"]), clocks
    except (StopIteration, KeyError, ValueError, TypeError):
        return None


def _smi_sample():
    """One amd-smi reading (see parse_smi_csv), or None."""
    import subprocess

    try:
        r = subprocess.run(["amd-smi", "metric", "-p", "-c", "--csv"], capture_output=True, text=True,
                           timeout=10)
    except (OSError, subprocess.SubprocessError):
        return None
    return parse_smi_csv(r.stdout)


def power_samples(step, seconds, stream):
    """Run `step` back to back for `seconds` on `stream` while another thread
    samples amd-smi every 0.25 s (after a 0.5 s settling time)."""
    import statistics
    import threading

    import torch

    samples, done = [], threading.Event()

    def sampler():
        if done.wait(0.5):
            return
        while not done.is_set():
            s_ = _smi_sample()
            if s_ is not None:
                samples.append(s_)
            done.wait(0.25)

    th = threading.Thread(target=sampler)
    th.start()
    t0 = time.time()
    n = 0
    with torch.cuda.stream(stream):
        while time.time() - t0 < seconds:
            for i in range(20):
                step(n + i)
            n += 20
            torch.cuda.synchronize()
    wall = time.time() - t0
    done.set()
    th.join()
    if not samples:
        return {"error": "amd-smi gave no socket power / clock readings"}
    watts = [s_[0] for s_ in samples]
    clocks = [c for s_ in samples for c in s_[1]]
    return {
        "tool": "amd-smi metric -p -c",
        "samples": len(samples),
        "steps": n,
        "us_per_step": round(wall / n * 1e6, 2),
        "socket_power_w": {"mean": round(statistics.mean(watts), 1), "max": max(watts)},
        "gfx_clock_mhz": {"mean": round(statistics.mean(clocks), 1), "min": min(clocks), "max": max(clocks)}
        if clocks else None,
    }


def per_step_stats(fn, k, stream):
    """Median, mean and min of k single steps, each between its own pair of
    HIP events on the library's stream (after the timed region; the value
    reported is still the K-step bracket)."""
    import statistics

    import torch

    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(k)]
    torch.cuda.synchronize()
    for i, (a, b) in enumerate(evs):
        a.record(stream)
        rc = fn(i)
        if rc:
            raise RuntimeError("step failed with status %d" % rc)
        b.record(stream)
    torch.cuda.synchronize()
    us = [a.elapsed_time(b) * 1e3 for a, b in evs]
    return {"median_us": round(statistics.median(us), 3), "mean_us": round(statistics.fmean(us), 3),
            "min_us": round(min(us), 3), "steps": k}


def graph_step_ms(step, copies, k, dev):
    """ms per step of `copies` steps (one per weight copy) captured in one HIP
    graph on a side stream and replayed until about k steps have run."""
    import ctypes

    import torch

    side = torch.cuda.Stream(device=dev)
    sp = ctypes.c_void_p(side.cuda_stream)
    side.wait_stream(torch.cuda.current_stream(dev))
    with torch.cuda.stream(side):
        for i in range(copies):
            if step(i, sp):
                raise RuntimeError("step failed before capture")
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        for i in range(copies):
            step(i, sp)
    reps = max(1, k // copies)
    with torch.cuda.stream(side):
        graph.replay()
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    with torch.cuda.stream(side):
        start.record(side)
        for _ in range(reps):
            graph.replay()
        end.record(side)
    torch.cuda.synchronize()
    return start.elapsed_time(end) / (reps * copies)


def smm_algorithmic(M, K, N):
    """Softmax+MatMul: bytes any method must move (X, Y, Z) and FLOPs (2MKN)."""
    return 2.0 * (M * K + K * N + M * N), 2.0 * M * K * N


def exp_rows_algorithmic(M, K):
    """Per launch of the exp/row-sum kernel: reads X, writes P and the sums."""
    return 2.0 * M * K * 2 + 4.0 * M


def smm_cpu_baseline(X, Y, bound, budget_s):
    import numpy as np

    from oracle import softmax_matmul as so

    orc = so.default_oracle()
    M, K = X.shape
    N = Y.shape[1]
    nbytes, flops = smm_algorithmic(M, K, N)
    threads = orc_threads()
    c = min(M, 2 * threads)
    t0 = time.perf_counter()
    orc.rows(X, Y, rows=np.arange(c))
    t_row = max((time.perf_counter() - t0) / c, 1e-6)
    n = int(max(1, min(M, budget_s // t_row)))
    rows = np.linspace(0, M - 1, n).round().astype(np.int64) if n < M else None
    reps = 1 if n < M else int(max(1, min(100000, budget_s // (t_row * M))))
    t0 = time.perf_counter()
    for _ in range(reps):
        orc.rows(X, Y, rows=rows)
    t_total = time.perf_counter() - t0
    t_full = (t_total / reps) * M / (M if rows is None else n)
    if bound == "hbm":
        value, unit = nbytes / t_full / 1e9, "GB/s"
    else:
        value, unit = flops / t_full / 1e12, "TFLOP/s"
    if rows is None:
        sample = "all %d rows, %d repetitions (%.1f s)" % (M, reps, t_total)
    else:
        sample = ("%d of %d rows (evenly spaced), %d repetition(s) in %.1f s, "
                  "time extrapolated x%.1f to the full step" % (n, M, reps, t_total, M / n))
    return {"value": round(value, 6), "unit": unit, "cores": threads, "kind": "oracle",
            "sample": sample, "seconds_per_step": t_full}


def orc_threads():
    import oracle

    return oracle.default_oracle().max_threads()


def run_softmax_matmul(name, args):
    import torch

    from paper_2606_26344_amd import gmlp
    from paper_2606_26344_amd import inputs as I
    from paper_2606_26344_amd import softmax_matmul as smm

    w = I.SOFTMAX_MATMUL_WORKLOADS[name]
    M, K, N = w.M, w.K, w.N
    nbytes, flops = smm_algorithmic(M, K, N)
    bound = "hbm" if flops / nbytes < RIDGE else "mfma"
    lib = gmlp.library()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    t_gen = time.perf_counter()
    X, Y = I.generate_softmax_matmul(M, K, N, seed=w.seed, logit_scale=w.logit_scale)
    t_gen = time.perf_counter() - t_gen
    x, y = gmlp.from_bf16_bits(X, dev), gmlp.from_bf16_bits(Y, dev)
    z = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
    p = torch.empty((M, K), dtype=torch.bfloat16, device=dev)
    sums = torch.empty((M,), dtype=torch.float32, device=dev)
    ws = smm.make_workspace(M, K, N, device=dev)
    stream = torch.cuda.current_stream(dev)
    st = ctypes.c_void_p(stream.cuda_stream)
    P = ctypes.c_void_p
    xp, yp, zp, pp, sp = (P(t.data_ptr()) for t in (x, y, z, p, sums))
    wsp = P(ws.buffer.data_ptr())
    auto = gmlp.PATH_AUTO

    def step(i):
        return lib.softmax_matmul_ws(xp, yp, zp, M, K, N, auto, wsp, ws.nbytes, st)

    def exp_rows_only(i):
        return lib.softmax_matmul_exp_rows(xp, pp, sp, M, K, st)

    def divide_only(i):
        return lib.softmax_matmul_divide_ws(pp, sp, yp, zp, M, K, N, auto, wsp, ws.nbytes, st)

    def timed(fn, k):
        start = torch.cuda.Event(enable_timing=True)
        end = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        start.record(stream)
        for i in range(k):
            rc = fn(i)
            if rc:
                raise gmlp.GmlpError(rc, gmlp.last_error())
        end.record(stream)
        torch.cuda.synchronize()
        return start.elapsed_time(end) / k

    for i in range(args.warmup):
        if step(i):
            raise gmlp.GmlpError(1, gmlp.last_error())
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    ms_per_step = timed(step, args.steps)
    wall = time.perf_counter() - wall0
    k_kernel = max(args.steps, 20)
    exp_ms = timed(exp_rows_only, k_kernel)
    mm_ms = timed(divide_only, k_kernel)
    plan = smm.describe(M, K, N)
    stats = per_step_stats(step, k_kernel, stream)

    sec = ms_per_step / 1e3
    if bound == "hbm":
        value, unit = nbytes / sec / 1e9, "GB/s"
    else:
        value, unit = flops / sec / 1e12, "TFLOP/s"
    dom_kernel = plan[1][0]
    if bound == "hbm":
        dom = 2.0 * (M * K + K * N + M * N) + 4.0 * M
        achieved, peak, r_unit = dom / (mm_ms / 1e3) / 1e9, HBM_PEAK_GBS, "GB/s"
        per_launch = "%.4g bytes" % dom
    else:
        achieved, peak, r_unit = flops / (mm_ms / 1e3) / 1e12, BF16_PEAK_TFLOPS, "TFLOP/s"
        per_launch = "%.4g flop" % flops
    exp_bytes = exp_rows_algorithmic(M, K)
    props = torch.cuda.get_device_properties(dev)
    result = {
        "metric": SMM_METRIC,
        "value": round(value, 3),
        "unit": unit,
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": "%s: M=%d, K=%d, N=%d, logits N(0, %g^2)" % (name, M, K, N, w.logit_scale),
            "M": M, "K": K, "N": N,
            "path": "gemv" if M <= 8 else "mfma",
            "kernels": [{"name": k, "grid": g, "block": b, "k_splits": s_} for k, g, b, s_ in plan],
            "parallelism": "single GPU",
        },
        "roofline": {
            "bound": bound,
            "achieved": round(achieved, 3),
            "peak": peak,
            "unit": r_unit,
            "frac": round(achieved / peak, 4),
            "traffic": committed_traffic(name, dom_kernel),
            "kernel": dom_kernel,
            "per_launch": per_launch,
            "avg_launch_us": round(mm_ms * 1e3, 3),
        },
        "step": {
            "gbs": round(nbytes / sec / 1e9, 3),
            "tflops": round(flops / sec / 1e12, 3),
            "frac_bf16_peak": round(flops / sec / 1e12 / BF16_PEAK_TFLOPS, 4),
            "exp_rows_alone_us": round(exp_ms * 1e3, 3),
            "exp_rows_gbs": round(exp_bytes / (exp_ms / 1e3) / 1e9, 3),
            "exp_rows_frac_hbm_peak": round(exp_bytes / (exp_ms / 1e3) / 1e9 / HBM_PEAK_GBS, 4),
            "exp_rows_traffic": committed_traffic(name, plan[0][0]),
            "matmul_divide_alone_us": round(mm_ms * 1e3, 3),
            "wall_s": round(wall, 4),
            "single_steps": stats,
        },
        "device": {"name": props.name, "cus": props.multi_processor_count,
                   "arch": getattr(props, "gcnArchName", "")},
        "input_generation_s": round(t_gen, 2),
    }
    if args.copy_calibration:
        src = torch.empty(COPY_BYTES, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.mul(src, 1, out=dst)
        torch.cuda.synchronize()
        result["copy_calibration_bytes"] = COPY_BYTES
        del src, dst
    if args.vendor_gemm:
        # Context: the vendor library's plain matmul on the same shape (no
        # softmax, no divide), and torch's softmax followed by it.
        a = torch.randn((M, K), device=dev).to(torch.bfloat16)
        plain = lambda i: torch.matmul(a, y, out=z) is None  # noqa: E731
        composed = lambda i: torch.matmul(torch.softmax(x, dim=1), y, out=z) is None  # noqa: E731
        for i in range(args.warmup):
            plain(i)
            composed(i)
        tm = timed(plain, k_kernel)
        ts = timed(composed, k_kernel)
        result["vendor_gemm"] = {"matmul_us": round(tm * 1e3, 3),
                                 "matmul_tflops": round(flops / (tm / 1e3) / 1e12, 3),
                                 "softmax_then_matmul_us": round(ts * 1e3, 3)}
        del a
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = smm_cpu_baseline(X, Y, bound, args.cpu_seconds)
    del x, y, z, p, sums, ws
    torch.cuda.empty_cache()
    return result


def vendor_gemm(T, D, F, args, wsets, x, stream):
    """The vendor library's time for the two matmul shapes of a step (no
    activation, no fusion): context for the MFMA kernels, not a baseline of
    the method.  Both weights of the first matmul are concatenated into one
    [D, 2F] operand, so it is one library call as the fused kernel is one
    launch.  Consecutive calls rotate through the same weight copies as the
    step, so that the 256 MB Infinity Cache serves neither."""
    import torch

    w2s = [torch.cat([wg, wu], dim=1).contiguous() for wg, wu, _ in wsets]
    wds = [wd for _, _, wd in wsets]
    h = torch.empty((T, F), dtype=torch.bfloat16, device=x.device).normal_()

    def timed(fn, k):
        for i in range(args.warmup):
            fn(i)
        torch.cuda.synchronize()
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for i in range(k):
            fn(i)
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) / k

    gu_ms = timed(lambda i: torch.matmul(x, w2s[i % len(w2s)]), args.steps)
    dn_ms = timed(lambda i: torch.matmul(h, wds[i % len(wds)]), args.steps)
    out = {"library": "torch.matmul (" + ("hipBLASLt" if torch.version.hip else "vendor") + ")",
           "gate_up_us": round(gu_ms * 1e3, 3), "down_us": round(dn_ms * 1e3, 3),
           "gate_up_tflops": round(4.0 * T * D * F / (gu_ms / 1e3) / 1e12, 3),
           "down_tflops": round(2.0 * T * D * F / (dn_ms / 1e3) / 1e12, 3)}
    del w2s, wds, h
    return out


def _read_counter_csvs(dirs):
    """Per-kernel mean of each counter over dispatches (rocprofv3 CSV)."""
    import csv
    import glob
    from collections import defaultdict

    tot = defaultdict(lambda: defaultdict(float))
    disp = defaultdict(lambda: defaultdict(set))
    span = defaultdict(dict)  # kernel -> dispatch -> duration (ns) in the counter run
    for d in dirs:
        for path in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
            with open(path) as fh:
                for r in csv.DictReader(fh):
                    k, c = r["Kernel_Name"], r["Counter_Name"]
                    tot[k][c] += float(r["Counter_Value"])
                    disp[k][c].add((path, r["Dispatch_Id"]))
                    if r.get("Start_Timestamp") and r.get("End_Timestamp"):
                        span[k][(path, r["Dispatch_Id"])] = (float(r["End_Timestamp"])
                                                             - float(r["Start_Timestamp"]))
    out = {k: {c: v / len(disp[k][c]) for c, v in cs.items()} for k, cs in tot.items()}
    for k, spans in span.items():
        out[k]["duration_ns"] = sum(spans.values()) / len(spans)
    return out


def _read_kernel_stats(dirs):
    import csv
    import glob

    rows = []
    for d in dirs:
        for path in glob.glob(os.path.join(d, "**", "*kernel_stats.csv"), recursive=True):
            with open(path) as fh:
                rows += list(csv.DictReader(fh))
    return rows


def summarize_profile(args):
    counters = _read_counter_csvs(args.summarize_profile)
    for k, cs in sorted(counters.items()):
        print(k)
        for c, v in sorted(cs.items()):
            print("    %-28s %.6g" % (c, v))
        if cs.get("GRBM_GUI_ACTIVE") and cs.get("duration_ns", 0) > 100e3:
            # GRBM_GUI_ACTIVE adds up the busy cycles of the 8 XCDs: cycles per
            # XCD over the dispatch's duration is the average shader clock, and
            # the dense bf16 peak scales with it (2.5 PFLOP/s at 2.4 GHz).  Only
            # for dispatches long enough (> 100 us) for the ratio to mean it.
            ghz = cs["GRBM_GUI_ACTIVE"] / 8.0 / cs["duration_ns"]
            print("    %-28s %.4g" % ("avg_clock_ghz", ghz))
            print("    %-28s %.4g" % ("bf16_peak_at_clock_tflops", BF16_PEAK_TFLOPS * ghz / 2.4))
    for r in _read_kernel_stats(args.summarize_profile):
        print("%-80s calls %6s  avg %10.3f us  total %12.3f us  %6.2f%%" % (
            r["Name"][:80], r["Calls"], float(r["AverageNs"]) / 1e3,
            float(r["TotalDurationNs"]) / 1e3, float(r["Percentage"])))
    if args.write_traffic:
        # Calibrate against the plain copy: it reads and writes COPY_BYTES.
        copy = [cs for k, cs in counters.items() if "elementwise" in k.lower()]
        fetch_copy = max((cs.get("FETCH_SIZE", 0.0) for cs in copy), default=0.0)
        write_copy = max((cs.get("WRITE_SIZE", 0.0) for cs in copy), default=0.0)
        f_fetch = COPY_BYTES / 1024.0 / fetch_copy if fetch_copy else None
        f_write = COPY_BYTES / 1024.0 / write_copy if write_copy else None
        rec = {"source_sha256": kernel_source_sha256(), "copy_bytes": COPY_BYTES,
               "copy_fetch_kib": fetch_copy, "copy_write_kib": write_copy,
               "fetch_factor": f_fetch, "write_factor": f_write, "kernels": {}}
        for k, cs in counters.items():
            if "gmlp::" in k:
                # The name gmlp_describe gives the kernel.
                short = k.split("(")[0].replace("void ", "", 1).replace("gmlp::", "")
                fe, wr = cs.get("FETCH_SIZE"), cs.get("WRITE_SIZE")
                tb = None
                if fe is not None and wr is not None and f_fetch and f_write:
                    tb = round(fe * 1024.0 * f_fetch + wr * 1024.0 * f_write)
                rec["kernels"][short] = {"fetch_kib_per_launch": fe, "write_kib_per_launch": wr,
                                         "traffic_bytes_per_launch": tb}
        with open(args.write_traffic, "w") as fh:
            json.dump(rec, fh, indent=1, sort_keys=True)
            fh.write("\n")
        print("wrote", args.write_traffic)
    return 0


def sweep_tokens(name, tokens, args):
    """Step time of the Gated MLP at each T in `tokens`, at the D and F of
    workload `name`: K steps after W warm-up steps, HIP events on the
    library's stream, weights rotated through enough copies to defeat the
    256 MB Infinity Cache.  Prints one JSON line per (T, path)."""
    import torch

    from paper_2606_26344_amd import gmlp
    from paper_2606_26344_amd import inputs as I

    w = I.WORKLOADS[name]
    D, F = w.D, w.F
    lib = gmlp.library()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    X, Wg, Wu, Wd = I.generate(max(tokens), D, F, seed=w.seed)
    copies = args.copies or max(3, math.ceil(MALL_DEFEAT_BYTES / (2.0 * 3 * D * F)))
    wsets = [tuple(gmlp.from_bf16_bits(a, dev) for a in (Wg, Wu, Wd))]
    for _ in range(copies - 1):
        wsets.append(tuple(t.clone() for t in wsets[0]))
    xa = gmlp.from_bf16_bits(X, dev)
    stream = torch.cuda.current_stream(dev)
    st = ctypes.c_void_p(stream.cuda_stream)
    P = ctypes.c_void_p
    wp = [tuple(P(t.data_ptr()) for t in s_) for s_ in wsets]
    for T in tokens:
        paths = [args.path]
        if args.path == "auto" and T <= 8:
            paths += ["gemv", "mfma", "fused"]
        if args.path == "auto" and 8 < T <= 64:
            paths += ["mfma"]
        if args.path == "auto" and T <= 64:
            paths += ["fused_mfma"]
        x = xa[:T].contiguous()
        y = torch.empty((T, D), dtype=torch.bfloat16, device=dev)
        ws = gmlp.Workspace(T, D, F, device=dev)
        for path in paths:
            path_id = gmlp._PATHS[path]

            def step(i):
                g, u, d = wp[i % copies]
                rc = lib.gmlp_forward_ex(P(x.data_ptr()), g, u, d, P(y.data_ptr()), T, D, F, path_id,
                                         P(ws.buffer.data_ptr()), ws.nbytes, st)
                if rc:
                    raise RuntimeError(gmlp.last_error())

            for i in range(args.warmup):
                step(i)
            torch.cuda.synchronize()
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            a.record(stream)
            for i in range(args.steps):
                step(i)
            b.record(stream)
            b.synchronize()
            us = a.elapsed_time(b) * 1e3 / args.steps
            nbytes, flops = algorithmic(T, D, F)
            print(json.dumps({
                "T": T, "D": D, "F": F, "path": path, "us_per_step": round(us, 2),
                "gbs": round(nbytes / us / 1e3, 1), "tflops": round(flops / us / 1e6, 1),
                "kernels": [k for k, *_ in gmlp.describe(T, D, F, path)],
            }), flush=True)
        del ws, x, y


# Fields of a workload's record that the suite keeps in its nested records.
SUITE_KEYS = ("value", "unit", "ms_per_step", "steps", "warmup", "config", "roofline", "step",
              "cpu_baseline")
SUITE_HEADLINE = "decode"


MFMA_CEILING = os.path.join(HERE, "paper_2606_26344_amd", "mfma_ceiling")


def mfma_ceiling(ms=20.0):
    """The board's sustained bf16 matrix-core rate: mfma_ceiling (built with
    the library) issues MFMAs back to back on register operands, random and
    then all-zero, for about `ms` each, with the GEMM kernels' instruction
    (32x32x16: the plain keys) and with 16x16x32 (keys suffixed _16x16x32).
    Under the board's power limit the random-data rate is what a GEMM on
    random data could reach at best with that instruction; the zero-data rate
    shows the clock-limited peak.  Context for the roofline, not its peak
    (that stays the published dense peak)."""
    import torch

    if not os.path.exists(MFMA_CEILING):
        return {"error": "mfma_ceiling is not built (python -m paper_2606_26344_amd.build)"}
    if torch.cuda.is_initialized():
        torch.cuda.synchronize()
    res = subprocess.run([MFMA_CEILING, "%g" % ms], capture_output=True, text=True, timeout=120)
    if res.returncode != 0:
        return {"error": "mfma_ceiling exited with %d: %s" % (res.returncode, res.stderr.strip()[-200:])}
    runs = [json.loads(ln) for ln in res.stdout.splitlines() if ln.startswith("{")]
    out = {"ms_per_run": ms, "command": "paper_2606_26344_amd/mfma_ceiling %g" % ms}
    for r in runs:
        # The GEMM kernels' instruction (32x32x16) under the plain keys.
        suffix = "" if r.get("mfma", "32x32x16") == "32x32x16" else "_" + r["mfma"]
        out["%s_data_tflops%s" % (r["data"], suffix)] = r["tflops"]
    return out


def mfma_instruction(kernel):
    """The MFMA instruction a gemm_mfma_kernel<GemmShape<NW, WM, WN, TM, TN,
    STAGES, BK>> issues: v_mfma_f32_16x16x32_bf16 where its tile has 256
    columns (WM TM 32) or 256 tokens (WN TN 32) and 64-row k-tiles, else
    v_mfma_f32_32x32x16_bf16."""
    if "GemmShape<" not in kernel:
        return "32x32x16"
    nw, wm, wn, tm, tn, stages, bk = [int(v) for v in kernel.split("GemmShape<")[1].split(">")[0].split(",")[:7]]
    return "16x16x32" if bk == 64 and (wm * tm * 32 >= 256 or wn * tn * 32 >= 256) else "32x32x16"


def run_suite(args):
    """The default benchmark: one JSON line whose value is the decode
    workload's (T = 1, the configuration the HBM half of the metric is quoted
    on), with the other four Gated MLP workloads (tiny, small_batch, prefill,
    large_prefill: the MFMA half of the metric) measured in the same run,
    each with its own roofline and CPU baseline, under "configs"."""
    from paper_2606_26344_amd import inputs as I

    result = run_workload(SUITE_HEADLINE, args)
    sub = argparse.Namespace(**vars(args))
    sub.cpu_seconds = max(2.0, args.cpu_seconds / 2)  # bounded total run time
    # The nested records follow the paper's protocol (20 warm-ups, then 100
    # timed runs, Section 6.1) unless more are asked for: a prefill step takes
    # about a millisecond, and a handful of warm-up steps leaves the clock
    # still settling under the board's power cap.
    sub.warmup = max(args.warmup, 20)
    sub.steps = max(args.steps, 100)
    sub.graph = sub.copy_calibration = sub.vendor_gemm = False
    sub.power = 0.0
    sub.path = "auto"  # the plan each workload's shape gets
    configs = {}
    for name in I.WORKLOADS:
        if name == SUITE_HEADLINE:
            continue
        rec = run_workload(name, sub)
        configs[name] = {k: rec[k] for k in SUITE_KEYS if k in rec}
        print("suite: %s %.3f %s, %.1f us per step" % (name, rec["value"], rec["unit"],
                                                       rec["ms_per_step"] * 1e3),
              file=sys.stderr, flush=True)
    # The matrix-core ceiling under the board's power limit, next to the
    # MFMA-bound records (measured once, after them).
    ceiling = mfma_ceiling()
    for rec in configs.values():
        if rec["roofline"]["bound"] == "mfma":
            ctx = dict(ceiling)
            # The dominant kernel's own instruction: 16x16x32 for the tiles
            # of 256 tokens or 256 columns, else 32x32x16.
            instr = mfma_instruction(rec["roofline"].get("kernel", ""))
            ctx["kernel_mfma"] = instr
            key = "random_data_tflops" + ("" if instr == "32x32x16" else "_" + instr)
            if key in ceiling:
                ctx["frac_of_random_data_ceiling"] = round(rec["roofline"]["achieved"] / ceiling[key], 4)
            rec["roofline"]["power_capped_mfma"] = ctx
    result["config"]["suite"] = [SUITE_HEADLINE] + list(configs)
    result["configs"] = configs
    return result


def main(argv=None):
    args = parse_args(argv)
    if args.summarize_profile:
        return summarize_profile(args)
    if args.mfma_ceiling:
        print(json.dumps(mfma_ceiling()), flush=True)
        return 0
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the Gated MLP here runs on a single MI355X "
              "(--gpus %d, WORLD_SIZE %d requested); run with --gpus 1." % (args.gpus, world),
              file=sys.stderr)
        return 2
    from paper_2606_26344_amd import inputs as I

    if args.workload == "suite" and not args.sweep_tokens:
        print(json.dumps(run_suite(args)), flush=True)
        return 0
    names = (list(I.WORKLOADS) + list(I.SOFTMAX_MATMUL_WORKLOADS) if args.workload == "all"
             else ["decode" if args.workload == "suite" else args.workload])
    for name in names:
        if name not in I.WORKLOADS and name not in I.SOFTMAX_MATMUL_WORKLOADS:
            print("unknown workload %r" % name, file=sys.stderr)
            return 2
    if args.sweep_tokens:
        if names[0] not in I.WORKLOADS:
            print("--sweep-tokens needs a Gated MLP workload", file=sys.stderr)
            return 2
        sweep_tokens(names[0], [int(t) for t in args.sweep_tokens.split(",")], args)
        return 0
    for name in names:
        run = run_softmax_matmul if name in I.SOFTMAX_MATMUL_WORKLOADS else run_workload
        print(json.dumps(run(name, args)), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
