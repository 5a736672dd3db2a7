#!/usr/bin/env python3
"""Throughput of the candidate-scoring step on one MI355X.

One step = validity filter (model V) -> performance prediction over the
accepted candidates (model P) -> top-k selection, over a pool that is
already resident in HBM, through the C ABI (libml2.so).  The default
workload is the 16M-candidate pool (16,777,216 x 128 features; V: 300 trees
of depth 6; P: 1000 trees of depth 8; k = 1024).

Prints ONE JSON line.  `value` is candidates scored+filtered per second.
The `roofline` object covers the dominant kernel (the performance walk),
with achieved node visits/s measured with HIP events on the launch stream.
The `cpu_baseline` object times the CPU oracle (all host cores) on a
bounded sample of the same pool.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--two-pass] [--graph]
    python bench.py --copy-probe      # plain 1 GiB device copies (counter scale)
    python bench.py --probe           # LDS, VALU and walk-loop microbenchmarks
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

HBM_PEAK_GBS = 8000.0
# Node-visit ceiling of the chip, from its unit counts and clock (256 CUs,
# 2.4 GHz).  A visit needs, per lane, two LDS reads (the 8-byte node and the
# 4-byte feature value) and, as counted on the walks (SQ_INSTS_VALU per
# wave-visit: 5.01 in the perf walk, 5.27 in the validity walk), five VALU
# instructions (node address, feature address, the comparison
# x[feature] < threshold, the step to the chosen child, and the share of the
# fold and of the staging).
#   VALU: the fp32 vector peak of 157.3 TFLOP/s is 78.6 T lane-FMAs/s, i.e.
#         128 lanes per clock per CU -> 78.6 T / 5 = 15.7 T visits/s.
#   LDS:  256 bytes per clock per CU (CDNA4 doubled CDNA3's 128; the
#         consecutive 16-byte read probe of --probe reaches 156 B/clk)
#         -> 157 TB/s / 12 B = 13.1 T visits/s.
# The lower one, the LDS ceiling, is the peak.  Beside it the line carries
# the walk loop's measured rate at the perf walk's shape (the probe of
# --probe: the same loop over a resident chunk, no row loads or restaging).
VALU_LANE_OPS_PER_S = 256 * 128 * 2.4e9
VALU_PER_VISIT = 5
VISIT_PEAK_VALU = VALU_LANE_OPS_PER_S / VALU_PER_VISIT
LDS_BYTES_PER_S = 256 * 256 * 2.4e9
VISIT_PEAK_LDS = LDS_BYTES_PER_S / 12
VISIT_PEAK_PER_S = min(VISIT_PEAK_VALU, VISIT_PEAK_LDS)
MALL_BYTES = 256 << 20  # MI355X Infinity Cache: pools below it are flushed between steps
# The perf walk's launch shape (depth, trees per lane, lanes per candidate,
# waves, features) where the walk-loop probe is built for it: the 16M pool,
# the explorer workload (64 visible columns) and the Skewed pool (depth 10).
PERF_WALK_SHAPE = {"roofline": (8, 4, 2, 8, 128), "explorer": (8, 8, 1, 8, 64),
                   "skewed": (10, 4, 1, 6, 64)}
# The validity walk's launch shape on the same pools.
VALIDITY_WALK_SHAPE = {"roofline": (6, 8, 2, 8, 128), "explorer": (6, 8, 1, 8, 64),
                       "skewed": (6, 8, 1, 8, 64)}
METRIC = "candidate configs scored+filtered/sec (validity+perf+top-k); % of HBM peak"
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "walk_traffic_16m.json")
KERNEL_SOURCE = os.path.join(ROOT, "paper_2411_10764_amd", "csrc", "walk_kernels.hip")


def _log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def _kernel_sha() -> str:
    with open(KERNEL_SOURCE, "rb") as fh:
        return hashlib.sha256(fh.read()).hexdigest()


def _traffic(kernel_sha: str, workload: str):
    """HBM bytes per launch of the workload's dominant walk (the perf walk of
    the 16M pool, the one-pass walk of the HBM diagnostic) from committed
    rocprofv3 counter runs, or None when absent or taken on a different
    kernel source."""
    try:
        with open(TRAFFIC_FILE) as fh:
            t = json.load(fh)
    except (OSError, ValueError):
        return None
    if t.get("kernel_source_sha256") != kernel_sha:
        return None
    return t.get("launches", {}).get(workload, {}).get("bytes_per_launch")


def copy_probe() -> None:
    import torch
    n = 1 << 28  # 1 GiB of float32
    a = torch.ones(n, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    for _ in range(5):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes": 4 * n, "launches": 5}))


def copy_bandwidth(dev) -> float:
    """A plain device-to-device copy of 1 GiB (torch's copy kernel), timed
    with HIP events: bytes read + written per second (GB/s), median of 5."""
    import torch
    n = 1 << 28
    a = torch.ones(n, dtype=torch.float32, device=dev)
    b = torch.empty_like(a)
    for _ in range(2):
        b.copy_(a)
    ts = []
    for _ in range(5):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        b.copy_(a)
        e1.record()
        torch.cuda.synchronize()
        ts.append(e0.elapsed_time(e1))
    del a, b
    return 2.0 * 4 * n / (float(np.median(ts)) / 1000.0) / 1e9


def probes() -> None:
    """Microbenchmarks of the units the walks use (include/ml2_probe.h), as
    one JSON line: LDS bytes per clock per CU by read width and pattern,
    32-bit add lane operations per second, and the walk's inner loop (a
    resident chunk, no row loads or restaging) in node visits per second at
    the 16M pool's two walk shapes.  Clock rates assume 2.4 GHz."""
    import torch
    from paper_2411_10764_amd import ml2
    torch.cuda.init()
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    clk = 2.4e9
    lds = {}
    names = ["b32_consecutive", "b64_consecutive", "b128_consecutive",
             "b32_random", "b64_random", "b128_random"]
    for mode, name in enumerate(names):
        ms, nbytes = ml2.ml2_probe_lds(mode, 2048, 4 * cus)
        lds[name] = round(nbytes / (ms * 1e-3) / clk / cus, 1)
    ms, ops = ml2.ml2_probe_valu(4096, 8 * cus)
    valu = ops / (ms * 1e-3)
    visit = {}
    # (depth, trees per lane, lanes per candidate, waves, features): the 16M
    # pool's validity and perf walks first, then other shapes of depth 8,
    # then the Skewed pool's perf walk (depth 10, 64 features) and shapes
    # whose tiles and chunk also fit the LDS there
    shapes = [(6, 8, 2, 8, 128), (8, 4, 2, 8, 128), (8, 2, 2, 8, 128), (8, 4, 2, 4, 128),
              (8, 8, 2, 4, 128), (8, 4, 2, 6, 128), (8, 8, 2, 6, 128), (8, 4, 2, 8, 64),
              (8, 8, 2, 8, 64), (8, 4, 1, 8, 64), (8, 8, 1, 8, 64),
              (10, 2, 1, 8, 64), (10, 1, 1, 8, 64), (10, 4, 1, 6, 64), (10, 4, 1, 4, 64),
              (10, 1, 2, 8, 64), (10, 2, 2, 8, 64), (10, 4, 2, 6, 64), (10, 4, 2, 4, 64)]
    for d, g, s_, w, f in shapes:
        ms, visits = ml2.ml2_probe_visit(d, g, s_, w, f, {6: 1024, 8: 512, 10: 256}[d], 4 * cus)
        visit[f"D{d}_G{g}_S{s_}_W{w}_F{f}"] = round(visits / (ms * 1e-3) / 1e12, 3)
    print(json.dumps({
        "probe": "ml2_probe_*", "cus": cus, "clock_ghz_assumed": clk / 1e9,
        "lds_bytes_per_clk_per_cu": lds,
        "lds_peak_bytes_per_clk_per_cu": LDS_BYTES_PER_S / clk / 256,
        "valu_tlane_ops_per_s": round(valu / 1e12, 2),
        "valu_peak_tlane_ops_per_s": round(VALU_LANE_OPS_PER_S / 1e12, 2),
        "walk_loop_tvisits_per_s": visit,
        "visit_peak_tvisits_per_s": round(VISIT_PEAK_PER_S / 1e12, 2),
    }), flush=True)


def mean_path(ens, X) -> float:
    """Mean number of splits on a candidate's paths through all trees of a
    ragged ensemble (its node visits), over the rows of X."""
    dl = ens.default_left
    total = 0.0
    for t in range(ens.num_trees):
        base = int(ens.offsets[t])
        node = np.zeros(X.shape[0], np.int64)
        active = ens.left[base + node] >= 0
        while active.any():
            g = base + node[active]
            x = X[np.flatnonzero(active), ens.feature[g]]
            left = (x < ens.threshold[g]) | (np.isnan(x) & (dl[g] != 0))
            node[active] = np.where(left, ens.left[g], ens.right[g])
            total += float(active.sum())
            active = ens.left[base + node] >= 0
    return total / X.shape[0]


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def cpu_baseline(w, rows: int, rows_one: int):
    """The oracle as it stands on the host cores: all usable threads on the
    first `rows` candidates, and one thread on the first `rows_one`."""
    import gen
    import oracle
    threads = gen.default_threads()
    X = w.features(rows=np.arange(rows, dtype=np.int64))
    V, P = oracle.OracleEnsemble(w.validity()), oracle.OracleEnsemble(w.perf())
    A = oracle.OracleEnsemble(w.second_level()) if w.a_trees else None

    def run(Xs, t):
        t0 = time.perf_counter()
        out = oracle.pipeline(V, P, Xs, w.k, threads=t)
        if A is not None:
            oracle.rerank(A, Xs, out["idx"], w.keep)
        return time.perf_counter() - t0

    dt = run(X, threads)
    dt1 = run(X[:rows_one], 1)
    steps = f"validity -> masked perf -> top-{w.k}" + (f" -> model A keeps {w.keep}" if A else "")
    return {"value": rows / dt, "unit": "candidates/s", "cores": threads, "kind": "oracle",
            "sample": f"first {rows} candidates of the {w.name} pool ({w.F} features), "
                      f"{steps}, {dt:.2f} s wall on {threads} threads "
                      f"({os.cpu_count()} visible cpus)",
            "single_core": {"value": rows_one / dt1, "unit": "candidates/s", "cores": 1,
                            "sample": f"first {rows_one} candidates, the same steps, "
                                      f"{dt1:.2f} s wall on one thread"},
            "cpu_model": cpu_model()}


def walk_loop_ceiling(shape):
    """T visits/s of the walk's inner loop at `shape` (the --probe
    microbenchmark, timed live on this device)."""
    import torch
    from paper_2411_10764_amd import ml2
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    d, g, s_, waves, f = shape
    ms, visits = ml2.ml2_probe_visit(d, g, s_, waves, f, {6: 1024, 8: 512, 10: 256}[d], 4 * cus)
    return visits / (ms * 1e-3) / 1e12


def explore(args, w, X, v, p, dev) -> int:
    """The explorer's rounds (Section 2; N = 10, alpha = 1 in Section 3): each
    round holds (alpha+1)N accepted rows by P, model A keeps N.  Timed twice:
    rescoring the pool every round (models retrained between rounds, as in
    the paper) and reusing the scores (models unchanged)."""
    import torch
    from paper_2411_10764_amd import ml2
    N = args.N
    k = int(round((args.alpha + 1) * N))
    a = ml2.ml2_load_ensemble(w.second_level()) if w.a_trees else None
    R = args.explore
    ex = ml2.Explorer(v, p, a, w.n, k, N, R)
    idx = torch.empty(N, dtype=torch.int32, device=dev)
    top = torch.empty(N, dtype=torch.float32, device=dev)
    num = torch.empty(1, dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream()
    out = {"metric": "explorer rounds/sec", "unit": "rounds/s", "n_gpus": 1,
           "higher_is_better": True, "dtype": "f32", "data": "synthetic",
           "config": {"workload": w.name, "candidates": w.n, "N": N, "alpha": args.alpha,
                      "held_per_round": k, "rounds": R,
                      "second_level": f"{w.a_trees} trees x depth {w.a_depth}" if a else None}}
    for mode, rescore in (("rescore", True), ("reuse", False)):
        ex.reset()
        ex.round(X, idx, top, num, rescore=True, stream=stream)  # warm, and scores for "reuse"
        torch.cuda.synchronize()
        ex.reset()
        ex.round(X, idx, top, num, rescore=True, stream=stream)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(R - 1):
            ex.round(X, idx, top, num, rescore=rescore, stream=stream)
        torch.cuda.synchronize()
        dt = time.perf_counter() - t0
        out[mode] = {"rounds_per_s": (R - 1) / dt, "ms_per_round": 1000 * dt / (R - 1),
                     "proposed_last_round": int(num.item())}
        _log(f"{mode}: {1000 * dt / (R - 1):.3f} ms per round over {R - 1} rounds")
    out["value"] = out["rescore"]["rounds_per_s"]
    ex.free()
    print(json.dumps(out), flush=True)
    return 0


def explore_stream(args, w, v, p, dev) -> int:
    """The explorer's rounds over a pool that arrives in row chunks (Section
    2; N = 10, alpha = 1 in Section 3): each round streams every chunk of the
    pool through ml2_stream_explorer_chunk.  Timed two ways: chunks that are
    slices of a pool resident in HBM (the scoring rate), and chunks copied
    from pinned host memory into two device staging buffers on a copy
    stream, overlapped with the scoring of the previous chunk (the rate with
    the host-to-device copies included)."""
    import torch
    import gen
    from paper_2411_10764_amd import ml2
    N = args.N
    k = int(round((args.alpha + 1) * N))
    rows = args.chunk_rows
    R = args.explore_stream
    a = ml2.ml2_load_ensemble(w.second_level()) if w.a_trees else None
    ex = ml2.StreamExplorer(v, p, a, rows, k, N, 2 * R + 4)
    spans = [(r0, min(rows, w.n - r0)) for r0 in range(0, w.n, rows)]
    idx = torch.empty(N, dtype=torch.int32, device=dev)
    top = torch.empty(N, dtype=torch.float32, device=dev)
    num = torch.empty(1, dtype=torch.int32, device=dev)
    main = torch.cuda.current_stream()

    _log(f"pool {w.n} x {w.F} in {len(spans)} chunks of {rows} rows; pinned host copy")
    host = torch.empty((w.n, w.F), dtype=torch.float32, pin_memory=True)
    hn = host.numpy()
    for r0, m in spans:
        gen.features(w.seed, m, w.F, w.K, row0=r0, out=hn[r0:r0 + m], missing=w.missing)
    X = torch.empty((w.n, w.F), dtype=torch.float32, device=dev)
    X.copy_(host)
    torch.cuda.synchronize()

    def resident_round():
        ex.begin(main)
        for r0, m in spans:
            ex.chunk(X[r0:r0 + m], r0, main)
        ex.end(idx, top, num, main)

    copy = torch.cuda.Stream()
    stage = [torch.empty((rows, w.F), dtype=torch.float32, device=dev) for _ in range(2)]
    copied = [torch.cuda.Event() for _ in range(2)]
    used = [torch.cuda.Event() for _ in range(2)]
    for e in used:
        e.record(main)

    def streamed_round():
        ex.begin(main)
        for c, (r0, m) in enumerate(spans):
            b = c % 2
            copy.wait_event(used[b])
            with torch.cuda.stream(copy):
                stage[b][:m].copy_(host[r0:r0 + m], non_blocking=True)
            copied[b].record(copy)
            main.wait_event(copied[b])
            ex.chunk(stage[b][:m], r0, main)
            used[b].record(main)
        ex.end(idx, top, num, main)

    out = {"metric": "explorer rounds/sec (pool streamed in row chunks)", "unit": "rounds/s",
           "n_gpus": 1, "higher_is_better": True, "dtype": "f32", "data": "synthetic",
           "config": {"workload": w.name, "candidates": w.n, "features": w.F, "N": N,
                      "alpha": args.alpha, "held_per_round": k, "chunk_rows": rows,
                      "chunks": len(spans), "rounds": R,
                      "second_level": f"{w.a_trees} trees x depth {w.a_depth}" if a else None}}
    for mode, fn in (("resident_chunks", resident_round), ("host_streamed", streamed_round)):
        ex.reset()
        fn()  # warm
        torch.cuda.synchronize()
        ex.reset()
        t0 = time.perf_counter()
        for _ in range(R):
            fn()
        torch.cuda.synchronize()
        dt = (time.perf_counter() - t0) / R
        out[mode] = {"rounds_per_s": 1.0 / dt, "ms_per_round": 1000.0 * dt,
                     "candidates_per_s": w.n / dt,
                     "proposed_last_round": int(num.item())}
        if mode == "host_streamed":
            out[mode]["host_to_device_gbs"] = 4.0 * w.F * w.n / dt / 1e9
        _log(f"{mode}: {1000.0 * dt:.3f} ms per round over {R} rounds")
    out["value"] = out["resident_chunks"]["rounds_per_s"]
    ex.free()
    print(json.dumps(out), flush=True)
    return 0


def _print(out) -> int:
    print(json.dumps(out), flush=True)
    return 0


def out_hbm(w, args, value, ms_per_step, t_val, t_perf, t_topk, n_valid, alg_bytes, fused,
            traffic, copy_gbs):
    """The HBM-bound diagnostic: small ensembles, so reading the pool bounds
    the step.  The roofline object covers the launch that reads every row
    once (4F bytes): with one pass the fused walk, which also writes the mask
    (1 byte) and the score (4 bytes); otherwise the validity walk (mask
    only), with the perf walk's re-read of the accepted rows beside it."""
    if fused:
        f_bytes = (4.0 * w.F + 1.0 + 4.0) * w.n
        achieved = f_bytes / (t_val / 1000.0) / 1e9
        step_gbs = alg_bytes / (ms_per_step / 1000.0) / 1e9
        return {
            "metric": METRIC, "value": value, "unit": "candidates/s", "n_gpus": 1,
            "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_per_step,
            "timing": "median of per-step HIP-event durations on the launch stream",
            "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
            "data": "synthetic (seeded knob + lognormal features, random perfect trees)",
            "config": {"workload": w.name, "diagnostic": "HBM-bound: not a benchmark configuration",
                       "candidates": w.n, "features": w.F,
                       "validity": f"{w.v_trees} trees x depth {w.v_depth}",
                       "perf": f"{w.p_trees} trees x depth {w.p_depth}", "k": w.k, "seed": w.seed,
                       "invalid_fraction": 1 - n_valid / w.n, "one_pass": True},
            "roofline": {
                "bound": "hbm", "kernel": "fused_kernel (V then P on every row, one pass)",
                "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": achieved / HBM_PEAK_GBS, "traffic": traffic,
                "traffic_unit": "bytes per launch (HBM read + write, copy-calibrated rocprofv3 "
                                "counters)",
                "work_per_launch": f"{f_bytes:.4g} bytes ({w.n} rows x {4 * w.F} B + mask + "
                                   "score)",
                "launch_ms": t_val,
                "copy_gbs": copy_gbs, "frac_of_copy": achieved / copy_gbs,
                "step": {"algorithmic_bytes": alg_bytes, "achieved_gbs": step_gbs,
                         "frac": step_gbs / HBM_PEAK_GBS, "frac_of_copy": step_gbs / copy_gbs},
            },
            "hbm_frac": step_gbs / HBM_PEAK_GBS,
            "kernel_ms": {"validity_perf_one_pass": t_val, "topk": t_topk},
            "cpu_baseline": None,
        }
    val_bytes = (4.0 * w.F + 1.0) * w.n
    perf_bytes = 4.0 * w.F * n_valid + 1.0 * w.n + 4.0 * w.n  # accepted rows, mask, scores
    achieved = val_bytes / (t_val / 1000.0) / 1e9
    return {
        "metric": METRIC, "value": value, "unit": "candidates/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_per_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic (seeded knob + lognormal features, random perfect trees)",
        "config": {"workload": w.name, "diagnostic": "HBM-bound: not a benchmark configuration",
                   "candidates": w.n, "features": w.F,
                   "validity": f"{w.v_trees} trees x depth {w.v_depth}",
                   "perf": f"{w.p_trees} trees x depth {w.p_depth}", "k": w.k, "seed": w.seed,
                   "invalid_fraction": 1 - n_valid / w.n},
        "roofline": {
            "bound": "hbm", "kernel": "validity_kernel (reads the pool once)",
            "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBS, "traffic": None,
            "work_per_launch": f"{val_bytes:.4g} bytes ({w.n} rows x {4 * w.F} B + mask)",
            "launch_ms": t_val,
            "copy_gbs": copy_gbs, "frac_of_copy": achieved / copy_gbs,
            "perf_kernel": {"achieved": perf_bytes / (t_perf / 1000.0) / 1e9,
                            "launch_ms": t_perf,
                            "bytes": perf_bytes},
            "step": {"algorithmic_bytes": alg_bytes,
                     "achieved_gbs": alg_bytes / (ms_per_step / 1000.0) / 1e9,
                     "frac": alg_bytes / (ms_per_step / 1000.0) / 1e9 / HBM_PEAK_GBS},
        },
        "hbm_frac": alg_bytes / (ms_per_step / 1000.0) / 1e9 / HBM_PEAK_GBS,
        "kernel_ms": {"validity": t_val, "perf": t_perf, "topk": t_topk},
        "cpu_baseline": None,
    }


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="roofline")
    ap.add_argument("--cpu-rows", type=int, default=1 << 20)
    ap.add_argument("--cpu-rows-one", type=int, default=1 << 17,
                    help="candidates of the single-thread oracle timing")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--copy-probe", action="store_true")
    ap.add_argument("--probe", action="store_true",
                    help="LDS / VALU / walk-loop microbenchmarks instead of the step")
    ap.add_argument("--explore", type=int, default=0, metavar="ROUNDS",
                    help="time ROUNDS explorer rounds (N = --N proposed per round, "
                         "(alpha+1)N held) instead of the scoring step")
    ap.add_argument("--explore-stream", type=int, default=0, metavar="ROUNDS",
                    help="time ROUNDS explorer rounds over the pool streamed in row chunks "
                         "(resident slices and pinned-host copies)")
    ap.add_argument("--chunk-rows", type=int, default=1 << 21)
    ap.add_argument("--graph", action="store_true",
                    help="time the step as a captured HIP graph, replayed once per step")
    ap.add_argument("--two-pass", action="store_true",
                    help="score with the validity walk and then the perf walk even where "
                         "one pass over the pool fits")
    ap.add_argument("--N", type=int, default=10)
    ap.add_argument("--alpha", type=float, default=1.0)
    args = ap.parse_args()

    if args.copy_probe:
        copy_probe()
        return 0
    if args.probe:
        probes()
        return 0
    if args.gpus != 1:
        print(f"bench.py: the scoring path runs on one GPU; --gpus {args.gpus} is not supported "
              "(the pool would shard by rows with one all-gather of the per-GPU top-k lists).",
              file=sys.stderr)
        return 2

    import torch
    import gen
    from paper_2411_10764_amd import ml2

    w = gen.WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    _log(f"workload {w.name}: n={w.n} F={w.F} V={w.v_trees}x{w.v_depth} "
         f"P={w.p_trees}x{w.p_depth} k={w.k}; generating features")
    if args.explore_stream:
        v = ml2.ml2_load_ensemble(w.validity())
        p = ml2.ml2_load_ensemble(w.perf())
        return explore_stream(args, w, v, p, dev)
    t0 = time.perf_counter()
    X = torch.empty((w.n, w.F), dtype=torch.float32, device=dev)
    chunk = 1 << 21
    host = np.empty((chunk, w.F), np.float32)
    for r0 in range(0, w.n, chunk):
        m = min(chunk, w.n - r0)
        gen.features(w.seed, m, w.F, w.K, row0=r0, out=host[:m], missing=w.missing)
        X[r0:r0 + m].copy_(torch.from_numpy(host[:m]))
    torch.cuda.synchronize()
    del host
    _log(f"features resident in HBM ({X.numel() * 4 / 2**30:.2f} GiB) in "
         f"{time.perf_counter() - t0:.1f} s")

    v = ml2.ml2_load_ensemble(w.validity())
    p = ml2.ml2_load_ensemble(w.perf())
    if args.explore:
        return explore(args, w, X, v, p, dev)

    pipe = ml2.Pipeline(v, p, w.n, w.k, device=dev)
    second = w.a_trees > 0
    if second:  # model A re-ranks the k held configurations and keeps w.keep
        a = ml2.ml2_load_ensemble(w.second_level())
        a_scores = torch.empty(w.k, dtype=torch.float32, device=dev)
        a_idx = torch.empty(w.keep, dtype=torch.int32, device=dev)
        a_top = torch.empty(w.keep, dtype=torch.float32, device=dev)
        a_num = torch.empty(1, dtype=torch.int32, device=dev)
        a_wsb = ml2.ml2_rerank_workspace_bytes(a, w.k)
        a_ws = torch.empty(a_wsb, dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream()
    # where both ensembles fit on chip together, ml2_score reads every row
    # once and walks V and P on it (one kernel); otherwise two walks
    fused = ml2.ml2_score_single_pass(v, p, X) and not args.two_pass

    def step(e=None, s=stream):  # s None: the current stream (a graph capture's)
        if e is not None:
            e[0].record(s)
        if fused:
            ml2.ml2_score(v, p, X, pipe.valid, None, pipe.score, s)
            if e is not None:
                e[1].record(s)
        else:
            ml2.ml2_score_validity(v, X, pipe.valid, None, s)
            if e is not None:
                e[1].record(s)
            ml2.ml2_score_perf(p, X, pipe.valid, pipe.score, s)
        if e is not None:
            e[2].record(s)
        ml2.ml2_filter_topk(pipe.valid, pipe.score, w.k, pipe.idx, pipe.top, pipe.num, pipe.ws,
                            pipe.ws_bytes, w.n, s)
        if e is not None:
            e[3].record(s)
        if second:
            ml2.ml2_rerank(a, X, pipe.idx, w.keep, a_scores, a_idx, a_top, a_num, a_ws, a_wsb,
                           m=w.k, stream=s)
        if e is not None:
            e[4].record(s)

    # Pools that fit the 256 MB MALL are flushed before every step (a 512 MB
    # read-modify-write on the same stream, outside the timed events), so
    # that each step reads the pool from HBM.
    flush = None
    if 4.0 * w.F * w.n < MALL_BYTES:
        flush = torch.zeros(2 * MALL_BYTES // 4, dtype=torch.float32, device=dev)

    for _ in range(args.warmup):
        if flush is not None:
            flush.add_(1.0)
        step()
    torch.cuda.synchronize()
    _log(f"warmup done ({args.warmup} steps)")

    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    start = time.perf_counter()
    for s in range(args.steps):
        if flush is not None:
            flush.add_(1.0)
        step(ev[s])
    torch.cuda.synchronize()
    wall = time.perf_counter() - start
    # medians over the timed steps of the HIP-event durations on the stream
    t_val = float(np.median([e[0].elapsed_time(e[1]) for e in ev]))
    t_perf = float(np.median([e[1].elapsed_time(e[2]) for e in ev]))
    t_topk = float(np.median([e[2].elapsed_time(e[3]) for e in ev]))
    t_rerank = float(np.median([e[3].elapsed_time(e[4]) for e in ev]))
    steps_ms = [e[0].elapsed_time(e[4]) for e in ev]
    ms_per_step = float(np.median(steps_ms))
    eager_ms = ms_per_step
    if args.graph:
        # the step captured once as a HIP graph and replayed: the same
        # launches, without the host's per-launch work between them; the
        # kernel split above is that of the eager steps
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            step(None, None)
        torch.cuda.synchronize()
        gev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(args.steps)]
        for s in range(args.steps):
            if flush is not None:
                flush.add_(1.0)
            gev[s][0].record(stream)
            g.replay()
            gev[s][1].record(stream)
        torch.cuda.synchronize()
        ms_per_step = float(np.median([e[0].elapsed_time(e[1]) for e in gev]))
        _log(f"graph replays: {ms_per_step:.3f} ms per step (median of {args.steps}; eager "
             f"{eager_ms:.3f} ms)")
        del g
    valid = pipe.valid.cpu().numpy()
    n_valid = int(valid.sum())
    num = int(pipe.num.item())
    _log(f"step {ms_per_step:.3f} ms (median of {args.steps}; mean {np.mean(steps_ms):.3f}, "
         f"wall {1000.0 * wall / args.steps:.3f}{' with MALL flushes' if flush is not None else ''}):"
         + (f" validity + perf in one pass {t_val:.3f} ms" if fused else
            f" validity {t_val:.3f} ms, perf {t_perf:.3f} ms") + f", top-k {t_topk:.3f} ms"
         + (f", re-rank {t_rerank:.3f} ms (kept {int(a_num.item())})" if second else "")
         + f"; valid {n_valid}/{w.n}, selected {num}")
    del flush

    value = w.n / (ms_per_step / 1000.0)
    launch = ({"launch": "hip_graph", "eager_ms_per_step": eager_ms} if args.graph else {})
    f_vp = w.K if w.visible_only else w.F
    alg_bytes = 4.0 * f_vp * w.n + w.n + 8.0 * w.k
    if second:
        alg_bytes += 4.0 * w.F * w.k + 8.0 * w.keep
    visits_v = w.n * w.v_trees * w.v_depth
    visits_p = n_valid * w.p_trees * w.p_depth
    if w.ragged:  # node visits are the paths' lengths, measured on accepted rows
        sample = np.flatnonzero(valid)[:4096].astype(np.int64)
        per_row = mean_path(w.perf(), w.features(rows=sample))
        visits_p = int(round(n_valid * per_row))
        _log(f"ragged P: {per_row / w.p_trees:.2f} splits per tree on average "
             f"(depth <= {w.p_depth})")
    sha = _kernel_sha()
    if fused:  # one kernel walks V and P on every row
        visits_p = w.n * (w.v_trees * w.v_depth + w.p_trees * w.p_depth)
        t_perf = t_val
    perf_visits_per_s = visits_p / (t_perf / 1000.0)
    traffic = _traffic(sha, w.name)
    copy_gbs = copy_bandwidth(dev)  # HBM fractions are also given against it
    if w.name == "hbm":
        res = out_hbm(w, args, value, ms_per_step, t_val, t_perf, t_topk, n_valid, alg_bytes,
                      fused, traffic if fused else None, copy_gbs)
        res["config"].update(launch)
        return _print(res)
    shape = PERF_WALK_SHAPE.get(w.name)
    loop = walk_loop_ceiling(shape) * 1e12 if shape else None
    vshape = None if fused else VALIDITY_WALK_SHAPE.get(w.name)
    vloop = walk_loop_ceiling(vshape) * 1e12 if vshape else None
    v_visits_per_s = visits_v / (t_val / 1000.0)
    roofline = {
        "bound": "alu",
        "limiter": "lds",
        "kernel": ("fused_kernel (V then P on every row, one pass over the pool)" if fused
                   else "perf_kernel (model P walk over accepted candidates)"),
        "peak_derivation": "node visits on chip (LDS + VALU, no HBM or MFMA term): LDS 256 "
                           "B/clk/CU x 256 CU x 2.4 GHz / 12 B per visit = "
                           f"{VISIT_PEAK_LDS / 1e12:.1f} T/s; VALU 128 lanes/clk/CU x 256 CU x "
                           f"2.4 GHz / {VALU_PER_VISIT} instructions per visit (counted) = "
                           f"{VISIT_PEAK_VALU / 1e12:.1f} T/s; peak = the lower (LDS)",
        "achieved": perf_visits_per_s / 1e12,
        "peak": VISIT_PEAK_PER_S / 1e12,
        "unit": "Tvisit/s",
        "frac": perf_visits_per_s / VISIT_PEAK_PER_S,
        "traffic": traffic,
        "traffic_unit": "bytes per launch (HBM read + write, copy-calibrated rocprofv3 counters)",
        "work_per_launch": (f"{visits_p} node visits ({w.n} rows x ({w.v_trees} + {w.p_trees}) "
                            f"trees x depth {w.p_depth})") if fused else
                           (f"{visits_p} node visits ({n_valid} accepted x {w.p_trees} trees "
                            + (f"x measured mean path)" if w.ragged else f"x depth {w.p_depth})")),
        "launch_ms": t_perf,
        "measured_ceiling": ({"achieved": loop / 1e12,
                              "frac": perf_visits_per_s / loop,
                              "what": "walk loop alone at the perf walk's shape "
                                      f"(depth {shape[0]}, {shape[1]} trees per lane, {shape[2]} "
                                      f"lanes per candidate, {shape[3]} waves, {shape[4]} "
                                      "features; ml2_probe_visit, timed live)"}
                             if loop else None),
        "validity_kernel": (None if fused else
                            {"achieved": v_visits_per_s / 1e12, "launch_ms": t_val,
                             "frac": v_visits_per_s / VISIT_PEAK_PER_S,
                             "measured_ceiling": (
                                 {"achieved": vloop / 1e12, "frac": v_visits_per_s / vloop,
                                  "what": "walk loop alone at the validity walk's shape "
                                          f"(depth {vshape[0]}, {vshape[1]} trees per lane, "
                                          f"{vshape[2]} lanes per candidate, {vshape[3]} waves, "
                                          f"{vshape[4]} features)"} if vloop else None)}),
        "hbm": {"algorithmic_bytes_per_step": alg_bytes,
                "achieved_gbs": alg_bytes / (ms_per_step / 1000.0) / 1e9,
                "peak_gbs": HBM_PEAK_GBS,
                "frac": alg_bytes / (ms_per_step / 1000.0) / 1e9 / HBM_PEAK_GBS,
                "copy_gbs": copy_gbs,
                "frac_of_copy": alg_bytes / (ms_per_step / 1000.0) / 1e9 / copy_gbs},
    }
    out = {
        "metric": METRIC, "value": value, "unit": "candidates/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_per_step,
        "timing": "median of per-step HIP-event durations on the launch stream"
                  + (", MALL flushed before each step" if 4.0 * w.F * w.n < MALL_BYTES else ""),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic (seeded knob + lognormal features, random perfect trees)",
        "config": {"workload": w.name, "candidates": w.n, "features": w.F,
                   "knob_features": w.K, "validity": f"{w.v_trees} trees x depth {w.v_depth}",
                   "perf": f"{w.p_trees} trees x depth {'<= ' if w.ragged else ''}{w.p_depth}"
                           + (" (ragged, default directions)" if w.ragged else ""),
                   "k": w.k, "missing_hidden_fraction": w.missing,
                   "seed": w.seed, "invalid_fraction": 1 - n_valid / w.n, **launch},
        **({"second_level": {"model_a": f"{w.a_trees} trees x depth {w.a_depth} over {w.F} "
                                        f"features", "keep": w.keep,
                             "validity_perf_features": f_vp}} if second else {}),
        "roofline": roofline,
        "hbm_frac": roofline["hbm"]["frac"],
        "kernel_ms": {**({"validity_perf_one_pass": t_val} if fused else
                         {"validity": t_val, "perf": t_perf}), "topk": t_topk,
                      **({"rerank": t_rerank} if second else {})},
    }
    del X
    torch.cuda.empty_cache()
    if not args.no_cpu:
        _log(f"cpu baseline: oracle on {args.cpu_rows} candidates")
        out["cpu_baseline"] = cpu_baseline(w, args.cpu_rows, args.cpu_rows_one)
    else:
        out["cpu_baseline"] = None
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
