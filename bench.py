#!/usr/bin/env python3
"""Benchmark of the W4A16 GEMM on one MI355X.

Workload: the Llama-7B attention-projection layer, K = N = 4096, group size
128, synthetic seeded data (``synth`` workload 1), with the batch sweep
M = 1, 2, 4, 8, 16, 32, 64, 128.  One step = one GEMM at every M of the
sweep (8 launches), each on the next of >= 1 GiB of packed weight copies so
the 256 MB Infinity Cache never serves the weights.  Packing is offline and
not timed.  Launches are replayed from HIP graphs (one graph per step, 16
graphs rotating the weight copies) so the host does not throttle
microsecond kernels.

Output: one JSON line.  ``value`` = TFLOP/s of the whole timed region
(sum of 2MNK over the launches / elapsed).  Also reported per M: time per
call, TFLOP/s, effective weight-stream GB/s, fraction of the MI355X roofline
(t_roof / t), and the speedup over a plain fp16 ``torch.matmul`` of the same
shape timed the same way in the same run (comparison only).  ``roofline``
covers the GEMM kernel: algorithmic bytes of the timed launches / elapsed
(HIP events on the launch stream) against 8 TB/s.  ``cpu_baseline`` times
the fp64 oracle on the host over the whole sweep (and checks the GPU
outputs against it).  Two further sections are reported beside the step,
outside its timed region: ``sparse_2of4`` (the 2:4 sparse kernel, K = N =
8192, M sweep), ``prefill`` (M = 256, 1024, 4096 in one launch per call,
against the fp16 matrix-core peak and fp16 ``torch.matmul``) and
``quantize`` (the weight quantiser, against the fp32 vector lane rate).

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline]
       [--no-sparse | --sparse-only] [--no-prefill | --prefill-only]
       [--no-quantize | --quantize-only]
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

K_DIM, N_DIM, GROUP = 4096, 4096, 128
M_SWEEP = [1, 2, 4, 8, 16, 32, 64, 128]
WID = 1
ROTATION_BYTES = 1 << 30  # >= 1 GiB of weight copies (Infinity Cache is 256 MB)
GRAPHS = 16
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "w4a16_gemm_4096x4096_msweep_traffic.json")


def log(msg):
    print("[bench] " + msg, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--per-m-reps", type=int, default=10)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-fp16", action="store_true")
    ap.add_argument("--no-sparse", action="store_true",
                    help="skip the 2:4 sparse section (K = N = 8192, g = 128, M sweep)")
    ap.add_argument("--sparse-only", action="store_true",
                    help="run only the 2:4 sparse section and print its JSON (for profiling it alone)")
    ap.add_argument("--no-prefill", action="store_true",
                    help="skip the large-batch section (M = 256, 1024, 4096 in one launch)")
    ap.add_argument("--prefill-only", action="store_true",
                    help="run only the large-batch section and print its JSON (for profiling it alone)")
    ap.add_argument("--no-quantize", action="store_true",
                    help="skip the quantiser section")
    ap.add_argument("--quantize-only", action="store_true",
                    help="run only the quantiser section and print its JSON (for profiling it alone)")
    ap.add_argument("--calibration-copy-mb", type=int, default=0,
                    help="run plain device-to-device copies of this many MB (outside the timed "
                         "region) so hardware byte counters can be scaled against a known size")
    return ap.parse_args()


def measured_traffic():
    """HBM bytes per launch from the committed counter summary, or None when
    the kernel source has changed since the counters were taken."""
    from paper_2408_11743_amd.profile_summary import kernel_sources_digest
    try:
        rec = json.load(open(TRAFFIC_FILE))
        if kernel_sources_digest() != rec["kernel_sources_sha256"]:
            return None
        return rec["step_avg_hbm_bytes_per_launch"]
    except (OSError, KeyError, ValueError):
        return None


SPARSE_K, SPARSE_N, SPARSE_WID = 8192, 8192, 4
# large batches: (K, N, synth workload) and the batch sizes
PREFILL_SHAPES = [(4096, 4096, 1), (28672, 8192, 3)]
PREFILL_M = [256, 1024, 4096]


def cpu_threads() -> int:
    return int(os.environ.get("OMP_NUM_THREADS", "0")) or len(os.sched_getaffinity(0))


def graph_time_us(launch, count, stream, reps, torch, np):
    """Median per-launch time of a graph of `count` launches (launch(i))."""
    gr = torch.cuda.CUDAGraph()
    with torch.cuda.stream(stream):
        launch(0)
        stream.synchronize()
        with torch.cuda.graph(gr, stream=stream):
            for i in range(count):
                launch(i)
        # replays for >= 30 ms first: clocks ramp up after host-side pauses
        t_end = time.perf_counter() + 0.03
        while True:
            gr.replay()
            torch.cuda.synchronize()
            if time.perf_counter() >= t_end:
                break
        times = []
        for _ in range(reps):
            a0 = torch.cuda.Event(enable_timing=True)
            a1 = torch.cuda.Event(enable_timing=True)
            a0.record(stream)
            gr.replay()
            a1.record(stream)
            a1.synchronize()
            times.append(a0.elapsed_time(a1) * 1e3 / count)
    del gr
    return float(np.median(times))


def sparse_section(args, mk, R, synth, torch, np, dev):
    """The 2:4 sparse workload (Section 4): K = N = 8192, g = 128, M sweep;
    per M the sparse kernel, the dense W4A16 kernel on the same matrix and
    fp16 torch.matmul on it, each over >= 1 GiB of rotated weight copies."""
    K, N, g = SPARSE_K, SPARSE_N, GROUP
    q, keep, s = synth.sparse24_weights(SPARSE_WID, K, N, g)
    qd, sd = torch.from_numpy(q).to(dev), torch.from_numpy(s).to(dev)
    L = mk.lib()
    copies = {}
    for sp_flag in (True, False):
        wp, sp = mk.pack(qd, sd, group=g, sparse=sp_flag)
        n = max(2, math.ceil(ROTATION_BYTES / (wp.numel() + 2 * sp.numel())))
        copies[sp_flag] = ([wp] + [wp.clone() for _ in range(n - 1)], sp)
    w16s, n16 = [], 0
    if not args.no_fp16:
        w16 = ((qd.to(torch.float32) - 8.0) * sd.to(torch.float32).repeat_interleave(g, dim=0)).to(torch.float16)
        n16 = max(2, math.ceil(ROTATION_BYTES / (w16.numel() * 2)))
        w16s = [w16] + [w16.clone() for _ in range(n16 - 1)]
        del w16
    ws = mk.Workspace(dev)
    wsbuf = ws.ensure(max(mk.marlin_workspace_bytes(M, N, K, g) for M in M_SWEEP))
    stream = torch.cuda.Stream(device=dev)
    rows = []
    for M in M_SWEEP:
        A = torch.from_numpy(synth.activations(SPARSE_WID, M, K)).to(dev)
        C = torch.empty((M, N), dtype=torch.float16, device=dev)
        t = {}
        for sp_flag in (True, False):
            wps, sp = copies[sp_flag]
            fn = L.marlin_gemm_sparse if sp_flag else L.marlin_gemm

            def launch(i, wps=wps, sp=sp, fn=fn):
                st = fn(A.data_ptr(), wps[i % len(wps)].data_ptr(), sp.data_ptr(), C.data_ptr(),
                        wsbuf.data_ptr(), wsbuf.numel(), M, N, K, g, stream.cuda_stream)
                if st != 0:
                    raise mk.MarlinError("marlin_gemm_sparse" if sp_flag else "marlin_gemm", st)
            t[sp_flag] = graph_time_us(launch, len(wps), stream, args.per_m_reps, torch, np)
        t16 = None
        if not args.no_fp16:
            t16 = graph_time_us(lambda i: torch.matmul(A, w16s[i % n16]), n16, stream, args.per_m_reps, torch, np)
        troof = R.sparse24_t_roof(M, N, K, g) * 1e6
        rec = {"M": M, "us": round(t[True], 3), "dense_w4_us": round(t[False], 3),
               "speedup_vs_dense_w4": round(t[False] / t[True], 3),
               "roof_us": round(troof, 3), "roof_frac": round(troof / t[True], 4),
               "launch": mk.marlin_describe_sparse(M, N, K, g)}
        if t16 is not None:
            rec["fp16_us"] = round(t16, 3)
            rec["speedup_vs_fp16"] = round(t16 / t[True], 3)
        rows.append(rec)
        log("sparse 2:4 %dx%d M=%3d: %.3f us (dense W4 %.3f us, fp16 %s us), roofline frac %.3f" %
            (K, N, M, t[True], t[False], "%.3f" % t16 if t16 else "-", troof / t[True]))
    del copies, w16s
    cpu = None
    if not args.no_cpu_baseline:
        # the fp64 oracle over the whole sweep (the sparse product is the dense
        # definition on the pruned matrix)
        import oracle
        tot, flops = 0.0, 0.0
        for M in M_SWEEP:
            A_np = synth.activations(SPARSE_WID, M, K)
            c0 = time.perf_counter()
            oracle.gemm(A_np, q, s, g)
            tot += time.perf_counter() - c0
            flops += R.flops(M, N, K)
        cpu = {"value": round(flops / tot / 1e12, 6), "unit": "TFLOP/s", "cores": cpu_threads(),
               "kind": "oracle", "seconds": round(tot, 3), "sample": "the whole M sweep, one run per M"}
        log("sparse oracle: %.2f s for the sweep" % tot)
    return {"workload": "2:4 sparse W4A16 GEMM, K=%d N=%d g=%d, M sweep %s" % (K, N, g, M_SWEEP),
            "bound": "hbm", "per_m": rows, "cpu_baseline": cpu}


def prefill_section(args, mk, R, synth, torch, np, dev):
    """Large batches in one launch (Section 3.4, Striped Partitioning, on
    batches well above 64): the Llama-7B attention projection and the
    70B-class MLP down projection at M = 256, 1024, 4096, g = 128, against
    fp16 torch.matmul on the dequantized matrix.  MFMA-bound: the roofline is
    the fp16 matrix-core peak.  Two weight copies alternate (at these M the
    weights are a small part of the traffic)."""
    L = mk.lib()
    stream = torch.cuda.Stream(device=dev)
    ws = mk.Workspace(dev)
    rows, cpu_rows = [], []
    for (K, N, wid) in PREFILL_SHAPES:
        g = GROUP
        q, s = synth.weights(wid, K, N, g)
        qd, sd = torch.from_numpy(q).to(dev), torch.from_numpy(s).to(dev)
        wp, sp = mk.pack(qd, sd, group=g)
        wps = [wp, wp.clone()]
        w16 = None
        if not args.no_fp16:
            w16 = ((qd.to(torch.float32) - 8.0) * sd.to(torch.float32).repeat_interleave(g, dim=0)).to(torch.float16)
        del qd, sd
        wsbuf = ws.ensure(max(mk.marlin_workspace_bytes(M, N, K, g) for M in PREFILL_M))
        for M in PREFILL_M:
            A = torch.from_numpy(synth.activations(wid, M, K)).to(dev)
            C = torch.empty((M, N), dtype=torch.float16, device=dev)

            def launch(i, M=M, A=A, C=C):
                st = L.marlin_gemm(A.data_ptr(), wps[i % 2].data_ptr(), sp.data_ptr(), C.data_ptr(),
                                   wsbuf.data_ptr(), wsbuf.numel(), M, N, K, g, stream.cuda_stream)
                if st != 0:
                    raise mk.MarlinError("marlin_gemm", st)
            t = graph_time_us(launch, 4, stream, args.per_m_reps, torch, np)
            rec = {"K": K, "N": N, "M": M, "us": round(t, 2),
                   "TFLOPs": round(R.flops(M, N, K) / t / 1e6, 1),
                   "mfma_frac": round(R.flops(M, N, K) / (t * 1e-6) / R.FP16_MFMA_FLOPS, 4),
                   "launch": mk.marlin_describe(M, N, K, g)}
            if w16 is not None:
                t16 = graph_time_us(lambda i: torch.matmul(A, w16), 4, stream, args.per_m_reps, torch, np)
                rec["fp16_us"] = round(t16, 2)
                rec["speedup_vs_fp16"] = round(t16 / t, 3)
            rows.append(rec)
            log("prefill %dx%d M=%4d: %.1f us, %.0f TFLOP/s (%.1f%% of the MFMA peak), fp16 %s us" %
                (K, N, M, t, rec["TFLOPs"], 100 * rec["mfma_frac"], rec.get("fp16_us", "-")))
            del A, C
        del wps, wp, sp, w16
        if not args.no_cpu_baseline:
            # the fp64 oracle at the smallest batch of the section, in full
            import oracle
            M = PREFILL_M[0]
            A_np = synth.activations(wid, M, K)
            c0 = time.perf_counter()
            oracle.gemm(A_np, q, s, g)
            dt = time.perf_counter() - c0
            cpu_rows.append({"K": K, "N": N, "M": M, "value": round(R.flops(M, N, K) / dt / 1e12, 6),
                             "seconds": round(dt, 3), "sample": "all %d x %d outputs" % (M, N)})
            log("prefill oracle %dx%d M=%d: %.2f s" % (K, N, M, dt))
    cpu = None
    if cpu_rows:
        cpu = {"unit": "TFLOP/s", "cores": cpu_threads(), "kind": "oracle", "per_shape": cpu_rows}
    return {"workload": "W4A16 GEMM, one launch per call, g=%d, (K, N) in %s, M in %s" %
                        (GROUP, [sh[:2] for sh in PREFILL_SHAPES], PREFILL_M),
            "bound": "mfma", "peak_TFLOPs": R.FP16_MFMA_FLOPS / 1e12, "per_m": rows, "cpu_baseline": cpu}


def quantize_section(args, mk, R, synth, torch, np, dev):
    """The quantiser (symmetric, zero point 8, g = 128, clipping search over
    the 10 default ratios) on the Llama-7B attention projection and the
    70B-class MLP down projection.  Bound by fp32 vector work (~75 operations
    per weight against 3 bytes of HBM traffic): ``alu_frac`` against the fp32
    vector lane rate, ``hbm_GBps`` for reference."""
    L = mk.lib()
    stream = torch.cuda.Stream(device=dev)
    ratios = list(mk.CLIP_RATIOS)
    rows, cpu_rows = [], []
    for (K, N, wid) in PREFILL_SHAPES:
        g = GROUP
        W = torch.from_numpy(synth.fp16_weights(wid, K, N)).to(dev)
        q = torch.empty((K, N), dtype=torch.uint8, device=dev)
        s = torch.empty((K // g, N), dtype=torch.float16, device=dev)

        def launch(i):
            mk.marlin_quantize(W, K, N, g, ratios, q, s, stream)
        t = graph_time_us(launch, 2, stream, args.per_m_reps, torch, np)
        ops = R.quant_ops(K, N, len(ratios))
        rec = {"K": K, "N": N, "group": g, "ratios": len(ratios), "us": round(t, 2),
               "Gweights_per_s": round(K * N / t / 1e3, 2),
               "alu_frac": round(ops / (t * 1e-6) / R.FP32_LANE_OPS, 4),
               "hbm_GBps": round(R.quant_bytes(K, N, g) / t / 1e3, 1)}
        rows.append(rec)
        log("quantize %dx%d g=%d, %d ratios: %.1f us, %.2f G weights/s, %.1f%% of the fp32 lane rate" %
            (K, N, g, len(ratios), t, rec["Gweights_per_s"], 100 * rec["alu_frac"]))
        if not args.no_cpu_baseline:
            # the quantiser's oracle (numpy, fp32) on all columns, or on the
            # first 1024 where that takes too long (columns are independent)
            from oracle import quant as oq
            cols = N if K * N <= 4096 * 4096 else 1024
            W_np = np.ascontiguousarray(W[:, :cols].cpu().numpy())
            c0 = time.perf_counter()
            oq.quantize(W_np, g, ratios)
            dt = time.perf_counter() - c0
            cpu_rows.append({"K": K, "N": N, "value": round(K * cols / dt / 1e9, 6), "unit": "G weights/s",
                             "seconds": round(dt, 3), "sample": "%d of %d columns" % (cols, N)})
            log("quantize oracle %dx%d: %.2f s for %d columns" % (K, N, dt, cols))
        del W, q, s
    cpu = None
    if cpu_rows:
        cpu = {"unit": "G weights/s", "cores": cpu_threads(), "kind": "oracle", "per_shape": cpu_rows}
    return {"workload": "quantiser fp16 -> (q, s), g=%d, %d clipping ratios, (K, N) in %s" %
                        (GROUP, len(mk.CLIP_RATIOS), [sh[:2] for sh in PREFILL_SHAPES]),
            "bound": "alu", "peak_lane_ops_per_s": R.FP32_LANE_OPS, "per_shape": rows, "cpu_baseline": cpu}


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(the GEMM would shard by columns, or by rows with an RCCL "
              "all-reduce of C). Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2408_11743_amd as mk
    import synth
    from paper_2408_11743_amd import roofline as R

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    dev = torch.device("cuda", 0)
    mk.lib()
    if args.calibration_copy_mb:
        nb = args.calibration_copy_mb << 20
        src = torch.ones(nb // 4, dtype=torch.int32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        log("calibration: 3 device copies of %d MiB" % args.calibration_copy_mb)
        del src, dst
    if args.sparse_only:
        print(json.dumps({"sparse_2of4": sparse_section(args, mk, R, synth, torch, np, dev)}), flush=True)
        return
    if args.prefill_only:
        print(json.dumps({"prefill": prefill_section(args, mk, R, synth, torch, np, dev)}), flush=True)
        return
    if args.quantize_only:
        print(json.dumps({"quantize": quantize_section(args, mk, R, synth, torch, np, dev)}), flush=True)
        return
    K, N, g = K_DIM, N_DIM, GROUP

    # ---- weights: pack once, replicate to >= 1 GiB ----
    q, s = synth.weights(WID, K, N, g)
    wp0, sp0 = mk.pack(torch.from_numpy(q).to(dev), torch.from_numpy(s).to(dev), group=g)
    wbytes = wp0.numel() + sp0.numel() * 2
    nrot = 8 * math.ceil(ROTATION_BYTES / wbytes / 8)
    wps = [wp0] + [wp0.clone() for _ in range(nrot - 1)]
    sps = [sp0] + [sp0.clone() for _ in range(nrot - 1)]
    log("weights %dx%d g=%d: %d B packed per copy, %d copies (%.2f GB)" %
        (K, N, g, wbytes, nrot, nrot * wbytes / 1e9))


    acts = {M: torch.from_numpy(synth.activations(WID, M, K)).to(dev) for M in M_SWEEP}
    outs = {M: torch.empty((M, N), dtype=torch.float16, device=dev) for M in M_SWEEP}
    ws = mk.Workspace(dev)
    wsb = max(mk.marlin_workspace_bytes(M, N, K, g) for M in M_SWEEP)
    wsbuf = ws.ensure(wsb)
    L = mk.lib()

    def launch(M, i, stream):
        st = L.marlin_gemm(acts[M].data_ptr(), wps[i].data_ptr(), sps[i].data_ptr(),
                           outs[M].data_ptr(), wsbuf.data_ptr(), wsbuf.numel(), M, N, K, g,
                           stream.cuda_stream)
        if st != 0:
            raise mk.MarlinError("marlin_gemm", st)

    # ---- graphs: one step (the M sweep) per graph, 16 graphs rotating copies ----
    stream = torch.cuda.Stream(device=dev)
    torch.cuda.synchronize()
    graphs = []
    with torch.cuda.stream(stream):
        for i, M in enumerate(M_SWEEP):  # eager warm-up of every variant
            launch(M, i % nrot, stream)
        stream.synchronize()
        for gi in range(GRAPHS):
            gr = torch.cuda.CUDAGraph()
            with torch.cuda.graph(gr, stream=stream):
                for j, M in enumerate(M_SWEEP):
                    launch(M, (gi * len(M_SWEEP) + j) % nrot, stream)
            graphs.append(gr)
    torch.cuda.synchronize()
    log("captured %d graphs of %d launches" % (GRAPHS, len(M_SWEEP)))

    step_flops = sum(R.flops(M, N, K) for M in M_SWEEP)
    step_bytes = sum(R.w4a16_bytes(M, N, K, g) for M in M_SWEEP)
    step_wbytes = len(M_SWEEP) * R.weight_bytes(N, K, g)

    # ---- warm-up and timed region ----
    with torch.cuda.stream(stream):
        for k in range(args.warmup):
            graphs[k % GRAPHS].replay()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    with torch.cuda.stream(stream):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        e0.record(stream)
        for k in range(args.steps):
            graphs[k % GRAPHS].replay()
        e1.record(stream)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
    ev_ms = e0.elapsed_time(e1)
    wall_ms = (t1 - t0) * 1e3
    ms_per_step = ev_ms / args.steps
    value = step_flops / (ms_per_step * 1e-3) / 1e12
    log("timed %d steps: %.3f ms/step (events), wall %.3f ms/step" %
        (args.steps, ms_per_step, wall_ms / args.steps))
    avg_launch_us = ms_per_step * 1e3 / len(M_SWEEP)
    achieved_gbs = step_bytes / (ms_per_step * 1e-3) / 1e9

    # ---- per-M: graph of nrot launches (one per weight copy) ----
    per_m = []
    for M in M_SWEEP:
        gr = torch.cuda.CUDAGraph()
        with torch.cuda.stream(stream):
            with torch.cuda.graph(gr, stream=stream):
                for i in range(nrot):
                    launch(M, i, stream)
            gr.replay()
            torch.cuda.synchronize()
            times = []
            for _ in range(args.per_m_reps):
                a0 = torch.cuda.Event(enable_timing=True)
                a1 = torch.cuda.Event(enable_timing=True)
                a0.record(stream)
                gr.replay()
                a1.record(stream)
                a1.synchronize()
                times.append(a0.elapsed_time(a1) * 1e3 / nrot)
        del gr
        t_us = float(np.median(times))
        troof = R.w4a16_t_roof(M, N, K, g) * 1e6
        per_m.append({
            "M": M, "us": round(t_us, 3), "us_min": round(min(times), 3),
            "tflops": round(R.flops(M, N, K) / (t_us * 1e-6) / 1e12, 3),
            "weight_GBps": round(R.weight_bytes(N, K, g) / (t_us * 1e-6) / 1e9, 1),
            "roof_us": round(troof, 3), "roof_frac": round(troof / t_us, 4),
            "bound": R.bound(M, N, K, g),
            "launch": mk.marlin_describe(M, N, K, g),
        })
        log("M=%3d: %.3f us/call  %.1f weight GB/s  roofline frac %.3f" %
            (M, t_us, per_m[-1]["weight_GBps"], troof / t_us))

    # ---- fp16 comparator: torch.matmul with rotated fp16 weights ----
    if not args.no_fp16:
        w16 = torch.from_numpy((s.astype(np.float32).repeat(g, axis=0) *
                                (q.astype(np.float32) - 8)).astype(np.float16)).to(dev)
        nrot16 = max(2, math.ceil(ROTATION_BYTES / (w16.numel() * 2)))
        w16s = [w16] + [w16.clone() for _ in range(nrot16 - 1)]
        for rec in per_m:
            M = rec["M"]
            A = acts[M]
            eager = torch.matmul(A, w16s[0])
            torch.cuda.synchronize()
            gr = torch.cuda.CUDAGraph()
            c16 = [None] * nrot16
            with torch.cuda.stream(stream):
                torch.matmul(A, w16s[0])
                stream.synchronize()
                with torch.cuda.graph(gr, stream=stream):
                    for i in range(nrot16):
                        c16[i] = torch.matmul(A, w16s[i])
                gr.replay()
                torch.cuda.synchronize()
                same = bool(torch.equal(c16[0], eager))
                times = []
                for _ in range(args.per_m_reps):
                    a0 = torch.cuda.Event(enable_timing=True)
                    a1 = torch.cuda.Event(enable_timing=True)
                    a0.record(stream)
                    gr.replay()
                    a1.record(stream)
                    a1.synchronize()
                    times.append(a0.elapsed_time(a1) * 1e3 / nrot16)
            del gr, c16
            t16 = float(np.median(times))
            rec["fp16_us"] = round(t16, 3)
            rec["speedup_vs_fp16"] = round(t16 / rec["us"], 3)
            rec["fp16_graph_matches_eager"] = same
            log("M=%3d: fp16 matmul %.3f us/call -> speedup %.2fx" % (M, t16, t16 / rec["us"]))
        del w16s, w16

    # ---- CPU baseline: the fp64 oracle over the same sweep (also a parity check) ----
    cpu = None
    parity = None
    if not args.no_cpu_baseline:
        import oracle
        threads = cpu_threads()
        tot = 0.0
        worst = 0.0
        ok = True
        for M in M_SWEEP:
            A_np = acts[M].cpu().numpy()
            runs = []
            for _ in range(3):
                c0 = time.perf_counter()
                ref = oracle.gemm(A_np, q, s, g)
                runs.append(time.perf_counter() - c0)
            tot += float(np.median(runs))
            launch(M, 0, torch.cuda.current_stream())
            torch.cuda.synchronize()
            got = outs[M].cpu().numpy().astype(np.float64)
            err = np.abs(got - ref)
            ok &= bool((err <= 2e-3 + 1e-2 * np.abs(ref)).all())
            worst = max(worst, float(err.max()))
        cpu = {"value": round(step_flops / tot / 1e12, 6), "unit": "TFLOP/s", "cores": threads,
               "kind": "oracle", "seconds": round(tot, 3),
               "sample": "the whole step (fp64 oracle at every M of the sweep, 4096x4096 g=128), "
                         "median of 3 runs per M"}
        parity = {"ok": ok, "max_abs_err": worst}
        log("oracle: %.2f s for one step on %d threads; GPU parity %s (max err %.3g)" %
            (tot, threads, ok, worst))

    sparse = None if args.no_sparse else sparse_section(args, mk, R, synth, torch, np, dev)
    prefill = None if args.no_prefill else prefill_section(args, mk, R, synth, torch, np, dev)
    quant = None if args.no_quantize else quantize_section(args, mk, R, synth, torch, np, dev)

    small = [r for r in per_m if r["M"] <= 16]
    out = {
        "metric": "W4A16 GEMM TFLOP/s & weight GB/s vs roofline, M=1..128; speedup vs fp16 GEMM",
        "value": round(value, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16",
        "data": "synthetic",
        "config": {"workload": "Llama-7B attention projection W4A16 GEMM, K=4096 N=4096 g=128, "
                               "M sweep 1..128, weights rotated over %.2f GB" % (nrot * wbytes / 1e9),
                   "K": K, "N": N, "group": g, "M": M_SWEEP, "weight_copies": nrot,
                   "launches_per_step": len(M_SWEEP)},
        "weight_GBps": round(step_wbytes / (ms_per_step * 1e-3) / 1e9, 1),
        "roofline": {"bound": "hbm", "achieved": round(achieved_gbs, 1),
                     "peak": R.HBM_BYTES_PER_S / 1e9, "unit": "GB/s",
                     "frac": round(achieved_gbs * 1e9 / R.HBM_BYTES_PER_S, 4),
                     "traffic": measured_traffic(),
                     "traffic_unit": "HBM bytes per launch (step average)",
                     "algorithmic_bytes_per_launch": round(step_bytes / len(M_SWEEP)),
                     "avg_launch_us": round(avg_launch_us, 3),
                     "kernel": "w4a16_stream_kernel"},
        "roof_frac_step": round(sum(R.w4a16_t_roof(M, N, K, g) for M in M_SWEEP) /
                                (ms_per_step * 1e-3), 4),
        "min_roof_frac_M_le_16": min(r["roof_frac"] for r in small),
        "per_m": per_m,
        "wall_ms_per_step": round(wall_ms / args.steps, 6),
        "cpu_baseline": cpu,
        "parity": parity,
        "sparse_2of4": sparse,
        "prefill": prefill,
        "quantize": quant,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
