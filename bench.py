#!/usr/bin/env python3
"""Benchmark of the W4A16 GEMM on one MI355X.

Headline workload: the 70B-class layers, (K, N) = (8192, 28672) and
(28672, 8192), group size 128, synthetic seeded data (``synth`` workload 3),
batch sweep M = 1, 2, 4, 8, 16, 32, 64, 128.  One step = one GEMM at every
(layer, M) of the sweep (16 launches), each on the next of 9 packed-weight
copies per layer (1.09 GB per layer, beyond the 256 MB Infinity Cache).
Packing is offline and not timed.  Launches are replayed from HIP graphs (one
graph per step, 9 graphs rotating the weight copies) so the host does not
throttle microsecond kernels.  Before the W warm-up steps, the step graphs are
replayed for 0.15 s (untimed) so that the shader clock has ramped up: a
timed region of 20 steps lasts only about 11 ms.

Output: one JSON line.  ``value`` = TFLOP/s of the whole timed region (sum of
2MNK over the launches / elapsed).  Per (layer, M) of the headline: time per
call (graph replays over the rotated copies), the eager single-call latency
(event-timed, and the host time of the call itself), TFLOP/s, effective
weight-stream GB/s, the fraction of the MI355X roofline (t_roof / t), the
launch configuration, and the speedup over a plain fp16 ``torch.matmul`` of
the same shape timed the same way in the same run (comparison only).
``roofline`` covers the step's GEMM launches: algorithmic bytes / elapsed
(HIP events on the launch stream) against 8 TB/s.  ``cpu_baseline`` times
the fp64 oracle on the host at M = 1, 16, 128 on both layers (and checks the
GPU outputs against it), plus one single-thread run.  ``clock`` records the
shader clock sampled during the run.

Sections beside the step, outside its timed region: ``attention_4096`` (the
Llama-7B attention projection, 4096 x 4096), ``mlp_7b`` (the Llama-7B MLP
layers, g = 128 and per-channel scales), ``sparse_2of4`` (the 2:4 sparse
kernel, 8192 x 8192), ``prefill`` (M = 256, 1024, 4096 in one launch per
call) and ``quantize`` (the weight quantiser).

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline]
       [--no-sections] [--no-clock] [--only SECTION] [--profile-cases C
       [--profile-layers headline|attention_4096|mlp_7b]]

Under a profiler, run with --no-clock --no-cpu-baseline (or --only /
--profile-cases): those start no child process.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import subprocess
import sys
import threading
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

GROUP = 128
M_SWEEP = [1, 2, 4, 8, 16, 32, 64, 128]
# (K, N, synth workload id, group); group -1 = one scale per output column
HEADLINE = [(8192, 28672, 3, 128), (28672, 8192, 3, 128)]
ATTENTION = [(4096, 4096, 1, 128)]
MLP_7B = [(4096, 11008, 2, 128), (11008, 4096, 2, 128), (4096, 11008, 2, -1), (11008, 4096, 2, -1)]
ROTATION_BYTES = 1 << 30  # >= 1 GiB of weight copies per layer (Infinity Cache is 256 MB)
CPU_MS = [1, 16, 64, 128]
RAMP_S = 0.15  # untimed step replays before the warm-up steps (clock ramp)
CLOCK_S = 4.0  # untimed step replays after the timed region, while the shader clock is read
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "w4a16_gemm_70b_layers_msweep_traffic.json")
SECTIONS = ("attention_4096", "mlp_7b", "sparse_2of4", "prefill", "quantize")

SPARSE_K, SPARSE_N, SPARSE_WID = 8192, 8192, 4
# large batches: (K, N, synth workload) and the batch sizes
PREFILL_SHAPES = [(4096, 4096, 1), (28672, 8192, 3)]
PREFILL_M = [256, 1024, 4096]


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
    ap.add_argument("--no-sections", action="store_true", help="the headline step only")
    ap.add_argument("--no-clock", action="store_true",
                    help="do not sample the shader clock (no child process: for runs under a profiler)")
    ap.add_argument("--only", choices=SECTIONS,
                    help="run only this section and print its JSON (for profiling it alone)")
    ap.add_argument("--profile-cases", type=int, default=0,
                    help="counter runs: launch every (layer, M) case of --profile-layers this many times "
                         "eagerly, in sweep order, print the case list and stop")
    ap.add_argument("--profile-layers", choices=("headline", "attention_4096", "mlp_7b", "sparse_2of4"),
                    default="headline")
    ap.add_argument("--calibration-copy-mb", type=int, default=0,
                    help="run plain device-to-device copies of this many MB first, so hardware byte "
                         "counters can be scaled against a known size")
    return ap.parse_args()


def measured_traffic():
    """HBM bytes per launch (step average) from the committed counter summary,
    or None when the kernel sources have changed since the counters were taken."""
    from paper_2408_11743_amd.profile_summary import kernel_sources_digest
    try:
        rec = json.load(open(TRAFFIC_FILE))
        if kernel_sources_digest() != rec["kernel_sources_sha256"]:
            return None
        return rec["step_avg_hbm_bytes_per_launch"]
    except (OSError, KeyError, ValueError):
        return None


def cpu_threads() -> int:
    return int(os.environ.get("OMP_NUM_THREADS", "0")) or len(os.sched_getaffinity(0))


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


class Range:
    """A named range in the profiler's marker trace (roctx), closed after the
    GPU work inside it has finished, so the kernels it covers lie within it."""

    def __init__(self, torch, name):
        self.torch, self.name = torch, name

    def __enter__(self):
        self.torch.cuda.synchronize()
        self.torch.cuda.nvtx.range_push(self.name)

    def __exit__(self, *exc):
        self.torch.cuda.synchronize()
        self.torch.cuda.nvtx.range_pop()


# ---------------- shader clock ----------------

# The sampler runs as a child process started before this process touches
# the GPU (a process that has initialised the GPU starts no other program):
# it appends one JSON line per amd-smi reading (wall time, shader clocks in
# MHz, or the error) to a file until a stop file appears.
_SAMPLER = r"""
import json, os, subprocess, sys, time
out, stop = sys.argv[1], sys.argv[2]

def clocks(obj, path=""):
    found = []
    if isinstance(obj, dict):
        for k, v in obj.items():
            p = (path + "/" + str(k)).lower()
            if isinstance(v, dict) and "value" in v and str(k).lower() in ("clk", "cur_clk") \
                    and ("gfx" in path.lower() or "sclk" in path.lower()):
                try:
                    found.append(float(v["value"]))
                except (TypeError, ValueError):
                    pass
            else:
                found += clocks(v, p)
    elif isinstance(obj, list):
        for i, v in enumerate(obj):
            found += clocks(v, path + "/%d" % i)
    return found

t_end = time.time() + 900
parent = os.getppid()
with open(out, "a") as f:
    while not os.path.exists(stop) and time.time() < t_end and os.getppid() == parent:
        rec = {"t": time.time()}
        try:
            r = subprocess.run(["amd-smi", "metric", "-g", "0", "-c", "--json"], capture_output=True,
                               text=True, timeout=20)
            rec["mhz"] = clocks(json.loads(r.stdout))
        except Exception as e:
            rec["error"] = "%s: %s" % (type(e).__name__, str(e)[:200])
        f.write(json.dumps(rec) + "\n")
        f.flush()
        time.sleep(1.0)
"""


class ClockSampler:
    """The shader clock, read with amd-smi about once a second by a child
    process started before the GPU is used."""

    def __init__(self):
        import tempfile
        d = tempfile.mkdtemp(prefix="bench_clock_")
        self.out, self.stop_file = os.path.join(d, "samples.jsonl"), os.path.join(d, "stop")
        self.proc = subprocess.Popen([sys.executable, "-c", _SAMPLER, self.out, self.stop_file],
                                     stdout=subprocess.DEVNULL, stderr=subprocess.DEVNULL)
        self.window = None

    def mark(self, t0, t1):
        """The wall-time window whose samples are reported."""
        self.window = (t0, t1)

    def finish(self):
        open(self.stop_file, "w").close()
        try:
            self.proc.wait(timeout=40)
        except subprocess.TimeoutExpired:
            self.proc.kill()
        recs = []
        try:
            recs = [json.loads(l) for l in open(self.out) if l.strip()]
        except (OSError, ValueError):
            pass
        if self.window:
            recs = [r for r in recs if self.window[0] <= r["t"] <= self.window[1]]
        s = sorted(round(sum(r["mhz"]) / len(r["mhz"]), 1) for r in recs if r.get("mhz"))
        rec = {"source": "amd-smi metric -g 0 -c --json (current shader clock, MHz, mean over the XCDs), "
                         "about once a second during %.0f s of untimed step replays after the timed region" % CLOCK_S,
               "samples": len(s)}
        if s:
            rec.update({"min_mhz": s[0], "median_mhz": s[len(s) // 2], "max_mhz": s[-1]})
        errs = [r["error"] for r in recs if "error" in r]
        if errs or not s:
            rec["error"] = errs[0] if errs else "no shader clock in amd-smi output"
        return rec


# ---------------- timing helpers ----------------

def graph_time_us(launch, count, stream, reps, torch, np):
    """(median, min) per-launch time of a graph of `count` launches (launch(i))."""
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
    return float(np.median(times)), float(min(times))


def eager_time_us(launch, count, stream, reps, torch, np):
    """Single eager calls (not in a graph), each alone on the GPU: median of
    the event-timed latency and of the host time spent in the call."""
    ev, host = [], []
    with torch.cuda.stream(stream):
        for i in range(reps):
            a0 = torch.cuda.Event(enable_timing=True)
            a1 = torch.cuda.Event(enable_timing=True)
            stream.synchronize()
            a0.record(stream)
            h0 = time.perf_counter()
            launch(i % count)
            h1 = time.perf_counter()
            a1.record(stream)
            a1.synchronize()
            ev.append(a0.elapsed_time(a1) * 1e3)
            host.append((h1 - h0) * 1e6)
    return float(np.median(ev)), float(np.median(host))


class Layer:
    """One weight matrix (K, N, g): packed once, replicated to >= 1 GiB of
    copies; the fp16 comparator's dequantised weights likewise."""

    def __init__(self, mk, synth, torch, dev, K, N, wid, g, fp16=True, min_copies=2):
        self.K, self.N, self.g, self.wid = K, N, g, wid
        q, s = synth.weights(wid, K, N, None if g == -1 else g)
        self.q, self.s = q, s
        qd, sd = torch.from_numpy(q).to(dev), torch.from_numpy(s).to(dev)
        wp, sp = mk.pack(qd, sd, group=g)
        self.wbytes = wp.numel() + sp.numel() * 2
        n = max(min_copies, math.ceil(ROTATION_BYTES / self.wbytes))
        self.wps = [wp] + [wp.clone() for _ in range(n - 1)]
        self.sps = [sp] + [sp.clone() for _ in range(n - 1)]
        self.w16s = []
        if fp16:
            rows = K if g == -1 else g
            w16 = ((qd.to(torch.float32) - 8.0) * sd.to(torch.float32).repeat_interleave(rows, dim=0)).to(torch.float16)
            n16 = max(2, math.ceil(ROTATION_BYTES / (w16.numel() * 2)))
            self.w16s = [w16] + [w16.clone() for _ in range(n16 - 1)]
            del w16
        del qd, sd
        torch.cuda.synchronize()

    @property
    def copies(self):
        return len(self.wps)

    def name(self):
        return "%dx%d g=%s" % (self.K, self.N, "K" if self.g == -1 else self.g)


def measure_cases(args, mk, R, torch, np, dev, layer, Ms, stream, L, ws, acts, outs, label):
    """Per-M records of one layer: graph replays over the rotated copies, the
    eager latency, and the fp16 comparator."""
    K, N, g = layer.K, layer.N, layer.g
    rows = []
    for M in Ms:
        A, C = acts[M], outs[M]

        def launch(i, M=M, A=A, C=C):
            st = L.marlin_gemm(A.data_ptr(), layer.wps[i].data_ptr(), layer.sps[i].data_ptr(), C.data_ptr(),
                               ws.data_ptr(), ws.numel(), M, N, K, g, stream.cuda_stream)
            if st != 0:
                raise mk.MarlinError("marlin_gemm", st)
        with Range(torch, "%s w4a16 K=%d N=%d g=%d M=%d" % (label, K, N, g, M)):
            t, tmin = graph_time_us(launch, layer.copies, stream, args.per_m_reps, torch, np)
        ev, host = eager_time_us(launch, layer.copies, stream, 20, torch, np)
        troof = R.w4a16_t_roof(M, N, K, g) * 1e6
        rec = {"K": K, "N": N, "group": g, "M": M, "us": round(t, 3), "us_min": round(tmin, 3),
               "eager_us": round(ev, 3), "host_us_per_call": round(host, 2),
               "tflops": round(R.flops(M, N, K) / (t * 1e-6) / 1e12, 3),
               "weight_GBps": round(R.weight_bytes(N, K, g) / (t * 1e-6) / 1e9, 1),
               "roof_us": round(troof, 3), "roof_frac": round(troof / t, 4),
               "bound": R.bound(M, N, K, g), "launch": mk.marlin_describe(M, N, K, g)}
        if layer.w16s:
            n16 = len(layer.w16s)
            t16, _ = graph_time_us(lambda i: torch.matmul(A, layer.w16s[i % n16]), n16, stream,
                                   args.per_m_reps, torch, np)
            rec["fp16_us"] = round(t16, 3)
            rec["speedup_vs_fp16"] = round(t16 / t, 3)
        rows.append(rec)
        log("%s %dx%d g=%s M=%3d: %.3f us (eager %.2f us, host %.1f us), %.0f weight GB/s, roofline frac %.3f%s" %
            (label, K, N, g, M, t, ev, host, rec["weight_GBps"], troof / t,
             ", fp16 %.2f us -> %.2fx" % (rec["fp16_us"], rec["speedup_vs_fp16"]) if "fp16_us" in rec else ""))
    return rows


def layer_section(args, mk, R, synth, torch, np, dev, shapes, label):
    """A per-M sweep of other layers, outside the timed region."""
    L = mk.lib()
    stream = torch.cuda.Stream(device=dev)
    wsb = mk.Workspace(dev)
    out = []
    for (K, N, wid, g) in shapes:
        layer = Layer(mk, synth, torch, dev, K, N, wid, g, fp16=not args.no_fp16)
        ws = wsb.ensure(max(mk.marlin_workspace_bytes(M, N, K, g) for M in M_SWEEP))
        acts = {M: torch.from_numpy(synth.activations(wid, M, K)).to(dev) for M in M_SWEEP}
        outs = {M: torch.empty((M, N), dtype=torch.float16, device=dev) for M in M_SWEEP}
        out += measure_cases(args, mk, R, torch, np, dev, layer, M_SWEEP, stream, L, ws, acts, outs, label)
        del layer, acts, outs
        torch.cuda.synchronize()
    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        tot, flops, rows = 0.0, 0.0, []
        for (K, N, wid, g) in shapes:
            q, s = synth.weights(wid, K, N, None if g == -1 else g)
            for M in CPU_MS:
                A_np = synth.activations(wid, M, K)
                c0 = time.perf_counter()
                oracle.gemm(A_np, q, s, g)
                dt = time.perf_counter() - c0
                tot += dt
                flops += R.flops(M, N, K)
                rows.append({"K": K, "N": N, "group": g, "M": M, "seconds": round(dt, 4)})
        cpu = {"value": round(flops / tot / 1e12, 6), "unit": "TFLOP/s", "cores": cpu_threads(),
               "kind": "oracle", "sample": "fp64 oracle, full products at M in %s on every layer of the section"
               % CPU_MS, "per_case": rows}
        log("%s oracle: %.2f s" % (label, tot))
    return {"workload": "W4A16 GEMM, %s, M sweep %s, weights rotated over >= 1 GiB per layer" %
                        (", ".join("%dx%d g=%s" % (K, N, "K" if g == -1 else g) for K, N, _, g in shapes), M_SWEEP),
            "per_m": out, "cpu_baseline": cpu}


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
            with Range(torch, "sparse %s M=%d" % ("2:4" if sp_flag else "dense", M)):
                t[sp_flag], _ = graph_time_us(launch, len(wps), stream, args.per_m_reps, torch, np)
        t16 = None
        if not args.no_fp16:
            t16, _ = graph_time_us(lambda i: torch.matmul(A, w16s[i % n16]), n16, stream, args.per_m_reps, torch, np)
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


def sparse_profile_cases(args, mk, synth, torch, dev):
    """Counter runs of the 2:4 kernel (--profile-cases C --profile-layers
    sparse_2of4): at each M of the sweep, C launches in a row on 8192 x 8192,
    each on the next of two packed copies, in sweep order."""
    K, N, g = SPARSE_K, SPARSE_N, GROUP
    q, keep, s = synth.sparse24_weights(SPARSE_WID, K, N, g)
    qd, sd = torch.from_numpy(q).to(dev), torch.from_numpy(s).to(dev)
    L = mk.lib()
    wp, sp = mk.pack(qd, sd, group=g, sparse=True)
    wps = [wp, wp.clone()]
    ws = mk.Workspace(dev)
    wsbuf = ws.ensure(max(mk.marlin_workspace_bytes(M, N, K, g) for M in M_SWEEP))
    stream = torch.cuda.Stream(device=dev)
    cases = []
    with torch.cuda.stream(stream):
        for M in M_SWEEP:
            A = torch.from_numpy(synth.activations(SPARSE_WID, M, K)).to(dev)
            C = torch.empty((M, N), dtype=torch.float16, device=dev)
            for i in range(args.profile_cases):
                st = L.marlin_gemm_sparse(A.data_ptr(), wps[i % 2].data_ptr(), sp.data_ptr(), C.data_ptr(),
                                          wsbuf.data_ptr(), wsbuf.numel(), M, N, K, g, stream.cuda_stream)
                if st != 0:
                    raise mk.MarlinError("marlin_gemm_sparse", st)
            cases.append({"K": K, "N": N, "group": g, "M": M, "sparse": True,
                          "launch": mk.marlin_describe_sparse(M, N, K, g)})
    torch.cuda.synchronize()
    print(json.dumps({"profile_cases": args.profile_cases, "layers": "sparse_2of4", "cases": cases}), flush=True)


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
            with Range(torch, "prefill K=%d N=%d M=%d" % (K, N, M)):
                t, _ = graph_time_us(launch, 4, stream, args.per_m_reps, torch, np)
            rec = {"K": K, "N": N, "M": M, "us": round(t, 2),
                   "TFLOPs": round(R.flops(M, N, K) / t / 1e6, 1),
                   "mfma_frac": round(R.flops(M, N, K) / (t * 1e-6) / R.FP16_MFMA_FLOPS, 4),
                   "launch": mk.marlin_describe(M, N, K, g)}
            if w16 is not None:
                t16, _ = graph_time_us(lambda i: torch.matmul(A, w16), 4, stream, args.per_m_reps, torch, np)
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
    70B-class MLP down projection.  Bound by fp32 vector work: ``alu_frac``
    is its vector instructions per weight (from the committed counter
    profile) against the non-packed vector issue rate; ``hbm_GBps`` for
    reference."""
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
        with Range(torch, "quantize K=%d N=%d" % (K, N)):
            t, _ = graph_time_us(launch, 2, stream, args.per_m_reps, torch, np)
        ops = R.quant_lane_ops(K, N, len(ratios))
        rec = {"K": K, "N": N, "group": g, "ratios": len(ratios), "us": round(t, 2),
               "Gweights_per_s": round(K * N / t / 1e3, 2),
               "alu_frac": round(ops / (t * 1e-6) / R.VALU_LANE_OPS, 4),
               "hbm_GBps": round(R.quant_bytes(K, N, g) / t / 1e3, 1)}
        rows.append(rec)
        log("quantize %dx%d g=%d, %d ratios: %.1f us, %.2f G weights/s, %.1f%% of the vector issue rate" %
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
            "bound": "alu", "peak_lane_ops_per_s": R.VALU_LANE_OPS,
            "valu_lane_ops_per_weight": R.QUANT_VALU_PER_WEIGHT_G128_10,
            "per_shape": rows, "cpu_baseline": cpu}


def run_section(name, args, mk, R, synth, torch, np, dev):
    if name == "attention_4096":
        return layer_section(args, mk, R, synth, torch, np, dev, ATTENTION, name)
    if name == "mlp_7b":
        return layer_section(args, mk, R, synth, torch, np, dev, MLP_7B, name)
    if name == "sparse_2of4":
        return sparse_section(args, mk, R, synth, torch, np, dev)
    if name == "prefill":
        return prefill_section(args, mk, R, synth, torch, np, dev)
    return quantize_section(args, mk, R, synth, torch, np, dev)


def single_thread_oracle():
    """The oracle on one thread (the 8192 x 28672 layer at M = 1), in a child
    process started with OMP_NUM_THREADS=1."""
    code = ("import json, time, oracle, synth\n"
            "q, s = synth.weights(3, 8192, 28672, 128)\n"
            "A = synth.activations(3, 1, 8192)\n"
            "oracle.gemm(A, q, s, 128)\n"
            "ts = []\n"
            "for _ in range(3):\n"
            "    t = time.perf_counter(); oracle.gemm(A, q, s, 128); ts.append(time.perf_counter() - t)\n"
            "print(json.dumps(sorted(ts)[1]))\n")
    env = dict(os.environ, OMP_NUM_THREADS="1")
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, env=env, cwd=ROOT, timeout=300)
    if r.returncode != 0:
        return {"error": r.stderr[-300:]}
    dt = float(r.stdout.strip().splitlines()[-1])
    return {"K": 8192, "N": 28672, "M": 1, "threads": 1, "seconds": round(dt, 4),
            "value": round(2.0 * 8192 * 28672 / dt / 1e12, 6), "unit": "TFLOP/s"}


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

    # child processes first: nothing is started once the GPU is in use
    headline = not (args.only or args.profile_cases)
    clock = ClockSampler() if headline and not args.no_clock else None
    single = single_thread_oracle() if headline and not args.no_cpu_baseline else None

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
    if args.only:
        print(json.dumps({args.only: run_section(args.only, args, mk, R, synth, torch, np, dev)}), flush=True)
        return
    if args.profile_cases and args.profile_layers == "sparse_2of4":
        sparse_profile_cases(args, mk, synth, torch, dev)
        return

    # ---- headline layers: pack once, replicate to >= 1 GiB per layer ----
    L = mk.lib()
    layers = []
    shapes = HEADLINE
    if args.profile_cases:
        shapes = {"headline": HEADLINE, "attention_4096": ATTENTION, "mlp_7b": MLP_7B}[args.profile_layers]
    for (K, N, wid, g) in shapes:
        layers.append(Layer(mk, synth, torch, dev, K, N, wid, g,
                            fp16=not (args.no_fp16 or args.profile_cases), min_copies=2))
        log("weights %s: %d B packed per copy, %d copies (%.2f GB)" %
            (layers[-1].name(), layers[-1].wbytes, layers[-1].copies, layers[-1].copies * layers[-1].wbytes / 1e9))
    acts = {(lay.K, lay.N, M): torch.from_numpy(synth.activations(lay.wid, M, lay.K)).to(dev)
            for lay in layers for M in M_SWEEP}
    outs = {(lay.K, lay.N, M): torch.empty((M, lay.N), dtype=torch.float16, device=dev)
            for lay in layers for M in M_SWEEP}
    wsb = mk.Workspace(dev)
    ws = wsb.ensure(max(mk.marlin_workspace_bytes(M, lay.N, lay.K, lay.g) for lay in layers for M in M_SWEEP))
    stream = torch.cuda.Stream(device=dev)
    cases = [(lay, M) for lay in layers for M in M_SWEEP]

    def launch(lay, M, i):
        st = L.marlin_gemm(acts[(lay.K, lay.N, M)].data_ptr(), lay.wps[i].data_ptr(), lay.sps[i].data_ptr(),
                           outs[(lay.K, lay.N, M)].data_ptr(), ws.data_ptr(), ws.numel(), M, lay.N, lay.K, lay.g,
                           stream.cuda_stream)
        if st != 0:
            raise mk.MarlinError("marlin_gemm", st)

    if args.profile_cases:
        # counter runs: each case C times in a row, eagerly, in sweep order
        with torch.cuda.stream(stream):
            for lay, M in cases:
                for i in range(args.profile_cases):
                    launch(lay, M, i % lay.copies)
        torch.cuda.synchronize()
        print(json.dumps({"profile_cases": args.profile_cases, "layers": args.profile_layers,
                          "cases": [{"K": lay.K, "N": lay.N, "group": lay.g, "M": M,
                                     "launch": mk.marlin_describe(M, lay.N, lay.K, lay.g)} for lay, M in cases]}),
              flush=True)
        return

    # ---- graphs: one step (every case) per graph, rotating the copies ----
    ngraphs = max(lay.copies for lay in layers)
    torch.cuda.synchronize()
    graphs = []
    with torch.cuda.stream(stream):
        for lay, M in cases:  # eager warm-up of every variant
            launch(lay, M, 0)
        stream.synchronize()
        for gi in range(ngraphs):
            gr = torch.cuda.CUDAGraph()
            with torch.cuda.graph(gr, stream=stream):
                for j, (lay, M) in enumerate(cases):
                    launch(lay, M, (gi * len(M_SWEEP) + j) % lay.copies)
            graphs.append(gr)
    torch.cuda.synchronize()
    log("captured %d graphs of %d launches" % (ngraphs, len(cases)))

    step_flops = sum(R.flops(M, lay.N, lay.K) for lay, M in cases)
    step_bytes = sum(R.w4a16_bytes(M, lay.N, lay.K, lay.g) for lay, M in cases)
    step_wbytes = sum(R.weight_bytes(lay.N, lay.K, lay.g) for lay, M in cases)

    # ---- clock ramp, warm-up and timed region ----
    # The shader clock ramps up over tens of milliseconds of load, while the
    # timed region of a short run lasts about ten: the step graphs are first
    # replayed for RAMP_S seconds (untimed), then the W warm-up steps.
    ramp_steps = 0
    t_ramp = time.perf_counter()
    with torch.cuda.stream(stream):
        while time.perf_counter() - t_ramp < RAMP_S:
            for _ in range(8):
                graphs[ramp_steps % ngraphs].replay()
                ramp_steps += 1
            stream.synchronize()
        for k in range(args.warmup):
            graphs[k % ngraphs].replay()
    torch.cuda.synchronize()
    log("clock ramp: %d untimed steps in %.0f ms" % (ramp_steps, (time.perf_counter() - t_ramp) * 1e3))
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    with Range(torch, "timed steps"):
        with torch.cuda.stream(stream):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            e0.record(stream)
            for k in range(args.steps):
                graphs[k % ngraphs].replay()
            e1.record(stream)
            torch.cuda.synchronize()
            t1 = time.perf_counter()
    if clock:
        # the shader clock under the step's own load: CLOCK_S seconds of
        # untimed step replays, the window whose amd-smi readings are reported
        w0 = time.time()
        k = 0
        with torch.cuda.stream(stream):
            while time.time() - w0 < CLOCK_S:
                for _ in range(8):
                    graphs[k % ngraphs].replay()
                    k += 1
                stream.synchronize()
        clock.mark(w0, time.time())
    del graphs
    ev_ms = e0.elapsed_time(e1)
    wall_ms = (t1 - t0) * 1e3
    ms_per_step = ev_ms / args.steps
    value = step_flops / (ms_per_step * 1e-3) / 1e12
    log("timed %d steps: %.3f ms/step (events), wall %.3f ms/step, %.1f TFLOP/s" %
        (args.steps, ms_per_step, wall_ms / args.steps, value))
    avg_launch_us = ms_per_step * 1e3 / len(cases)
    achieved_gbs = step_bytes / (ms_per_step * 1e-3) / 1e9

    # ---- per case: graph of one launch per weight copy, eager latency, fp16 ----
    per_m = []
    for lay in layers:
        la = {M: acts[(lay.K, lay.N, M)] for M in M_SWEEP}
        lo = {M: outs[(lay.K, lay.N, M)] for M in M_SWEEP}
        per_m += measure_cases(args, mk, R, torch, np, dev, lay, M_SWEEP, stream, L, ws, la, lo, "70b")
    for lay in layers:
        lay.w16s = []
    torch.cuda.synchronize()

    # by kernel class: the stream kernel's launches (M <= 32) and the rest
    by_kernel = {}
    for r in per_m:
        k = r["launch"].split("<")[0]
        d = by_kernel.setdefault(k, {"launches_per_step": 0, "algorithmic_bytes": 0.0, "us": 0.0})
        d["launches_per_step"] += 1
        d["algorithmic_bytes"] += R.w4a16_bytes(r["M"], r["N"], r["K"], r["group"])
        d["us"] += r["us"]
    for k, d in by_kernel.items():
        d["achieved_GBps"] = round(d["algorithmic_bytes"] / (d["us"] * 1e-6) / 1e9, 1)
        d["frac"] = round(d["algorithmic_bytes"] / (d["us"] * 1e-6) / R.HBM_BYTES_PER_S, 4)
        d["algorithmic_bytes"] = round(d["algorithmic_bytes"])
        d["us"] = round(d["us"], 3)

    # ---- CPU baseline: the fp64 oracle on the host (also a full-output parity check) ----
    cpu = None
    parity = None
    if not args.no_cpu_baseline:
        import oracle
        threads = cpu_threads()
        tot, flops, rows = 0.0, 0.0, []
        worst, ok = 0.0, True
        for lay in layers:
            for M in CPU_MS:
                A_np = acts[(lay.K, lay.N, M)].cpu().numpy()
                runs = []
                for _ in range(3):
                    c0 = time.perf_counter()
                    ref = oracle.gemm(A_np, lay.q, lay.s, lay.g)
                    runs.append(time.perf_counter() - c0)
                dt = float(np.median(runs))
                tot += dt
                flops += R.flops(M, lay.N, lay.K)
                rows.append({"K": lay.K, "N": lay.N, "M": M, "seconds": round(dt, 4),
                             "GFLOPs": round(R.flops(M, lay.N, lay.K) / dt / 1e9, 2)})
                launch(lay, M, 0)
                torch.cuda.synchronize()
                got = outs[(lay.K, lay.N, M)].cpu().numpy().astype(np.float64)
                err = np.abs(got - ref)
                ok &= bool((err <= 2e-3 + 1e-2 * np.abs(ref)).all())
                worst = max(worst, float(err.max()))
                log("oracle %dx%d M=%d: %.3f s" % (lay.K, lay.N, M, dt))
        cpu = {"value": round(flops / tot / 1e12, 6), "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
               "sample": "fp64 oracle, full products of both 70B-class layers at M in %s (median of 3 runs "
                         "each, %.1f GFLOP per run set)" % (CPU_MS, flops / 1e9),
               "seconds": round(tot, 3), "cpu_model": cpu_model(), "per_case": rows,
               "single_thread": single}
        parity = {"ok": ok, "max_abs_err": worst, "cases": "both layers at M in %s, every output" % CPU_MS,
                  "bar": "|C_gpu - C_ref| <= 2e-3 + 1e-2 |C_ref|"}
        log("oracle: %.2f s on %d threads (%s); GPU parity %s (max err %.3g)" %
            (tot, threads, cpu["cpu_model"], ok, worst))

    sections = {}
    if not args.no_sections:
        del acts, outs, layers
        torch.cuda.synchronize()
        for name in SECTIONS:
            sections[name] = run_section(name, args, mk, R, synth, torch, np, dev)
            torch.cuda.synchronize()

    clock_rec = clock.finish() if clock else None
    small = [r for r in per_m if r["M"] <= 16]
    copies = {"%dx%d" % (K, N): int(math.ceil(ROTATION_BYTES / (K * N / 2 + 2 * (K // g) * N))) for K, N, _, g in HEADLINE}
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
        "config": {"workload": "70B-scale single-GPU layer shapes, W4A16 GEMM (K=8192 N=28672) and "
                               "(K=28672 N=8192), g=128, M sweep 1..128, weights rotated over >1 GB per layer",
                   "layers": [[K, N] for K, N, _, _ in HEADLINE], "group": GROUP, "M": M_SWEEP,
                   "weight_copies": copies, "launches_per_step": len(cases)},
        "weight_GBps": round(step_wbytes / (ms_per_step * 1e-3) / 1e9, 1),
        "roofline": {"bound": "hbm", "achieved": round(achieved_gbs, 1),
                     "peak": R.HBM_BYTES_PER_S / 1e9, "unit": "GB/s",
                     "frac": round(achieved_gbs * 1e9 / R.HBM_BYTES_PER_S, 4),
                     "traffic": measured_traffic(),
                     "traffic_unit": "HBM bytes per launch (step average)",
                     "algorithmic_bytes_per_launch": round(step_bytes / len(cases)),
                     "avg_launch_us": round(avg_launch_us, 3),
                     "kernel": "; ".join("%s at %s" % (k, ", ".join("%dx%d M=%d" % (r["K"], r["N"], r["M"])
                                                                   for r in per_m if r["launch"].startswith(k + "<")))
                                         for k in by_kernel) + ": every launch of the step",
                     "by_kernel": by_kernel},
        "roof_frac_step": round(sum(R.w4a16_t_roof(M, lay_n, lay_k, GROUP) for lay_k, lay_n, _, _ in HEADLINE
                                    for M in M_SWEEP) / (ms_per_step * 1e-3), 4),
        "min_roof_frac_M_le_16": min(r["roof_frac"] for r in small),
        "per_m": per_m,
        "wall_ms_per_step": round(wall_ms / args.steps, 6),
        "clock_ramp_steps": ramp_steps,
        "clock": clock_rec,
        "cpu_baseline": cpu,
        "parity": parity,
    }
    out.update(sections)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
