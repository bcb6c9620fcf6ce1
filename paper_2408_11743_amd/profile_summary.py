"""Summarise rocprofv3 output of bench.py into the text kept under profiles/.

Usage (after the three profiling runs, see the command block this prints):

    python -m paper_2408_11743_amd.profile_summary --trace DIR --fetch DIR \
        --write DIR --bench BENCH_JSON --out OUT_PREFIX [--copy-mb 256]

or, for bench.py --prefill-only or --quantize-only, a kernel trace alone (its
CSV, not only the statistics: --kernel-trace --stats --output-format csv):

    python -m paper_2408_11743_amd.profile_summary --trace DIR --bench BENCH_JSON --out OUT_PREFIX

and for the matrix-core counters of bench.py --prefill-only --no-fp16 (one
--pmc pass with PREFILL_COUNTERS):

    python -m paper_2408_11743_amd.profile_summary --pmc DIR --bench BENCH_JSON --out OUT_PREFIX

Reads
  DIR/*kernel_stats.csv          (rocprofv3 --kernel-trace --stats)
  DIR/*counter_collection.csv    (rocprofv3 --pmc FETCH_SIZE, then WRITE_SIZE)
  BENCH_JSON                     (the JSON line bench.py printed in the trace run)
and writes OUT_PREFIX_kernel_trace.md, OUT_PREFIX_traffic.md and
OUT_PREFIX_traffic.json.  The counters are scaled by what they read for the
plain device copies bench.py makes with --calibration-copy-mb (bytes known).
Each M of the sweep is attributed to its kernel instantiation through
marlin_describe, the library's own account of the launch it makes.
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import os
import statistics

HERE = os.path.dirname(os.path.abspath(__file__))
# Device sources the GEMM kernels are built from: a counter summary holds
# for the kernels only while these are unchanged.
KERNEL_SOURCES = ("gemm.hip", "tile.hip", "device.h", "internal.h")
COPY_KERNEL = "copyBuffer"


def kernel_sources_digest() -> str:
    h = hashlib.sha256()
    for name in KERNEL_SOURCES:
        h.update(name.encode())
        h.update(open(os.path.join(HERE, "csrc", name), "rb").read())
    return h.hexdigest()


def _one(pattern: str) -> str:
    files = sorted(glob.glob(pattern, recursive=True))
    if not files:
        raise SystemExit("no file matches %s" % pattern)
    return files[0]


def kernel_stats(trace_dir: str) -> dict[str, dict]:
    out = {}
    with open(_one(os.path.join(trace_dir, "**", "*kernel_stats.csv"))) as f:
        for r in csv.DictReader(f):
            out[r["Name"]] = {"calls": int(r["Calls"]), "avg_ns": float(r["AverageNs"]),
                              "total_ns": float(r["TotalDurationNs"])}
    return out


def counter_per_dispatch(pmc_dir: str, counter: str) -> list[tuple[str, float]]:
    """(kernel name, counter value summed over the dispatch's instances), per dispatch."""
    per = {}
    with open(_one(os.path.join(pmc_dir, "**", "*counter_collection.csv"))) as f:
        for r in csv.DictReader(f):
            if r["Counter_Name"] != counter:
                continue
            key = int(r["Dispatch_Id"])
            name, val = per.get(key, (r["Kernel_Name"], 0.0))
            per[key] = (name, val + float(r["Counter_Value"]))
    return [per[k] for k in sorted(per)]


def short(name: str) -> str:
    """'void marlin::(anonymous namespace)::w4a16_stream_kernel<1, 1, 8, 1, false>(...)' -> 'w4a16_stream_kernel<1, 1, 8, 1, false>'."""
    base = name.replace("(anonymous namespace)::", "").replace("void ", "", 1)
    base = base.split("(")[0].strip()
    return base.split("::")[-1]


def dispatch_runs(trace_dir: str, prefix: str, gap_ns: int = 20_000_000) -> list:
    """Runs of consecutive dispatches of kernels named prefix*: a run ends at
    any other kernel or at an idle gap of more than gap_ns (a case's replays
    are back to back; the host prepares the next case in between).  Runs of
    one dispatch (the eager launch before a graph capture, followed by the
    capture's own fill kernels) are left out."""
    trace = []
    with open(_one(os.path.join(trace_dir, "**", "*kernel_trace.csv"))) as f:
        for r in csv.DictReader(f):
            trace.append((int(r["Start_Timestamp"]), int(r["End_Timestamp"]), short(r["Kernel_Name"])))
    trace.sort()
    runs, cur, last_end = [], [], None
    for t0, t1, name in trace:
        if name.startswith(prefix):
            if cur and last_end is not None and t0 - last_end > gap_ns:
                runs.append(cur)
                cur = []
            cur.append((name, (t1 - t0) / 1e3))
            last_end = t1
        elif cur:
            runs.append(cur)
            cur = []
    if cur:
        runs.append(cur)
    return [r for r in runs if len(r) > 1]


def quantize_summary(a, bench: dict) -> None:
    """Kernel trace of bench.py --quantize-only: one row per shape."""
    import paper_2408_11743_amd.roofline as R
    cases = bench["quantize"]["per_shape"]
    runs = dispatch_runs(a.trace, "quantize_kernel")
    if len(runs) != len(cases):
        raise SystemExit("%d quantiser runs in the trace for %d cases" % (len(runs), len(cases)))
    md = ["# Kernel trace: weight quantiser, g = 128, clipping search over %d ratios" % cases[0]["ratios"], "",
          "Command (`TMPDIR=/tmp`, from the repository root):", "", "```", a.trace_cmd, "```", "",
          "Per shape: the median kernel duration over the shape's replayed dispatches",
          "(rocprofv3), the bench's event time per call of an unprofiled run (--bench),",
          "and the fraction of the fp32 vector lane rate (78.65 T operations/s: the",
          "published 157.3 TFLOP/s counts a fused multiply-add as two) that the",
          "quantiser's algorithmic operations (`roofline.quant_ops`) reach in the",
          "kernel time; HBM GB/s for reference (fp16 read, codes and scales written):", "",
          "| K | N | kernel | dispatches | median kernel us | bench us | G weights/s | ALU frac | HBM GB/s |",
          "|---|---|---|---|---|---|---|---|---|"]
    for case, run in zip(cases, runs):
        names = sorted({n for n, _ in run})
        med = statistics.median(d for _, d in run)
        K, N = case["K"], case["N"]
        ops = R.quant_ops(K, N, case["ratios"])
        md.append("| %d | %d | `%s` | %d | %.1f | %.1f | %.2f | %.3f | %.0f |" % (
            K, N, ", ".join(names), len(run), med, case["us"], K * N / med / 1e3,
            ops / (med * 1e-6) / R.FP32_LANE_OPS, R.quant_bytes(K, N, case["group"]) / med / 1e3))
    md.append("")
    open(a.out + "_kernel_trace.md", "w").write("\n".join(md) + "\n")
    print("wrote", a.out + "_kernel_trace.md")


PREFILL_COUNTERS = ("SQ_INSTS_MFMA", "SQ_VALU_MFMA_BUSY_CYCLES", "SQ_INSTS_VALU", "SQ_INSTS_LDS",
                    "SQ_LDS_BANK_CONFLICT", "SQ_WAVES", "GRBM_GUI_ACTIVE")


def prefill_counter_summary(a, bench: dict) -> None:
    """Counters of bench.py --prefill-only --no-fp16 (one --pmc pass): matrix
    core utilisation per case.

    Every case has its own MFMA count per dispatch (M*N*K differs), so the
    GEMM dispatches are grouped by runs of equal SQ_INSTS_MFMA, in the order
    of the bench's cases.  Utilisation = MFMA busy cycles / (SIMDs x kernel
    cycles), kernel cycles being GRBM_GUI_ACTIVE per XCD (the counter sums
    the 8 XCDs)."""
    cases = bench["prefill"]["per_m"]
    per = {}
    with open(_one(os.path.join(a.pmc, "**", "*counter_collection.csv"))) as f:
        for r in csv.DictReader(f):
            if not short(r["Kernel_Name"]).startswith("w4a16_"):
                continue
            d = per.setdefault(int(r["Dispatch_Id"]), {"name": short(r["Kernel_Name"])})
            d[r["Counter_Name"]] = d.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    runs, cur = [], []
    for k in sorted(per):
        d = per[k]
        if cur and d.get("SQ_INSTS_MFMA") != cur[-1].get("SQ_INSTS_MFMA"):
            runs.append(cur)
            cur = []
        cur.append(d)
    if cur:
        runs.append(cur)
    if len(runs) != len(cases):
        raise SystemExit("%d groups of equal MFMA counts for %d cases" % (len(runs), len(cases)))
    simds, xcds = 256 * 4, 8
    md = ["# Matrix-core utilisation: W4A16 GEMM at large batches (rocprofv3 counters)", "",
          "Command (`TMPDIR=/tmp`, from the repository root; one counter pass):", "", "```", a.pmc_cmd, "```", "",
          "Per case, medians over its dispatches: MFMA instructions, the MFMA pipe's busy",
          "cycles, and the kernel's cycles (GRBM_GUI_ACTIVE per XCD).  Utilisation = busy",
          "cycles / (1024 SIMDs x kernel cycles): the fraction of the matrix-core peak at",
          "the clock the chip actually ran (about 2.1 GHz under this load, below the",
          "2.4 GHz of the published peak).  VALU per MFMA counts the other vector",
          "instructions (dequantisation, fold).", "",
          "| K | N | M | kernel | dispatches | MFMA / dispatch | MFMA busy | kernel cycles | utilisation | VALU per MFMA | LDS bank conflicts |",
          "|---|---|---|---|---|---|---|---|---|---|---|"]
    for case, run in zip(cases, runs):
        med = {c: statistics.median(d.get(c, 0.0) for d in run) for c in PREFILL_COUNTERS}
        cyc = med["GRBM_GUI_ACTIVE"] / xcds
        util = med["SQ_VALU_MFMA_BUSY_CYCLES"] / (simds * cyc) if cyc else float("nan")
        other = (med["SQ_INSTS_VALU"] - med["SQ_INSTS_MFMA"]) / med["SQ_INSTS_MFMA"] if med["SQ_INSTS_MFMA"] else 0
        md.append("| %d | %d | %d | `%s` | %d | %.0f | %.3g | %.3g | %.3f | %.2f | %.0f |" % (
            case["K"], case["N"], case["M"], run[0]["name"], len(run), med["SQ_INSTS_MFMA"],
            med["SQ_VALU_MFMA_BUSY_CYCLES"], cyc, util, other, med["SQ_LDS_BANK_CONFLICT"]))
    md.append("")
    open(a.out + "_counters.md", "w").write("\n".join(md) + "\n")
    print("wrote", a.out + "_counters.md")


def prefill_summary(a, bench: dict) -> None:
    """Kernel trace of bench.py --prefill-only: one row per (K, N, M) case.

    Cases can share a kernel instantiation, so the per-dispatch trace is
    used: the replayed GEMM dispatches of one case form one run, which the
    fp16 comparator's kernels (and the weight set-up between shapes) end; the
    i-th run belongs to the i-th case of the bench output."""
    sec = bench["prefill"]
    cases = sec["per_m"]
    runs = dispatch_runs(a.trace, "w4a16_")
    if len(runs) != len(cases):
        raise SystemExit("%d GEMM runs in the trace for %d cases (run with the fp16 comparator)" %
                         (len(runs), len(cases)))
    import paper_2408_11743_amd.roofline as R
    md = ["# Kernel trace: W4A16 GEMM at large batches, one launch per call, g = 128", "",
          "Command (`TMPDIR=/tmp`, from the repository root):", "", "```", a.trace_cmd, "```", "",
          "Per case: the kernel the library launched (its own account, `launch`), the",
          "median kernel duration over the case's dispatches (rocprofv3), the bench's",
          "event time per launch of an unprofiled run (--bench), the fp16",
          "`torch.matmul` time beside it, and the fraction of the fp16 matrix-core",
          "peak (2.5 PFLOP/s) that the kernel duration gives:", "",
          "| K | N | M | kernel | dispatches | median kernel us | bench us | fp16 us | TFLOP/s (kernel) | MFMA frac |",
          "|---|---|---|---|---|---|---|---|---|---|"]
    for case, run in zip(cases, runs):
        names = {n for n, _ in run}
        want = case["launch"].split(" cols=")[0]
        if names != {want}:
            raise SystemExit("case %s: trace has %s, expected %s" % (case, names, want))
        med = statistics.median(d for _, d in run)
        fl = R.flops(case["M"], case["N"], case["K"])
        md.append("| %d | %d | %d | `%s` | %d | %.1f | %.1f | %s | %.0f | %.3f |" % (
            case["K"], case["N"], case["M"], want, len(run), med, case["us"],
            "%.1f" % case["fp16_us"] if "fp16_us" in case else "-", fl / med / 1e6,
            fl / (med * 1e-6) / R.FP16_MFMA_FLOPS))
    md += ["", "Configuration per case: " + "; ".join(
        "%dx%d M=%d: cols=%s" % (c["K"], c["N"], c["M"], c["launch"].split(" cols=")[1]) for c in cases), ""]
    open(a.out + "_kernel_trace.md", "w").write("\n".join(md) + "\n")
    print("wrote", a.out + "_kernel_trace.md")


def main() -> None:
    ap = argparse.ArgumentParser()
    ap.add_argument("--trace")
    ap.add_argument("--pmc", help="counter run of bench.py --prefill-only --no-fp16 (prefill counters)")
    ap.add_argument("--pmc-cmd", default="")
    ap.add_argument("--fetch")
    ap.add_argument("--write")
    ap.add_argument("--bench", required=True)
    ap.add_argument("--out", required=True)
    ap.add_argument("--copy-mb", type=int, default=256)
    ap.add_argument("--trace-cmd", default="")
    ap.add_argument("--fetch-cmd", default="")
    ap.add_argument("--write-cmd", default="")
    a = ap.parse_args()

    import paper_2408_11743_amd as mk

    bench = json.loads(open(a.bench).read().strip().splitlines()[-1])
    if "prefill" in bench and "config" not in bench:  # bench.py --prefill-only
        if a.pmc:
            prefill_counter_summary(a, bench)
        else:
            prefill_summary(a, bench)
        return
    if not a.trace:
        raise SystemExit("--trace is required for this bench output")
    if "quantize" in bench and "config" not in bench:  # bench.py --quantize-only
        quantize_summary(a, bench)
        return
    if not a.fetch or not a.write:
        raise SystemExit("--fetch and --write are required for the M sweeps")
    import paper_2408_11743_amd.roofline as R
    sparse = "config" not in bench  # bench.py --sparse-only
    if sparse:
        sec = bench["sparse_2of4"]
        K, N, g = 8192, 8192, 128
        Ms = [r["M"] for r in sec["per_m"]]
        bench_per_m = sec["per_m"]
        describe = {M: mk.marlin_describe_sparse(M, N, K, g) for M in Ms}
        alg_bytes = R.sparse24_bytes
        title = "2:4 sparse W4A16 GEMM"
    else:
        K, N, g = bench["config"]["K"], bench["config"]["N"], bench["config"]["group"]
        Ms = bench["config"]["M"]
        bench_per_m = bench.get("per_m", [])
        describe = {M: mk.marlin_describe(M, N, K, g) for M in Ms}
        alg_bytes = R.w4a16_bytes
        title = "W4A16 GEMM"
    # kernel name as a profiler prints it, e.g. "w4a16_stream_kernel<1, 1, 8, 1, false>"
    kname = {M: describe[M].split(" cols=")[0] for M in Ms}

    # ---- kernel trace ----
    stats = kernel_stats(a.trace)
    rows, step_ns = [], 0.0
    for M in Ms:
        hits = [(n, v) for n, v in stats.items() if short(n) == kname[M]]
        if not hits:
            raise SystemExit("kernel %s (M=%d) not in the trace" % (kname[M], M))
        avg = hits[0][1]["avg_ns"]  # all launches of one instantiation (all Ms that share it)
        cfg = "cols=" + describe[M].split(" cols=")[1] if " cols=" in describe[M] else ""
        rows.append((M, kname[M], cfg, hits[0][1]["calls"], avg))
        step_ns += avg
    md = ["# Kernel trace: %s, K = %d, N = %d, g = %d, M sweep %s" % (title, K, N, g, Ms), "",
          "Command (`TMPDIR=/tmp`, from the repository root):", "", "```", a.trace_cmd, "```", "",
          "Average duration per launch of each kernel instantiation over all its",
          "launches in the run (warm-up included; other kernels, such as the fp16",
          "comparator's, are not matched):", "",
          "| M | kernel | configuration | launches | avg kernel us | bench us per launch |",
          "|---|---|---|---|---|---|"]
    per_m = {r["M"]: r["us"] for r in bench_per_m}
    for M, k, cfg, calls, avg in rows:
        md.append("| %d | `%s` | %s | %d | %.3f | %.3f |" % (M, k, cfg, calls, avg / 1e3, per_m.get(M, float("nan"))))
    md += ["", "Mean over the %d launches of one step: %.3f us of kernel time (rocprofv3)." % (len(Ms), step_ns / len(Ms) / 1e3)]
    if not sparse:
        md += ["%.3f us per launch measured by bench.py with HIP events over its timed region" % bench["roofline"]["avg_launch_us"],
               "(`roofline.avg_launch_us`, an unprofiled run: --bench)."]
    md += ["The event time of a launch (bench us per launch, graph replays) also holds",
           "the dispatch gap between consecutive graph nodes, which the kernel time",
           "excludes (an empty kernel costs about 1.7 us per launch in a graph).",
           "Shared instantiations (same kernel for several M) report one average for all",
           "of their launches, so the per-M rows are approximate where a kernel is shared.", ""]
    open(a.out + "_kernel_trace.md", "w").write("\n".join(md) + "\n")

    # ---- traffic ----
    fetch = counter_per_dispatch(a.fetch, "FETCH_SIZE")
    write = counter_per_dispatch(a.write, "WRITE_SIZE")
    copy_bytes = a.copy_mb * (1 << 20)
    # The calibration copies are the largest copy dispatches of the run (the
    # weight clones bench.py makes use the same copy kernel, on smaller
    # buffers: 8.65 MB packed copies, 134 MB fp16 copies in the sparse section).
    def largest(samples):
        v = [x for n, x in samples if COPY_KERNEL in n]
        return [x for x in v if x >= 0.9 * max(v)] if v else []

    cf, cw = largest(fetch), largest(write)
    if not cf or not cw:
        raise SystemExit("no calibration copies in the counter runs (--calibration-copy-mb)")
    f_scale = copy_bytes / (statistics.median(cf) * 1024.0)
    w_scale = copy_bytes / (statistics.median(cw) * 1024.0)

    def per_kernel(samples, scale):
        out = {}
        for n, v in samples:
            out.setdefault(short(n), []).append(v * 1024.0 * scale)
        return {k: statistics.median(v) for k, v in out.items()}

    fk, wk = per_kernel(fetch, f_scale), per_kernel(write, w_scale)
    trows, hbm = [], {}
    step_bytes = 0.0
    for M in Ms:
        k = kname[M]
        fb, wb = fk.get(k), wk.get(k)
        if fb is None or wb is None:
            raise SystemExit("kernel %s (M=%d) has no counter samples" % (k, M))
        alg = alg_bytes(M, N, K, g)
        trows.append((M, k, fb, wb, fb + wb, alg))
        hbm["M=%d %s" % (M, k)] = round(fb + wb)
        step_bytes += fb + wb
    md = ["# HBM traffic: %s, K = %d, N = %d, g = %d, M sweep %s" % (title, K, N, g, Ms), "",
          "Commands (two counter passes, each its own run, `TMPDIR=/tmp`):", "", "```",
          a.fetch_cmd, a.write_cmd, "```", "",
          "Calibration: the same runs make plain device copies of %d MiB (the runtime's" % a.copy_mb,
          "copy kernel).  Per copy FETCH_SIZE reads %.0f KiB for %d KiB read (scale x%.3f)," %
          (statistics.median(cf), copy_bytes // 1024, f_scale),
          "WRITE_SIZE %.0f KiB for %d KiB written (scale x%.3f)." % (statistics.median(cw), copy_bytes // 1024, w_scale),
          "", "Per dispatch (median over the dispatches of each instantiation), scaled:", "",
          "| M | kernel | fetch MB | write MB | HBM MB | algorithmic MB | ratio |",
          "|---|---|---|---|---|---|---|"]
    for M, k, fb, wb, tb, alg in trows:
        md.append("| %d | `%s` | %.2f | %.2f | %.2f | %.2f | %.2f |" % (M, k, fb / 1e6, wb / 1e6, tb / 1e6, alg / 1e6, tb / alg))
    digest = kernel_sources_digest()
    md += ["", ("Algorithmic bytes: K*N/4 + K*N/8 + 2*(K/g)*N + 2*M*K + 2*M*N (kept codes, row indices)."
                if sparse else "Algorithmic bytes: K*N/2 + 2*(K/g)*N + 2*M*K + 2*M*N."), "",
           "Step average per launch: %.2f MB (bench.py reports it as `roofline.traffic`" % (step_bytes / len(Ms) / 1e6),
           "while the kernel sources (%s under `paper_2408_11743_amd/csrc/`) hash to `%s...`)." %
           (", ".join(KERNEL_SOURCES), digest[:16]), ""]
    open(a.out + "_traffic.md", "w").write("\n".join(md) + "\n")
    rec = {"workload": "%s K=%d N=%d g=%d, M sweep %s (bench.py)" % (title, K, N, g, Ms),
           "kernel_sources_sha256": digest,
           "counter_scale": {"FETCH_SIZE": round(f_scale, 4), "WRITE_SIZE": round(w_scale, 4),
                             "calibration": "device copies of %d MiB" % a.copy_mb},
           "hbm_bytes_per_launch": hbm, "step_launches": Ms,
           "step_avg_hbm_bytes_per_launch": round(step_bytes / len(Ms))}
    json.dump(rec, open(a.out + "_traffic.json", "w"), indent=1)
    print("wrote", a.out + "_kernel_trace.md", a.out + "_traffic.md", a.out + "_traffic.json")


if __name__ == "__main__":
    main()
