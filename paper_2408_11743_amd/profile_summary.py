"""Summarise rocprofv3 output of bench.py into the text kept under profiles/.

Modes (each reads the JSON line bench.py printed in the same run, --bench):

* headline kernel trace -- ``rocprofv3 --kernel-trace --marker-trace --stats
  --output-format csv`` of ``bench.py``: every kernel dispatch is attributed
  to the bench's named ranges (one per (layer, M) case, one for the timed
  steps), giving the median kernel duration per case and the mean over the
  timed steps' launches beside the bench's event times::

      --trace DIR --bench JSON --out PREFIX

* per-case counters -- ``rocprofv3 --pmc ...`` of ``bench.py --profile-cases C``
  (each case launched C times in a row, in the order the JSON lists):
  HBM traffic from a FETCH_SIZE and a WRITE_SIZE pass, scaled by the same
  passes' plain device copies (--calibration-copy-mb)::

      --fetch DIR --write DIR --bench JSON --out PREFIX [--copy-mb 256]

  or matrix-core and vector counters (one pass of CASE_COUNTERS)::

      --pmc DIR --bench JSON --out PREFIX

* bench.py --only prefill / quantize / sparse_2of4: kernel trace (and for
  prefill the matrix-core counters, --pmc), as before.
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
# Sources the GEMM kernels and their launch plans are built from: a counter
# summary holds for the kernels only while these are unchanged.
KERNEL_SOURCES = ("gemm.hip", "pair.hip", "tile.hip", "wide.hip", "device.h", "internal.h", "plan.h", "plan.cpp")
COPY_KERNEL = "copyBuffer"


def kernel_sources_digest() -> str:
    h = hashlib.sha256()
    for name in KERNEL_SOURCES:
        h.update(name.encode())
        h.update(open(os.path.join(HERE, "csrc", name), "rb").read())
    return h.hexdigest()


def _one(pattern: str) -> str:
    files = sorted(glob.glob(pattern, recursive=True))
    if len(files) != 1:  # none, or results of several runs in one directory
        raise SystemExit("%d files match %s (one run per output directory)" % (len(files), pattern))
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
          "and the fraction of the vector issue rate (78.6 T lane operations/s: 256 CUs x",
          "4 SIMDs x 32 lanes x 2.4 GHz) that the kernel's issued vector instructions",
          "(`roofline.quant_lane_ops`, its instruction count) reach in the kernel time;",
          "HBM GB/s for reference (fp16 read, codes and scales written):", "",
          "| K | N | kernel | dispatches | median kernel us | bench us | G weights/s | ALU frac | HBM GB/s |",
          "|---|---|---|---|---|---|---|---|---|"]
    for case, run in zip(cases, runs):
        names = sorted({n for n, _ in run})
        med = statistics.median(d for _, d in run)
        K, N = case["K"], case["N"]
        ops = R.quant_lane_ops(K, N, case["ratios"])
        md.append("| %d | %d | `%s` | %d | %.1f | %.1f | %.2f | %.3f | %.0f |" % (
            K, N, ", ".join(names), len(run), med, case["us"], K * N / med / 1e3,
            ops / (med * 1e-6) / R.VALU_LANE_OPS, R.quant_bytes(K, N, case["group"]) / med / 1e3))
    md.append("")
    open(a.out + "_kernel_trace.md", "w").write("\n".join(md) + "\n")
    print("wrote", a.out + "_kernel_trace.md")


QUANT_COUNTERS = ("SQ_INSTS_VALU", "SQ_ACTIVE_INST_VALU", "SQ_WAVES", "SQ_WAVE_CYCLES", "SQ_BUSY_CYCLES",
                  "GRBM_GUI_ACTIVE")


def quantize_counter_summary(a, bench: dict) -> None:
    """Vector-instruction counters of bench.py --only quantize (one --pmc pass
    of QUANT_COUNTERS): issued vector instructions per weight and the issue
    rate per SIMD, which fixes the lane rate the quantiser is measured
    against."""
    import paper_2408_11743_amd.roofline as R
    cases = bench["quantize"]["per_shape"]
    per = {}
    with open(_one(os.path.join(a.pmc, "**", "*counter_collection.csv"))) as f:
        for r in csv.DictReader(f):
            if not short(r["Kernel_Name"]).startswith("quantize_kernel"):
                continue
            d = per.setdefault(int(r["Dispatch_Id"]), {"grid": int(r["Grid_Size"])})
            d[r["Counter_Name"]] = d.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    simds, xcds = 256 * 4, 8
    md = ["# Vector-instruction counters: weight quantiser, g = 128, %d clipping ratios" % cases[0]["ratios"], "",
          "Command (`TMPDIR=/tmp`, from the repository root; one counter pass):", "", "```", a.pmc_cmd, "```", "",
          "Medians over each shape's dispatches (a shape is recognised by its grid: one",
          "thread per (group, column)).  VALU per weight = SQ_INSTS_VALU x 64 lanes /",
          "weights.  Kernel cycles = GRBM_GUI_ACTIVE / 8 XCDs.  Clocks per VALU",
          "instruction and SIMD = kernel cycles / (SQ_INSTS_VALU / 1024 SIMDs): below 4,",
          "an unpacked wave64 vector instruction cannot take four clocks, so the issue",
          "rate is taken as 32 lanes per SIMD and clock (`roofline.VALU_LANE_OPS`, 78.6",
          "T lane operations/s at 2.4 GHz); the issue utilisation is 2 / that ratio.", "",
          "| K | N | dispatches | VALU / wave | VALU per weight | kernel cycles | clocks per VALU instr and SIMD | issue utilisation |",
          "|---|---|---|---|---|---|---|---|"]
    for c in cases:
        K, N, g = c["K"], c["N"], c["group"]
        grid = (K // g) * ((N + 255) // 256) * 256
        ds = [d for d in per.values() if d["grid"] == grid]
        if not ds:
            raise SystemExit("no quantiser dispatches of grid %d" % grid)
        med = {k: statistics.median(d.get(k, 0.0) for d in ds) for k in QUANT_COUNTERS}
        cyc = med["GRBM_GUI_ACTIVE"] / xcds
        per_simd = med["SQ_INSTS_VALU"] / simds
        md.append("| %d | %d | %d | %.0f | %.2f | %.3g | %.2f | %.3f |" % (
            K, N, len(ds), med["SQ_INSTS_VALU"] / med["SQ_WAVES"], med["SQ_INSTS_VALU"] * 64 / (K * N), cyc,
            cyc / per_simd, 2 * per_simd / cyc))
    md += ["", "The library's account of the same kernel (`roofline.quant_lane_ops`, from its",
           "gfx950 assembly): %.2f lane operations per weight at %d ratios." % (
               R.QUANT_VALU_BASE + R.QUANT_VALU_PER_RATIO * cases[0]["ratios"], cases[0]["ratios"]), ""]
    open(a.out + "_counters.md", "w").write("\n".join(md) + "\n")
    print("wrote", a.out + "_counters.md")


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


def _timestamps_csv(trace_dir: str, pattern: str) -> list[dict]:
    with open(_one(os.path.join(trace_dir, "**", pattern))) as f:
        return list(csv.DictReader(f))


def marker_ranges(trace_dir: str) -> list[tuple[str, int, int]]:
    """(name, start ns, end ns) of the bench's named ranges (roctx push/pop
    pairs; rocprofv3 writes one row per range, or one per push and pop)."""
    rows = _timestamps_csv(trace_dir, "*marker_api_trace.csv")
    out, stack = [], []
    for r in sorted(rows, key=lambda r: int(r["Start_Timestamp"])):
        name = r.get("Message") or r.get("Function") or ""
        t0, t1 = int(r["Start_Timestamp"]), int(r["End_Timestamp"])
        fn = r.get("Function", "")
        if fn.startswith("roctxRangePush"):
            stack.append((r.get("Message", name), t0))
        elif fn.startswith("roctxRangePop"):
            if stack:
                n, s = stack.pop()
                out.append((n, s, t1))
        elif t1 > t0:
            out.append((name, t0, t1))
    return out


def dispatches(trace_dir: str) -> list[tuple[int, int, str]]:
    rows = _timestamps_csv(trace_dir, "*kernel_trace.csv")
    return sorted((int(r["Start_Timestamp"]), int(r["End_Timestamp"]), short(r["Kernel_Name"])) for r in rows)


def headline_trace_summary(a, bench: dict) -> None:
    """Kernel time per headline case and over the timed steps, from the
    named ranges of a profiled bench.py run."""
    import paper_2408_11743_amd.roofline as R
    ranges = marker_ranges(a.trace)
    disp = [d for d in dispatches(a.trace) if d[2].startswith("w4a16_")]

    def inside(name):
        rs = [(s, e) for n, s, e in ranges if n == name]
        if not rs:
            raise SystemExit("no range named %r in the marker trace" % name)
        s, e = rs[-1]
        return [d for d in disp if s <= d[0] <= e]

    md = ["# Kernel trace: W4A16 GEMM, 70B-class layers, g = 128, M sweep %s" % bench["config"]["M"], "",
          "Command (`TMPDIR=/tmp`, from the repository root):", "", "```", a.trace_cmd, "```", "",
          "Per case: the kernel the library launched (`launch`), its dispatches inside the",
          "case's range (graph replays over the rotated weight copies), their median",
          "kernel duration (rocprofv3), the bench's event time per launch of the same",
          "replays, and the HBM roofline fraction of the kernel time (algorithmic bytes /",
          "kernel time / 8 TB/s; at M = 128 the bound is the MFMA peak, t_roof / t):", "",
          "| K | N | M | kernel | dispatches | median kernel us | bench us | roofline frac (kernel) |",
          "|---|---|---|---|---|---|---|---|"]
    for c in bench["per_m"]:
        name = "70b w4a16 K=%d N=%d g=%d M=%d" % (c["K"], c["N"], c["group"], c["M"])
        ds = inside(name)
        want = c["launch"].split(" cols=")[0]
        names = {d[2] for d in ds}
        if names != {want}:
            raise SystemExit("case %s: trace has %s, expected %s" % (name, names, want))
        med = statistics.median((d[1] - d[0]) / 1e3 for d in ds)
        troof = R.w4a16_t_roof(c["M"], c["N"], c["K"], c["group"]) * 1e6
        md.append("| %d | %d | %d | `%s` | %d | %.2f | %.2f | %.3f |" % (
            c["K"], c["N"], c["M"], want, len(ds), med, c["us"], troof / med))
    steps = inside("timed steps")
    n_l = bench["config"]["launches_per_step"]
    mean = statistics.fmean((d[1] - d[0]) / 1e3 for d in steps)
    alg = bench["roofline"]["algorithmic_bytes_per_launch"]
    md += ["", "Timed steps: %d dispatches (%d steps x %d launches in the profiled run)." % (
               len(steps), len(steps) // n_l, n_l),
           "Mean kernel duration per launch: %.3f us (rocprofv3); bench.py's HIP-event" % mean,
           "time per launch over the same region: %.3f us (`roofline.avg_launch_us`; it" %
           bench["roofline"]["avg_launch_us"],
           "also holds the dispatch gap between consecutive graph nodes).",
           "Algorithmic bytes per launch (step average) %d: %.1f GB/s of kernel time," % (alg, alg / mean / 1e3),
           "a roofline fraction of %.4f (bench.py, event time: %.4f)." % (
               alg / (mean * 1e-6) / R.HBM_BYTES_PER_S, bench["roofline"]["frac"]), ""]
    open(a.out + "_kernel_trace.md", "w").write("\n".join(md) + "\n")
    print("wrote", a.out + "_kernel_trace.md")


def case_groups(pmc_dir: str, counters: tuple, cases: list, per_case: int) -> list[list[dict]]:
    """The GEMM dispatches of a --profile-cases run, grouped per case:
    dispatch order, per_case consecutive dispatches per case."""
    per = {}
    with open(_one(os.path.join(pmc_dir, "**", "*counter_collection.csv"))) as f:
        for r in csv.DictReader(f):
            if not short(r["Kernel_Name"]).startswith("w4a16_"):
                continue
            d = per.setdefault(int(r["Dispatch_Id"]), {"name": short(r["Kernel_Name"])})
            d[r["Counter_Name"]] = d.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    ds = [per[k] for k in sorted(per)]
    if len(ds) != per_case * len(cases):
        raise SystemExit("%d GEMM dispatches for %d cases x %d" % (len(ds), len(cases), per_case))
    groups = [ds[i * per_case:(i + 1) * per_case] for i in range(len(cases))]
    for c, g in zip(cases, groups):
        want = c["launch"].split(" cols=")[0]
        if {d["name"] for d in g} != {want}:
            raise SystemExit("case %s: dispatches of %s" % (c, {d["name"] for d in g}))
    return groups


CASE_COUNTERS = ("SQ_INSTS_MFMA", "SQ_VALU_MFMA_BUSY_CYCLES", "SQ_INSTS_VALU", "SQ_INSTS_LDS",
                 "SQ_LDS_BANK_CONFLICT", "SQ_WAVES", "GRBM_GUI_ACTIVE")


def case_counter_summary(a, bench: dict) -> None:
    """Matrix-core utilisation and vector work per case (one --pmc pass)."""
    cases, C = bench["cases"], bench["profile_cases"]
    groups = case_groups(a.pmc, CASE_COUNTERS, cases, C)
    simds, xcds = 256 * 4, 8
    md = ["# Matrix-core and vector counters: W4A16 GEMM, %s layers, M sweep" % bench["layers"], "",
          "Command (`TMPDIR=/tmp`, from the repository root; one counter pass, every case",
          "launched %d times in a row):" % C, "", "```", a.pmc_cmd, "```", "",
          "Medians over each case's dispatches.  MFMA utilisation = MFMA busy cycles /",
          "(1024 SIMDs x kernel cycles), kernel cycles = GRBM_GUI_ACTIVE / 8 XCDs: the",
          "fraction of the matrix-core peak at the clock the chip ran.  VALU per MFMA:",
          "the other vector instructions per MFMA instruction (dequantisation, fold).", "",
          "| K | N | g | M | kernel | MFMA / dispatch | MFMA busy | kernel cycles | MFMA util | VALU per MFMA | LDS instr | LDS bank conflicts |",
          "|---|---|---|---|---|---|---|---|---|---|---|---|"]
    for c, g in zip(cases, groups):
        med = {k: statistics.median(d.get(k, 0.0) for d in g) for k in CASE_COUNTERS}
        cyc = med["GRBM_GUI_ACTIVE"] / xcds
        util = med["SQ_VALU_MFMA_BUSY_CYCLES"] / (simds * cyc) if cyc else float("nan")
        other = (med["SQ_INSTS_VALU"] - med["SQ_INSTS_MFMA"]) / med["SQ_INSTS_MFMA"] if med["SQ_INSTS_MFMA"] else 0
        md.append("| %d | %d | %s | %d | `%s` | %.0f | %.3g | %.3g | %.3f | %.2f | %.3g | %.0f |" % (
            c["K"], c["N"], "K" if c["group"] == -1 else c["group"], c["M"], g[0]["name"], med["SQ_INSTS_MFMA"],
            med["SQ_VALU_MFMA_BUSY_CYCLES"], cyc, util, other, med["SQ_INSTS_LDS"], med["SQ_LDS_BANK_CONFLICT"]))
    md.append("")
    open(a.out + "_counters.md", "w").write("\n".join(md) + "\n")
    print("wrote", a.out + "_counters.md")


def case_traffic_summary(a, bench: dict) -> None:
    """HBM bytes per case from a FETCH_SIZE and a WRITE_SIZE pass of
    bench.py --profile-cases, scaled by the passes' calibration copies."""
    import paper_2408_11743_amd.roofline as R
    cases, C = bench["cases"], bench["profile_cases"]
    gf = case_groups(a.fetch, ("FETCH_SIZE",), cases, C)
    gw = case_groups(a.write, ("WRITE_SIZE",), cases, C)
    fetch = counter_per_dispatch(a.fetch, "FETCH_SIZE")
    write = counter_per_dispatch(a.write, "WRITE_SIZE")
    copy_bytes = a.copy_mb * (1 << 20)

    def largest(samples):
        v = [x for n, x in samples if COPY_KERNEL in n]
        return [x for x in v if x >= 0.9 * max(v)] if v else []

    cf, cw = largest(fetch), largest(write)
    if not cf or not cw:
        raise SystemExit("no calibration copies in the counter runs (--calibration-copy-mb)")
    f_scale = copy_bytes / (statistics.median(cf) * 1024.0)
    w_scale = copy_bytes / (statistics.median(cw) * 1024.0)
    md = ["# HBM traffic: %s W4A16 GEMM, %s layers, M sweep (rocprofv3 counters)" % (
              "2:4 sparse" if any(c.get("sparse") for c in cases) else "dense", bench["layers"]), "",
          "Commands (two counter passes, each its own run, `TMPDIR=/tmp`; every case launched",
          "%d times in a row, each launch on the next weight copy):" % C, "", "```",
          a.fetch_cmd, a.write_cmd, "```", "",
          "Calibration: the same runs make plain device copies of %d MiB (the runtime's" % a.copy_mb,
          "copy kernel).  Per copy FETCH_SIZE reads %.0f KiB for %d KiB read (scale x%.3f)," %
          (statistics.median(cf), copy_bytes // 1024, f_scale),
          "WRITE_SIZE %.0f KiB for %d KiB written (scale x%.3f)." % (statistics.median(cw), copy_bytes // 1024, w_scale),
          "", "Per case (median over its dispatches), scaled:", "",
          "| K | N | g | M | kernel | fetch MB | write MB | HBM MB | algorithmic MB | ratio |",
          "|---|---|---|---|---|---|---|---|---|---|"]
    hbm, tot = {}, 0.0
    for c, f, w in zip(cases, gf, gw):
        fb = statistics.median(d["FETCH_SIZE"] for d in f) * 1024.0 * f_scale
        wb = statistics.median(d["WRITE_SIZE"] for d in w) * 1024.0 * w_scale
        alg = (R.sparse24_bytes if c.get("sparse") else R.w4a16_bytes)(c["M"], c["N"], c["K"], c["group"])
        md.append("| %d | %d | %s | %d | `%s` | %.2f | %.2f | %.2f | %.2f | %.3f |" % (
            c["K"], c["N"], "K" if c["group"] == -1 else c["group"], c["M"], f[0]["name"], fb / 1e6, wb / 1e6,
            (fb + wb) / 1e6, alg / 1e6, (fb + wb) / alg))
        hbm["K=%d N=%d g=%d M=%d" % (c["K"], c["N"], c["group"], c["M"])] = round(fb + wb)
        tot += fb + wb
    digest = kernel_sources_digest()
    md += ["", "Algorithmic bytes: K*N/2 + 2*(K/g)*N + 2*M*K + 2*M*N%s." % (
               " (2:4 sparse: K*N/4 of kept codes and K*N/8 of row indices in place of K*N/2)"
               if any(c.get("sparse") for c in cases) else ""), "",
           ("Average per launch over the cases: %.2f MB (measured" if any(c.get("sparse") for c in cases) else
            "Average per launch over the cases: %.2f MB (bench.py reports it as `roofline.traffic`") %
           (tot / len(cases) / 1e6),
           "while the kernel sources (%s under `paper_2408_11743_amd/csrc/`) hash to `%s...`)." %
           (", ".join(KERNEL_SOURCES), digest[:16]), ""]
    open(a.out + "_traffic.md", "w").write("\n".join(md) + "\n")
    rec = {"workload": "W4A16 GEMM, %s layers, M sweep (bench.py --profile-cases)" % bench["layers"],
           "kernel_sources_sha256": digest,
           "counter_scale": {"FETCH_SIZE": round(f_scale, 4), "WRITE_SIZE": round(w_scale, 4),
                             "calibration": "device copies of %d MiB" % a.copy_mb},
           "hbm_bytes_per_launch": hbm, "step_avg_hbm_bytes_per_launch": round(tot / len(cases))}
    json.dump(rec, open(a.out + "_traffic.json", "w"), indent=1)
    print("wrote", a.out + "_traffic.md", a.out + "_traffic.json")


def sparse_summary(a, bench: dict) -> None:
    """Kernel trace of bench.py --only sparse_2of4 (with --marker-trace): per
    M the 2:4 kernel's and the dense kernel's median duration on 8192 x 8192."""
    import paper_2408_11743_amd.roofline as R
    ranges = marker_ranges(a.trace)
    disp = [d for d in dispatches(a.trace) if d[2].startswith("w4a16_")]
    K = N = 8192
    g = 128
    md = ["# Kernel trace: 2:4 sparse W4A16 GEMM, K = N = 8192, g = 128, M sweep", "",
          "Command (`TMPDIR=/tmp`, from the repository root):", "", "```", a.trace_cmd, "```", "",
          "Per M: median kernel duration of the 2:4 kernel and of the dense W4A16 kernel on",
          "the same (pruned) matrix, each over its case's replays, and the 2:4 kernel's",
          "fraction of the HBM roofline of its algorithmic bytes (3/8 byte per weight plus",
          "scales, A and C) in kernel time:", "",
          "| M | 2:4 kernel | median us | dense kernel | median us | speedup | roofline frac (kernel) |",
          "|---|---|---|---|---|---|---|"]
    for c in bench["sparse_2of4"]["per_m"]:
        M = c["M"]
        res = []
        for tag in ("2:4", "dense"):
            rs = [(s, e) for n, s, e in ranges if n == "sparse %s M=%d" % (tag, M)]
            if not rs:
                raise SystemExit("no range for sparse %s M=%d" % (tag, M))
            s, e = rs[-1]
            ds = [d for d in disp if s <= d[0] <= e]
            res.append((sorted({d[2] for d in ds}), statistics.median((d[1] - d[0]) / 1e3 for d in ds)))
        troof = R.sparse24_t_roof(M, N, K, g) * 1e6
        md.append("| %d | `%s` | %.2f | `%s` | %.2f | %.3f | %.3f |" % (
            M, ", ".join(res[0][0]), res[0][1], ", ".join(res[1][0]), res[1][1], res[1][1] / res[0][1],
            troof / res[0][1]))
    md.append("")
    open(a.out + "_kernel_trace.md", "w").write("\n".join(md) + "\n")
    print("wrote", a.out + "_kernel_trace.md")


def main() -> None:
    ap = argparse.ArgumentParser()
    ap.add_argument("--trace")
    ap.add_argument("--pmc", help="one counter pass (prefill counters, or CASE_COUNTERS of --profile-cases)")
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

    bench = json.loads(open(a.bench).read().strip().splitlines()[-1])
    if "profile_cases" in bench:  # bench.py --profile-cases
        if a.pmc:
            case_counter_summary(a, bench)
        else:
            case_traffic_summary(a, bench)
        return
    if "prefill" in bench and "config" not in bench:  # bench.py --only prefill
        if a.pmc:
            prefill_counter_summary(a, bench)
        else:
            prefill_summary(a, bench)
        return
    if not a.trace and not ("quantize" in bench and a.pmc):
        raise SystemExit("--trace is required for this bench output")
    if "quantize" in bench and "config" not in bench:  # bench.py --only quantize
        if a.pmc:
            quantize_counter_summary(a, bench)
        else:
            quantize_summary(a, bench)
        return
    if "sparse_2of4" in bench and "config" not in bench:  # bench.py --only sparse_2of4
        sparse_summary(a, bench)
        return
    headline_trace_summary(a, bench)


if __name__ == "__main__":
    main()
