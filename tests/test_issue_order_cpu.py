"""The kernels wait for their direct-to-LDS loads by counting the vector-memory
operations issued after them (which complete in order): the stream and
sparse kernels wait for a stage's activation rows while its weight and scale
loads and D - 1 later stages may still be in flight; the tile kernel waits
for a stage's activation and weight blocks while its scale loads and P - 2
later stages may be; the wide kernel waits for a stage's activation rows and
scales while its weight loads and P - 2 later stages may be.  That holds only if the compiler emits each stage's
loads as one group, direct-to-LDS loads first, in issue order.  The compiler
may interleave independent loads (it once moved a weight load between the
activation loads of a stage, and reading rows before their load had landed
gave wrong outputs), so the kernels pin the order; this test compiles the
kernel sources for gfx950 and checks, for every instantiation, that the
buffer loads form identical stage groups of the size the waits assume.

The same assembly pins the memory-coherence bits the cross-work-group
combination relies on (device-coherent slot stores and loads, a returning
atomic for the arrival count, no whole-cache maintenance).
"""
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2408_11743_amd", "csrc")


def _hipcc():
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    p = os.path.join(rocm, "bin", "hipcc")
    return p if os.path.exists(p) else shutil.which("hipcc")


@pytest.fixture(scope="module")
def assembly(tmp_path_factory):
    hipcc = _hipcc()
    if not hipcc:
        pytest.skip("hipcc not available")
    d = tmp_path_factory.mktemp("asm")
    procs = {}
    from paper_2408_11743_amd import build as B
    for src in ("gemm", "pair", "tile", "wide"):
        out = str(d / (src + ".s"))
        flags = B.SOURCE_FLAGS.get(src + ".hip", B.DEVICE_FLAGS)
        cmd = [hipcc, "--offload-arch=gfx950", "-O3", "-std=c++17", "-I", os.path.join(ROOT, "include"), "-I", CSRC,
               *flags, "--cuda-device-only", "-S", "-o", out, os.path.join(CSRC, src + ".hip")]
        procs[src] = (subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.PIPE), out)
    text = {}
    for src, (pr, out) in procs.items():
        _, err = pr.communicate()
        assert pr.returncode == 0, err.decode()[-2000:]
        text[src] = open(out).read()
    return text


def _kernels(text):
    for m in re.finditer(r"^(_ZN6marlin\S*(w4a16_(?:stream|sparse|tile|wide|pair)_kernel)I((?:Li\d+E)*)Lb(\d)E\S*):",
                         text, re.M):
        body = text[m.end():text.index(".Lfunc_end", m.end())]
        ints = [int(x) for x in re.findall(r"Li(\d+)E", m.group(3))]
        yield m.group(1), m.group(2), ints, m.group(4) == "1", body


def _expected_group(kind, ints, per_channel):
    if kind == "w4a16_pair_kernel":  # half of a block's 16 row loads, 4 weight words, 2 scale runs
        return "L" * 8 + "R" * (4 + (0 if per_channel else 2))
    if kind == "w4a16_wide_kernel":
        MBW, NBW, P = ints
        return "L" * (MBW + (0 if per_channel else 1)) + "R" * NBW
    if kind == "w4a16_tile_kernel":
        WN, WM, MBW, NBW, KS = ints
        NW, TR = WN * WM, 16 * MBW * WM
        dma_a, dma_w, scale = TR // (4 * NW), NBW // WM, (2 if NBW == 4 else 1)
        return "L" * (KS * (dma_a + dma_w)) + "R" * (scale if per_channel else KS * scale)
    MB, NB, D, AR, KW = ints
    weights = (6 if NB == 8 else 3 if NB == 4 else 2) if kind == "w4a16_sparse_kernel" else NB
    return "L" * AR + "R" * (weights + (0 if per_channel else (NB + 1) // 2))


def test_every_kernel_issues_its_loads_in_stage_groups(assembly):
    n = 0
    bad = []
    for src, text in assembly.items():
        for name, kind, ints, pc, body in _kernels(text):
            seq = "".join("L" if " lds" in line else "R" for line in body.splitlines()
                          if "buffer_load" in line and not line.strip().startswith(";"))
            group = _expected_group(kind, ints, pc)
            n += 1
            if not seq or len(seq) % len(group) or seq != group * (len(seq) // len(group)):
                bad.append("%s: expected groups %s, got %s" % (name, group, seq))
    assert n >= 100, "kernels not found in the assembly (%d)" % n
    assert not bad, "\n".join(bad)


def test_combination_uses_device_coherent_accesses(assembly):
    # Tiles shared by several work-groups are combined through fp32 slots in
    # the workspace and one arrival counter per tile.  The slots are written
    # and read with relaxed agent-scope atomics, which must come out as plain
    # dword stores and loads carrying the device-coherence bit (sc1), so they
    # bypass the per-XCD L2s' incoherence without any whole-cache writeback or
    # invalidate; the arrival is an atomic add that returns the old count
    # (sc0), which decides the reducer.  Nothing else in the kernels uses
    # dword global stores or loads (C is written as 8-byte stores).
    n = 0
    bad = []
    for src, text in assembly.items():
        for name, kind, ints, pc, body in _kernels(text):
            n += 1
            lines = [l.strip() for l in body.splitlines() if l.strip() and not l.strip().startswith(";")]
            stores = [l for l in lines if l.startswith("global_store_dword ")]
            loads = [l for l in lines if l.startswith("global_load_dword ")]
            atomics = [l for l in lines if "atomic" in l.split()[0]]
            if not stores or not loads or not atomics:
                bad.append("%s: no combination code found" % name)
            bad += ["%s: %s" % (name, l) for l in stores + loads if not l.endswith(" sc1")]
            bad += ["%s: %s" % (name, l) for l in atomics
                    if not (l.startswith("global_atomic_add ") and l.endswith(" sc0"))]
            bad += ["%s: %s" % (name, l) for l in lines if l.split()[0] in ("buffer_wbl2", "buffer_inv")]
    assert n >= 100, "kernels not found in the assembly (%d)" % n
    assert not bad, "\n".join(bad[:20])
