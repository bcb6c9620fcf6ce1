"""Build libmarlin_mi355x.so (the HIP library) in-tree with hipcc for gfx950.

Each source is compiled to an object of its own (in parallel), then the
objects are linked into the shared library.

Usage: python -m paper_2408_11743_amd.build [--verbose]
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libmarlin_mi355x.so")
SOURCES = ["api.cpp", "plan.cpp", "gemm.hip", "pair.hip", "tile.hip", "wide.hip", "pack.hip", "quant.hip", "noalloc.hip"]
ARCH = "gfx950"

# Packed fp32 instructions are disabled for all device code: plain float code
# is compiled to scalar-per-lane fp32 instructions.
# MFMA results are kept in ordinary vector registers (the kernels have
# registers to spare at one wave per SIMD), so the fp32 fold after each
# stage reads them without accumulator-register moves.
DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                "-mllvm", "-amdgpu-mfma-vgpr-form=1"]
# The wide kernel's accumulators are written by MFMAs only, so it lets the
# compiler place them in the accumulation registers.
SOURCE_FLAGS = {"wide.hip": ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]}
_NOISE = "is not a recognized feature for this target"


def hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    return os.path.join(rocm, "bin", "hipcc")


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    msg = "\n".join(l for l in (r.stdout + r.stderr).splitlines() if _NOISE not in l)
    return r.returncode, msg


def build(verbose: bool = False, out: str = LIB, extra: list[str] | None = None) -> str:
    tmpdir = tempfile.mkdtemp(prefix="marlin_build_")
    try:
        common = ["--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC", "-I", INCLUDE, "-I", CSRC]
        objs, cmds = [], []
        for s in SOURCES:
            obj = os.path.join(tmpdir, s + ".o")
            objs.append(obj)
            flags = SOURCE_FLAGS.get(s, DEVICE_FLAGS)
            cmds.append([hipcc(), *common, *flags, *(extra or []), "-c", "-o", obj, os.path.join(CSRC, s)])
        jobs = min(len(cmds), max(1, min(16, os.cpu_count() or 1)))
        with ThreadPoolExecutor(jobs) as ex:
            results = list(ex.map(lambda c: _run(c, verbose), cmds))
        for (rc, msg), c in zip(results, cmds):
            if msg.strip() and (verbose or rc != 0):
                sys.stderr.write(msg + "\n")
            if rc != 0:
                raise RuntimeError("hipcc failed: %s" % " ".join(c))
        tmp = out + ".tmp%d" % os.getpid()
        rc, msg = _run([hipcc(), "--offload-arch=" + ARCH, "-shared", "-fPIC", "-o", tmp, *objs], verbose)
        if rc != 0:
            sys.stderr.write(msg + "\n")
            raise RuntimeError("hipcc failed linking %s" % out)
        os.replace(tmp, out)
    finally:
        shutil.rmtree(tmpdir, ignore_errors=True)
    return out


if __name__ == "__main__":
    print(build(verbose="--verbose" in sys.argv))
