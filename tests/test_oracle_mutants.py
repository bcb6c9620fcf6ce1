"""Planted mistakes in a copy of the oracle must each trip at least one pin.

Every mutant below is a plausible slip in writing the paper's definition
(Section 3.4): a wrong zero point, a dropped term, a transposed operand, a
wrong group index, a wrong binary16 field, a sign error, an output never
cleared, a missing low-nibble mask.  Each is applied to a temporary copy of
oracle.c on the CPU, compiled with gcc, and the full pin suite runs against
it in a child process (a crash also counts as caught).  The unmodified copy
must pass.
"""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "oracle.c")
PINS = os.path.join(ROOT, "tests", "oracle_pins.py")

MUTANTS = {
    "zero_point_7": [("(double)((qrow[n] & 0xf) - 8)", "(double)((qrow[n] & 0xf) - 7)")],
    "unsigned_code": [("(double)((qrow[n] & 0xf) - 8)", "(double)((qrow[n] & 0xf))")],
    "sign_flip": [("crow[n] += a * w;", "crow[n] -= a * w;")],
    "drop_last_k": [("for (int64_t k = 0; k < K; ++k) {\n                const double a",
                     "for (int64_t k = 0; k < K - 1; ++k) {\n                const double a")],
    "skip_first_k": [("for (int64_t k = 0; k < K; ++k) {\n                const double a",
                      "for (int64_t k = 1; k < K; ++k) {\n                const double a")],
    "group_mod": [("return k / g;", "return k % g;")],
    "group_off_by_one": [("return k / g;", "return (k + 1) / g;")],
    "scales_transposed": [("const double w = srow[n] *",
                           "const double w = sd[n * G + scale_row(k, K, g)] *")],
    "codes_transposed": [("const uint8_t *qrow = q + k * N;",
                          "const uint8_t *qrow = q + (k % N) * N;")],
    "a_wrong_row": [("const double a = Ad[m * K + k];", "const double a = Ad[k];")],
    "no_clear": [("for (int64_t n = n0; n < n1; ++n) crow[n] = 0.0;", "")],
    "no_nibble_mask": [("(double)((qrow[n] & 0xf) - 8)", "(double)((qrow[n]) - 8)")],
    "f16_bias": [("v = ldexp((double)(1024 + f), e - 25);", "v = ldexp((double)(1024 + f), e - 24);")],
    "f16_subnormal": [("v = ldexp((double)f, -24);", "v = ldexp((double)f, -25);")],
    "f16_no_sign": [("return sign ? -v : v;", "return v;")],
    "dequant_zero_point": [("(double)(code - 8)", "(double)(code - 9)")],
    "sampled_group": [("s[scale_row(k, K, g) * N + n]", "s[scale_row(k, K, g) * N + (n ^ 1)]")],
    "ragged_groups_floor": [("const int64_t G = (g <= 0 || g >= K) ? 1 : (K + g - 1) / g;",
                             "const int64_t G = (g <= 0 || g >= K) ? 1 : K / g;\n    if (K % g) return;")],
}


def _build(tmpdir, name, edits):
    src = open(SRC).read()
    for old, new in edits:
        assert old in src, (name, old)
        src = src.replace(old, new)
    c = os.path.join(tmpdir, name + ".c")
    so = os.path.join(tmpdir, name + ".so")
    open(c, "w").write(src)
    subprocess.run(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c99", "-o", so, c, "-lm"],
                   check=True)
    return so


def _run_pins(so):
    env = dict(os.environ, OMP_NUM_THREADS="2")
    r = subprocess.run([sys.executable, PINS, so], capture_output=True, text=True, timeout=300,
                       env=env)
    return r.returncode, r.stdout + r.stderr


@pytest.fixture(scope="module")
def tmpdir_mod(tmp_path_factory):
    d = tmp_path_factory.mktemp("mutants")
    yield str(d)
    shutil.rmtree(str(d), ignore_errors=True)


def test_unmodified_copy_passes(tmpdir_mod):
    rc, out = _run_pins(_build(tmpdir_mod, "clean", []))
    assert rc == 0, out


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(tmpdir_mod, name):
    rc, out = _run_pins(_build(tmpdir_mod, name, MUTANTS[name]))
    assert rc != 0, "planted mistake %s passed every pin:\n%s" % (name, out)
