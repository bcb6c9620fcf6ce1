"""The quantiser oracle against its pins, and planted mistakes in copies of it.

Each mutant is a plausible slip in writing the definition (symmetric uniform
quantisation with zero point 8, Section 2.2 Eq. 1, and the group-wise
clipping search, Section 3.5): a wrong zero point, step count or rounding
(floor, truncation), a
clamp that loses the code 0, a search that keeps the worst ratio or ignores
the ratio, a dropped or sign-flipped error term, a range taken without the
magnitude.  Each copy of ``oracle/quant.py`` must fail at least one pin; the
unmodified copy must pass.
"""
import importlib.util
import os

import pytest

import quant_pins
from oracle import quant as oracle_quant

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "quant.py")

MUTANTS = {
    "zero_point_7": [("q = (t + _F(8))", "q = (t + _F(7))")],
    "sixteen_steps": [("s16 = ((a + a) / _F(15))", "s16 = ((a + a) / _F(16))")],
    "step_a_over_8": [("s16 = ((a + a) / _F(15))", "s16 = (a / _F(8))")],
    "floor_rounding": [("t = np.clip(np.rint(v * inv)", "t = np.clip(np.floor(v * inv)")],
    "truncation": [("t = np.clip(np.rint(v * inv)", "t = np.clip(np.trunc(v * inv)")],
    "clamp_loses_code_0": [("_F(-8), _F(7))", "_F(-7), _F(7))")],
    "keeps_worst_ratio": [("better = err < best_err", "better = (err > best_err) | np.isinf(best_err)")],
    "ratio_ignored": [("a = r * amax", "a = amax")],
    "error_sign": [("d = v - _codes(v, sf, inv) * sf", "d = v + _codes(v, sf, inv) * sf")],
    "error_drops_last_row": [("for k in range(g):  # the group's rows", "for k in range(g - 1):  # the group's rows")],
    "range_without_magnitude": [("amax = np.abs(V).max(axis=1)", "amax = V.max(axis=1)")],
    "group_transposed": [("V = W.astype(_F).reshape(G, g, N)", "V = W.astype(_F).reshape(g, G, N).transpose(1, 0, 2)")],
}


def _load(tmp_path, name, edits):
    src = open(SRC).read()
    for old, new in edits:
        assert old in src, (name, old)
        src = src.replace(old, new)
    path = tmp_path / (name + ".py")
    path.write_text(src)
    spec = importlib.util.spec_from_file_location("quant_" + name, str(path))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


@pytest.mark.parametrize("pin", quant_pins.PINS, ids=lambda p: p.__name__)
def test_oracle_meets_pin(pin):
    pin(oracle_quant.quantize)


def test_unmodified_copy_passes(tmp_path):
    quant_pins.run_all(_load(tmp_path, "same", []).quantize)


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(tmp_path, name):
    q = _load(tmp_path, name, MUTANTS[name]).quantize
    with pytest.raises(Exception):
        quant_pins.run_all(q)
