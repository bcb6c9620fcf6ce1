"""Byte / FLOP accounting of the bench, pinned to figures the paper prints."""
import json
import os

import pytest

from paper_2408_11743_amd import roofline as R

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_constants.json")))


def test_ideal_speedup_matches_paper():
    # Section 5.1: the maximum 3.87x at 4 bits and group size 128
    c = GOLD["ideal_speedup_4bit_g128"]
    x = R.ideal_weight_speedup(c["bits"], c["group"], c["scale_bits"])
    assert abs(x - c["value"]) < 0.01
    assert x > c["value"]  # the paper truncates 3.878


def test_ideal_speedup_equals_byte_ratio_for_large_layer():
    # the same ratio falls out of the full byte counts when A and C vanish
    K = N = 1 << 15
    r = R.fp16_bytes(1, N, K) / R.w4a16_bytes(1, N, K, 128)
    assert abs(r - R.ideal_weight_speedup(4, 128)) < 1e-3


def test_b_opt_matches_paper():
    # Section 3.1: FLOP/byte ratio about 200 on the A10 gives b_opt about 50,
    # with 100 FLOPs per 4-bit weight load
    assert R.b_opt(GOLD["a10_flop_per_byte"]["value"], bits=4) == GOLD["a10_b_opt"]["value"]
    assert GOLD["a10_flop_per_byte"]["value"] * 0.5 == GOLD["a10_flops_per_4bit_weight_load"]["value"]


def test_memory_bits_formula_matches_paper():
    # Section 3.4: 16MK + 4KN + 16MN bits
    formula = GOLD["memory_bits_formula"]["value"]
    for (M, N, K) in [(1, 4096, 4096), (16, 11008, 4096), (128, 8192, 28672)]:
        assert R.paper_memory_bits(M, N, K) == eval(formula, {"M": M, "N": N, "K": K})
        # scales add exactly 2 bytes per (group, column)
        assert R.w4a16_bytes(M, N, K, 128) - R.paper_memory_bits(M, N, K) / 8 == 2 * (K // 128) * N


def test_flops_and_roofline_regimes():
    assert R.flops(16, 4096, 4096) == 2 * 16 * 4096 * 4096
    # on MI355X the ridge at g = 128 sits near M = 81: M <= 64 is HBM-bound
    assert 75 < R.ridge_m(128) < 85
    assert R.bound(64, 4096, 4096, 128) == "hbm"
    assert R.bound(128, 4096, 4096, 128) == "mfma"


@pytest.mark.parametrize("M,us", [(1, 1.083), (16, 1.114), (32, 1.147)])
def test_t_roof_values_4096(M, us):
    # 4096 x 4096, g = 128: bytes / 8 TB/s
    assert abs(R.w4a16_t_roof(M, 4096, 4096, 128) * 1e6 - us) < 2e-3
