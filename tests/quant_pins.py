"""Pins of the quantiser oracle: facts fixed by the definition (symmetric
uniform quantisation with zero point 8, Section 2.2 Eq. 1; group-wise
clipping search, Section 3.5), checked without re-deriving its formula.

Each pin takes a ``quantize(W, group, ratios) -> (q, s)`` implementation, so
the same pins run on the oracle and on planted-mistake copies of it.

* ``representable``: weights that are exactly s0 * (c - 8) for a power-of-two
  s0 and codes c that reach 0 in every group come back as (c, s0) once the
  ratio 15/16 is offered (the range [-7.5 s0, 7.5 s0] has steps of exactly
  s0) and the search must prefer it over the ratio 1, whose error is > 0.
* ``rtn_bound``: with the ratio 1 alone nothing is clipped, so every weight is
  within half a step of its reconstruction (plus at most 7.5 * 2^-11 steps
  where the fp16 rounding of s shrank the range), and the range is the
  largest weight's magnitude (to the fp16 rounding of s).
* ``search``: the chosen ratio's error (fp64) is the smallest of the errors of
  each ratio run alone, and never above plain rounding's.
* ``zero``: a zero group has s = 0 and every code 8.
* ``scaling``: multiplying W by 4 multiplies s by 4 and keeps q (powers of two
  commute with every rounding step away from under/overflow).
* ``per_channel``: group -1 and group K agree.
* ``exact_rounding``: every code is the exact quotient v/s of the fp16 inputs
  rounded to the nearest integer (half to even) and clamped to -8..7, checked
  with exact rationals for every weight whose quotient is not within 2^-16 of
  a half-integer.  That window is the tie set: the oracle (and the kernel)
  divide by multiplying with the fp32 reciprocal of s, which is within
  2^-22 of v/s for |v/s| < 16, so outside the window both roundings agree
  and inside it either neighbour may be taken.
"""
from __future__ import annotations

import math
from fractions import Fraction

import numpy as np

from oracle.quant import group_errors_f64

CLIP = tuple(1.0 - 0.05 * i for i in range(10))


def _weights(seed, K, N):
    rng = np.random.default_rng([seed, 77, K, N])
    sigma = rng.uniform(0.5, 1.5, size=(1, N)) / np.sqrt(K)
    w = rng.standard_t(5, size=(K, N)) * sigma
    return w.astype(np.float16)


def pin_representable(quantize):
    rng = np.random.default_rng(11)
    K, N, g = 256, 24, 128
    c = rng.integers(0, 16, size=(K, N))
    c[::g, :] = 0  # every group reaches the code 0 (weight -8 s0)
    e = rng.integers(-9, -3, size=(K // g, N))
    s0 = np.ldexp(1.0, e).astype(np.float16)
    W = (np.repeat(s0.astype(np.float64), g, axis=0) * (c - 8)).astype(np.float16)
    for ratios in ([1.0, 15.0 / 16.0], [15.0 / 16.0, 1.0], [15.0 / 16.0]):
        q, s = quantize(W, g, ratios)
        assert np.array_equal(s.astype(np.float64), s0.astype(np.float64)), ("scale", ratios)
        assert np.array_equal(q.astype(np.int64), c), ("codes", ratios)
    # the ratio 1 alone cannot reproduce them (its step is 16/15 s0)
    q1, s1 = quantize(W, g, [1.0])
    assert (group_errors_f64(W, g, q1, s1) > 0).all()


def pin_rtn_bound(quantize):
    for K, N, g in [(256, 40, 128), (384, 16, -1)]:
        W = _weights(3, K, N)
        q, s = quantize(W, g, [1.0])
        assert q.dtype == np.uint8 and q.max() <= 15
        gg = K if g == -1 else g
        S = np.repeat(s.astype(np.float64), gg, axis=0)
        err = np.abs(W.astype(np.float64) - S * (q.astype(np.float64) - 8.0))
        # half a step, plus what the clamp adds where s rounded down in fp16
        # (by at most 2^-11 relative) and the largest weight lies up to
        # 7.5 * 2^-11 steps beyond the code 7
        assert (err <= 0.5 * S * (1 + 15 * 2.0 ** -11)).all(), "rounding error beyond half a step"
        amax = np.abs(W.astype(np.float64)).reshape(K // gg, gg, N).max(axis=1)
        assert (7.5 * s.astype(np.float64) >= amax * (1 - 2.0 ** -10)).all(), "range does not cover max|v|"
        assert (7.5 * s.astype(np.float64) <= amax * (1 + 2.0 ** -10)).all(), "range wider than max|v|"


def pin_search(quantize):
    K, N, g = 256, 48, 128
    W = _weights(5, K, N)
    q, s = quantize(W, g, CLIP)
    chosen = group_errors_f64(W, g, q, s)
    alone = np.stack([group_errors_f64(W, g, *quantize(W, g, [r])) for r in CLIP])
    assert (chosen <= alone.min(axis=0) * (1 + 1e-5) + 1e-30).all(), "not the smallest error"
    assert (chosen <= alone[0] * (1 + 1e-5) + 1e-30).all(), "worse than plain rounding"
    # the chosen (q, s) is the one of some ratio run alone
    hits = np.zeros(chosen.shape, dtype=bool)
    for r in CLIP:
        qr, sr = quantize(W, g, [r])
        same_s = sr == s
        same_q = (qr == q).reshape(K // g, g, N).all(axis=1)
        hits |= same_s & same_q
    assert hits.all()
    # clipping helps on heavy-tailed weights
    assert chosen.sum() < alone[0].sum()


def pin_zero(quantize):
    W = _weights(7, 256, 16)
    W[128:, 3] = 0
    W[:, 5] = 0
    q, s = quantize(W, 128, CLIP)
    assert s[1, 3] == 0 and s[0, 5] == 0 and s[1, 5] == 0
    assert (q[128:, 3] == 8).all() and (q[:, 5] == 8).all()
    assert (s[:, [0, 1, 2, 4]] > 0).all()


def pin_scaling(quantize):
    W = _weights(9, 256, 32)
    q, s = quantize(W, 128, CLIP)
    q4, s4 = quantize((W.astype(np.float32) * 4).astype(np.float16), 128, CLIP)
    assert np.array_equal(q, q4)
    assert np.array_equal(s4.astype(np.float32), s.astype(np.float32) * 4)


def pin_per_channel(quantize):
    W = _weights(13, 384, 16)
    a = quantize(W, -1, CLIP)
    b = quantize(W, 384, CLIP)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1]) and a[1].shape == (1, 16)


def pin_exact_rounding(quantize):
    K, N, g = 256, 12, 128
    W = _weights(21, K, N)
    q, s = quantize(W, g, CLIP)
    window = Fraction(1, 1 << 16)
    checked = ties = 0
    for j in range(K // g):
        for n in range(N):
            sv = Fraction(float(s[j, n]))
            rows = range(j * g, (j + 1) * g)
            if sv == 0:
                assert all(q[k, n] == 8 for k in rows)
                continue
            for k in rows:
                x = Fraction(float(W[k, n])) / sv
                fl = math.floor(x)
                frac = x - fl
                if abs(frac - Fraction(1, 2)) <= window:
                    ties += 1
                    continue
                code = min(max(fl + (1 if frac > Fraction(1, 2) else 0), -8), 7) + 8
                assert int(q[k, n]) == code, ("code", k, n, float(x), int(q[k, n]), code)
                checked += 1
    assert checked >= 0.99 * K * N and ties <= 0.01 * K * N, (checked, ties)


PINS = [pin_representable, pin_rtn_bound, pin_search, pin_zero, pin_scaling, pin_per_channel, pin_exact_rounding]


def run_all(quantize):
    for p in PINS:
        p(quantize)
