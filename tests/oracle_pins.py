"""Pins that tie the FP64 oracle to facts other than itself.

Each pin takes a loaded oracle library (ctypes handle) and raises
AssertionError when the oracle disagrees with what the paper and the
mathematics fix.  ``tests/test_oracle_pins.py`` runs them on the real oracle;
``tests/test_oracle_mutants.py`` runs them on copies of the oracle source with
planted mistakes and checks that every mistake trips at least one pin.

Run as a script (``python tests/oracle_pins.py LIB.so``) it executes every pin
against that library and exits 0 only if all pass.

What each pin stands on:
  f16_decode       numpy's binary16 -> binary64 conversion (a library routine)
  exact_rational   brute-force exact rational arithmetic on tiny shapes
  identity         q = 8 + I, s = 1 gives C = A (closed form)
  zero             q = 8 gives C = 0 for any A, s (closed form)
  one_hot          one-hot rows of A pick single weights: C[m,n] = s[r,n]*(q[k,n]-8)
                   at chosen k on group boundaries, non-square shapes, ragged K
  integer_sums     A = 1, s = 1 gives column sums of (q - 8) (numpy integer sum);
                   high nibbles of the code bytes are ignored
  power_of_two     scaling s by 2 scales C by exactly 2
  group_channel    equal group scales equal one per-channel scale
  linearity        C(A1 + A2) = C(A1) + C(A2) with exactly representable data
  blas             C matches numpy's fp64 matmul of A with the dequantised W
  dequant          s = 1 gives q - 8; q = 9 gives the group-expanded scales
  sampled          the sampled routine equals the full routine bit for bit
  sparse24         2:4 sparse weights: the exact sum over kept entries only equals
                   the oracle on the dense codes with code 8 at pruned entries
"""
from __future__ import annotations

import ctypes
import sys
from fractions import Fraction

import numpy as np

vp = ctypes.c_void_p


def _p(a):
    return a.ctypes.data_as(vp)


def _bind(lib):
    i64 = ctypes.c_int64
    lib.oracle_f16_to_f64.argtypes = [ctypes.c_uint16]
    lib.oracle_f16_to_f64.restype = ctypes.c_double
    lib.oracle_dequant.argtypes = [vp, vp, i64, i64, i64, vp]
    lib.oracle_dequant.restype = None
    lib.oracle_gemm.argtypes = [vp, vp, vp, i64, i64, i64, i64, vp]
    lib.oracle_gemm.restype = None
    lib.oracle_gemm_sampled.argtypes = [vp, vp, vp, i64, i64, i64, i64, vp, vp, i64, vp]
    lib.oracle_gemm_sampled.restype = None
    return lib


def _gemm(lib, A, q, s, g):
    """Call the oracle with C pre-filled with NaN (so an unwritten output shows)."""
    A = np.ascontiguousarray(A, dtype=np.float16).view(np.uint16)
    q = np.ascontiguousarray(q, dtype=np.uint8)
    s = np.ascontiguousarray(s, dtype=np.float16).view(np.uint16)
    M, K = A.shape
    N = q.shape[1]
    C = np.full((M, N), np.nan)
    lib.oracle_gemm(_p(A), _p(q), _p(s), M, N, K, g, _p(C))
    return C


def _dequant(lib, q, s, g):
    q = np.ascontiguousarray(q, dtype=np.uint8)
    s = np.ascontiguousarray(s, dtype=np.float16).view(np.uint16)
    K, N = q.shape
    w = np.full((K, N), np.nan)
    lib.oracle_dequant(_p(q), _p(s), K, N, g, _p(w))
    return w


def _rng(*key):
    return np.random.default_rng(list(key))


def _rand_inputs(rng, M, K, N, G):
    A = rng.standard_normal((M, K)).astype(np.float16)
    q = rng.integers(0, 16, size=(K, N), dtype=np.uint8)
    s = rng.uniform(0.01, 0.05, size=(G, N)).astype(np.float16)
    return A, q, s


def pin_f16_decode(lib):
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    ref = bits.view(np.float16).astype(np.float64)
    got = np.array([lib.oracle_f16_to_f64(int(b)) for b in bits])
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan), "NaN patterns differ"
    assert np.array_equal(got[~nan], ref[~nan]), "binary16 decode differs from numpy"
    # signed zeros keep their sign
    assert np.array_equal(np.signbit(got[~nan]), np.signbit(ref[~nan]))


def pin_exact_rational(lib):
    cases = [(1, 128, 1, 128), (2, 256, 8, 128), (3, 128, 16, 128), (2, 256, 8, 256),
             (3, 200, 8, 128), (2, 256, 4, 64)]
    for ci, (M, K, N, g) in enumerate(cases):
        G = -(-K // g)
        for mode in ("random", "low", "high"):
            rng = _rng(7, ci, len(mode))
            A, q, s = _rand_inputs(rng, M, K, N, G)
            if mode == "low":
                q[:] = 0
            elif mode == "high":
                q[:] = 15
            C = _gemm(lib, A, q, s, g)
            Af = [[Fraction(float(x)) for x in row] for row in A.astype(np.float64)]
            sf = [[Fraction(float(x)) for x in row] for row in s.astype(np.float64)]
            for m in range(M):
                for n in range(N):
                    terms = [Af[m][k] * sf[k // g][n] * (int(q[k, n]) - 8) for k in range(K)]
                    exact = sum(terms, Fraction(0))
                    bound = K * 2.0 ** -52 * float(sum(abs(t) for t in terms))
                    err = abs(Fraction(C[m, n]) - exact) if np.isfinite(C[m, n]) else float("inf")
                    assert err <= bound, (ci, mode, m, n, float(exact), C[m, n])


def pin_identity(lib):
    for K, g in ((256, 128), (384, 384), (256, 64)):
        rng = _rng(11, K, g)
        M = 5
        A = rng.standard_normal((M, K)).astype(np.float16)
        q = np.full((K, K), 8, dtype=np.uint8) + np.eye(K, dtype=np.uint8)
        s = np.ones((K // g, K), dtype=np.float16)
        C = _gemm(lib, A, q, s, g)
        assert np.array_equal(C, A.astype(np.float64)), "identity weights must reproduce A"


def pin_zero(lib):
    rng = _rng(13)
    A, q, s = _rand_inputs(rng, 4, 256, 32, 2)
    q[:] = 8
    C = _gemm(lib, A, q, s, 128)
    assert np.array_equal(C, np.zeros_like(C)), "code 8 is weight zero"


def pin_one_hot(lib):
    for (M, K, N, g, ks) in ((6, 384, 24, 128, [0, 127, 128, 255, 256, 383]),
                             (4, 200, 8, 128, [0, 127, 128, 199]),
                             (3, 512, 16, 512, [0, 300, 511])):
        G = -(-K // g)
        rng = _rng(17, K, N)
        _, q, s = _rand_inputs(rng, M, K, N, G)
        s = rng.uniform(0.5, 2.0, size=(G, N)).astype(np.float16)
        A = np.zeros((M, K), dtype=np.float16)
        for m, k in enumerate(ks):
            A[m, k] = 1.0
        C = _gemm(lib, A, q, s, g)
        for m, k in enumerate(ks):
            want = s[k // g].astype(np.float64) * (q[k].astype(np.int64) - 8)
            assert np.array_equal(C[m], want), ("one-hot row", K, g, m, k)


def pin_integer_sums(lib):
    rng = _rng(19)
    K, N = 384, 40
    q = rng.integers(0, 16, size=(K, N), dtype=np.uint8)
    A = np.ones((2, K), dtype=np.float16)
    A[1] = -1.0
    s = np.ones((K // 128, N), dtype=np.float16)
    want = q.astype(np.int64).sum(axis=0) - 8 * K
    C = _gemm(lib, A, q, s, 128)
    assert np.array_equal(C[0], want.astype(np.float64))
    assert np.array_equal(C[1], -want.astype(np.float64))
    # only the low nibble of each byte is the code
    C2 = _gemm(lib, A, q | np.uint8(0xA0), s, 128)
    assert np.array_equal(C2, C), "high nibble must be ignored"
    # per-group power-of-two scales: C = sum_r s_r * (column sum over group r)
    s = np.array([[0.5], [2.0], [4.0]], dtype=np.float16).repeat(N, axis=1)
    per_group = (q.astype(np.int64) - 8).reshape(3, 128, N).sum(axis=1)
    want = (s.astype(np.float64) * per_group).sum(axis=0)
    C = _gemm(lib, A[:1], q, s, 128)
    assert np.array_equal(C[0], want)


def pin_power_of_two(lib):
    rng = _rng(23)
    A, q, s = _rand_inputs(rng, 3, 256, 16, 2)
    C1 = _gemm(lib, A, q, s, 128)
    C2 = _gemm(lib, A, q, (s.astype(np.float32) * 2).astype(np.float16), 128)
    assert np.array_equal(C2, 2 * C1)


def pin_group_channel(lib):
    rng = _rng(29)
    A, q, _ = _rand_inputs(rng, 3, 384, 16, 1)
    row = rng.uniform(0.01, 0.05, size=(1, 16)).astype(np.float16)
    Cg = _gemm(lib, A, q, np.repeat(row, 3, axis=0), 128)
    Cc = _gemm(lib, A, q, row, 384)
    assert np.array_equal(Cg, Cc)


def pin_linearity(lib):
    rng = _rng(31)
    K, N = 256, 16
    A1 = rng.integers(-8, 8, size=(3, K)).astype(np.float16)
    A2 = rng.integers(-8, 8, size=(3, K)).astype(np.float16)
    q = rng.integers(0, 16, size=(K, N), dtype=np.uint8)
    s = (2.0 ** rng.integers(-4, 3, size=(2, N))).astype(np.float16)
    C12 = _gemm(lib, (A1.astype(np.float32) + A2.astype(np.float32)).astype(np.float16), q, s, 128)
    assert np.array_equal(C12, _gemm(lib, A1, q, s, 128) + _gemm(lib, A2, q, s, 128))


def pin_dequant(lib):
    rng = _rng(37)
    K, N = 256, 24
    q = rng.integers(0, 16, size=(K, N), dtype=np.uint8)
    w = _dequant(lib, q, np.ones((2, N), dtype=np.float16), 128)
    assert np.array_equal(w, q.astype(np.float64) - 8)
    s = rng.uniform(0.5, 2.0, size=(2, N)).astype(np.float16)
    w = _dequant(lib, np.full((K, N), 9, dtype=np.uint8), s, 128)
    assert np.array_equal(w, np.repeat(s.astype(np.float64), 128, axis=0))


def pin_blas(lib):
    rng = _rng(41)
    M, K, N = 16, 512, 256
    A, q, s = _rand_inputs(rng, M, K, N, 4)
    C = _gemm(lib, A, q, s, 128)
    W = _dequant(lib, q, s, 128)
    ref = A.astype(np.float64) @ W
    assert np.allclose(C, ref, rtol=1e-12, atol=1e-13)


def pin_sampled(lib):
    rng = _rng(43)
    M, K, N = 5, 384, 64
    A, q, s = _rand_inputs(rng, M, K, N, 3)
    C = _gemm(lib, A, q, s, 128)
    mi = np.array([0, 4, 2, 3, 1], dtype=np.int64)
    ni = np.array([0, 63, 17, 32, 5], dtype=np.int64)
    out = np.full(5, np.nan)
    Au = np.ascontiguousarray(A).view(np.uint16)
    su = np.ascontiguousarray(s).view(np.uint16)
    lib.oracle_gemm_sampled(_p(Au), _p(q), _p(su), M, N, K, 128, _p(mi), _p(ni), 5, _p(out))
    assert np.array_equal(out, C[mi, ni])


def pin_sparse24(lib):
    # 2:4 sparse weights (Section 4): the product over the kept entries only,
    # in exact rationals, equals the oracle on the dense code matrix whose
    # pruned entries hold code 8 (weight 0), within the summation bound.
    for ci, (M, K, N, g) in enumerate([(2, 128, 8, 128), (3, 256, 4, 128), (1, 256, 16, 256)]):
        rng = _rng(31, ci)
        G = -(-K // g)
        A, q, s = _rand_inputs(rng, M, K, N, G)
        pat = np.array([[1, 1, 0, 0], [1, 0, 1, 0], [1, 0, 0, 1], [0, 1, 1, 0], [0, 1, 0, 1], [0, 0, 1, 1]], bool)
        keep = pat[rng.integers(0, 6, size=(K // 4, N))].transpose(0, 2, 1).reshape(K, N)
        qd = np.where(keep, q, np.uint8(8)).astype(np.uint8)
        C = _gemm(lib, A, qd, s, g)
        Af = [[Fraction(float(x)) for x in row] for row in A.astype(np.float64)]
        sf = [[Fraction(float(x)) for x in row] for row in s.astype(np.float64)]
        for m in range(M):
            for n in range(N):
                terms = [Af[m][k] * sf[k // g][n] * (int(q[k, n]) - 8) for k in range(K) if keep[k, n]]
                exact = sum(terms, Fraction(0))
                bound = K * 2.0 ** -52 * float(sum(abs(t) for t in terms))
                assert abs(Fraction(C[m, n]) - exact) <= bound, (ci, m, n)


PINS = [pin_f16_decode, pin_exact_rational, pin_identity, pin_zero, pin_one_hot,
        pin_integer_sums, pin_power_of_two, pin_group_channel, pin_linearity,
        pin_dequant, pin_blas, pin_sampled, pin_sparse24]


def run_all(lib_path: str) -> list[str]:
    lib = _bind(ctypes.CDLL(lib_path))
    failed = []
    for pin in PINS:
        try:
            pin(lib)
        except AssertionError:
            failed.append(pin.__name__)
    return failed


if __name__ == "__main__":
    bad = run_all(sys.argv[1])
    print("failed pins:", bad)
    sys.exit(1 if bad else 0)
