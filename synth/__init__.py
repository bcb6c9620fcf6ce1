"""Seeded synthetic workloads shared by the oracle tests, the GPU tests and the bench.

This module draws random numbers and nothing else: it holds none of the
method's arithmetic (no dequantisation, no product, no layout).  Both the
oracle side and the HIP side receive exactly these arrays.

Workload recipe (the value distributions of the paper's decode-time layers,
Section 3.4 "Kernel Design", with the shapes of the Llama-2-7B / 70B-class
layers the paper benchmarks in Section 5.1):

* activations A: fp16 [M, K], A ~ N(0, 1) drawn in fp64 and rounded to fp16
  (round-to-nearest-even, numpy's cast);
* weights: int4 codes q ~ U{0..15} stored one code per byte, [K, N];
  the kernel's weight is w = s * (q - 8) (symmetric, zero point 8);
* scales: one fp16 scale per group of g consecutive rows of K in each
  column, s = fp16(u / (8 * sqrt(K))), u ~ U[0.5, 1.5]; g = K means one
  scale per output channel.  With these scales Var(C) is O(1).
* non-centred and outlier activations for the parity tests: A ~ U[0, 8]
  (every product of a column has one sign, so the sums are large next to
  their signed parts), and A ~ N(0, 1) with 1% of the K columns (the same in
  every row) multiplied by 64;
* unquantised fp16 weights (input of the quantiser), [K, N]: per column a
  spread sigma = u / sqrt(K), u ~ U[0.5, 1.5], times N(0, 1) draws, and one
  entry in 1000 multiplied by 8 (the outlier weights of trained LLM layers,
  which are what a clipping search trades against); drawn in fp32, rounded
  to fp16.

Seeds: numpy's PCG64 (``default_rng``) keyed by a tuple, so every draw is
reproducible from (workload id, shape).  Weights and activations use
separate keys so that one packed weight serves every M of a sweep.
"""
from __future__ import annotations

import math

import numpy as np

__all__ = [
    "WORKLOADS",
    "weights",
    "activations",
    "activations_uniform",
    "activations_outlier_columns",
    "sparse24_weights",
    "fp16_weights",
    "num_groups",
]

# Named workloads: id -> (description, list of (K, N), list of group sizes, M sweep).
# g = None stands for "one scale per output channel" (g = K).
WORKLOADS = {
    0: ("tiny W4A16 GEMM", [(1024, 1024)], [128], [16]),
    1: ("Llama-7B attention projection", [(4096, 4096)], [128], [1, 2, 4, 8, 16, 32, 64, 128]),
    2: ("Llama-7B MLP", [(4096, 11008), (11008, 4096)], [128, None], [1, 2, 4, 8, 16, 32, 64, 128]),
    3: ("70B-class layer", [(8192, 28672), (28672, 8192)], [128], [1, 2, 4, 8, 16, 32, 64, 128]),
    4: ("2:4 sparse W4A16", [(8192, 8192)], [128], [1, 2, 4, 8, 16, 32, 64, 128]),
}


def num_groups(K: int, g: int | None) -> int:
    """Number of scale rows: ceil(K / g), or 1 for per-channel scales."""
    if g is None or g == K or g == -1:
        return 1
    return -(-K // g)


def _group_key(K: int, g: int | None) -> int:
    return K if (g is None or g == -1) else int(g)


def weights(wid: int, K: int, N: int, g: int | None, *, scale_max: float | None = None):
    """Draw (q, s): q uint8 [K, N] codes in 0..15, s float16 [G, N].

    ``scale_max`` is unused by the default recipe; it exists so tests can
    draw scales from another range without a second generator.
    """
    rng = np.random.default_rng([int(wid), 1, int(K), int(N), _group_key(K, g)])
    q = rng.integers(0, 16, size=(K, N), dtype=np.uint8)
    G = num_groups(K, g)
    u = rng.uniform(0.5, 1.5, size=(G, N))
    denom = 8.0 * math.sqrt(K)
    s = (u / denom) if scale_max is None else (u * (scale_max / 1.5))
    return q, s.astype(np.float16)


def activations(wid: int, M: int, K: int):
    """Draw A float16 [M, K], A ~ N(0, 1) rounded to fp16."""
    rng = np.random.default_rng([int(wid), 0, int(M), int(K)])
    return rng.standard_normal((M, K)).astype(np.float16)


def activations_uniform(wid: int, M: int, K: int, lo: float = 0.0, hi: float = 8.0):
    """Draw A float16 [M, K], A ~ U[lo, hi) rounded to fp16 (non-centred
    activations: every product of a column has the same sign)."""
    rng = np.random.default_rng([int(wid), 4, int(M), int(K)])
    return rng.uniform(lo, hi, size=(M, K)).astype(np.float16)


def activations_outlier_columns(wid: int, M: int, K: int, frac: float = 0.01, factor: float = 64.0):
    """Draw A float16 [M, K]: N(0, 1), with a random `frac` of the K columns
    (the same columns in every row) multiplied by `factor` -- the outlier
    features of LLM activations."""
    rng = np.random.default_rng([int(wid), 5, int(M), int(K)])
    a = rng.standard_normal((M, K))
    cols = rng.random(K) < frac
    a[:, cols] *= factor
    return a.astype(np.float16)


def sparse24_weights(wid: int, K: int, N: int, g: int | None):
    """Draw a 2:4-structured weight along K.

    Returns (q_dense, keep, s): q_dense uint8 [K, N] with pruned positions set
    to the code 8 (weight 0), and keep bool [K, N] marking the two kept
    positions in every group of 4 consecutive k of each column.  The kept
    codes are U{0..15} (a kept code may itself be 8).  The two positions
    are uniform over the six 2-of-4 patterns.  s is fp16 [G, N] (G groups
    of g rows, one for g None), U[0.5, 1.5] / (8 sqrt(K)).
    """
    if K % 4:
        raise ValueError("K must be a multiple of 4 for 2:4 sparsity")
    rng = np.random.default_rng([int(wid), 2, int(K), int(N), _group_key(K, g)])
    q = rng.integers(0, 16, size=(K, N), dtype=np.uint8)
    patterns = np.array([[1, 1, 0, 0], [1, 0, 1, 0], [1, 0, 0, 1],
                         [0, 1, 1, 0], [0, 1, 0, 1], [0, 0, 1, 1]], dtype=bool)
    pick = rng.integers(0, 6, size=(K // 4, N))
    keep = patterns[pick].transpose(0, 2, 1).reshape(K, N)
    q = np.where(keep, q, np.uint8(8)).astype(np.uint8)
    G = num_groups(K, g)
    u = rng.uniform(0.5, 1.5, size=(G, N))
    s = (u / (8.0 * math.sqrt(K))).astype(np.float16)
    return q, keep, s


def fp16_weights(wid: int, K: int, N: int):
    """Draw W float16 [K, N]: unquantised weights (recipe in the module doc)."""
    rng = np.random.default_rng([int(wid), 3, int(K), int(N)])
    sigma = (rng.uniform(0.5, 1.5, size=(1, N)) / math.sqrt(K)).astype(np.float32)
    w = rng.standard_normal((K, N), dtype=np.float32)
    w *= sigma
    outlier = rng.random((K, N), dtype=np.float32) < 1e-3
    w[outlier] *= 8.0
    return w.astype(np.float16)
