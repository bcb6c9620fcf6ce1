"""Reference for the packed weight and scale layouts (test infrastructure only).

Written from the layout definitions in the library's public header, with
plain numpy index arithmetic: it lets the tests check the GPU pack and
unpack kernels word for word.  The GEMM parity tests do not depend on it
(they compare the GEMM on packed data against the oracle on unpacked codes).

Why the layout has this shape (Section 3.4): "Maximizing Loading Bandwidth"
asks for the widest (16-byte) load per thread over tiles laid out
contiguously; "Dequantization and Tensor Cores" asks that each thread's
vector hold exactly its operands for several matrix-core steps, with codes
interleaved inside each 32-bit word for paired decoding; "Groups and
Instruction Ordering" packs each thread's scales for several blocks into one
vector.  The concrete orders below are this library's, for the gfx950
16x16x32 fp16 MFMA; the paper's own order was for Ampere mma.sync.
"""
from __future__ import annotations

import numpy as np

# nibble position of element j of a lane's 8 consecutive k
NIBBLE_OF = np.array([(j >> 1) + 4 * (j & 1) for j in range(8)], dtype=np.uint32)


def _num_groups(K, group):
    return 1 if group in (-1, None) or group >= K else K // group


def pack_weights(q: np.ndarray) -> np.ndarray:
    """uint8 codes [K, N] -> uint32 words in the packed order (flat)."""
    K, N = q.shape
    assert K % 128 == 0 and N % 64 == 0
    C, KU = N // 64, K // 128
    c, ku, nb, l, t, j = np.meshgrid(np.arange(C), np.arange(KU), np.arange(4),
                                     np.arange(64), np.arange(4), np.arange(8),
                                     indexing="ij")
    n = 64 * c + 16 * nb + (l % 16)
    k = 128 * ku + 32 * t + 8 * (l // 16) + j
    codes = (q[k, n] & 0xF).astype(np.uint32)
    words = (codes << (4 * NIBBLE_OF[j])).sum(axis=-1, dtype=np.uint64).astype(np.uint32)
    return words.reshape(-1)


def unpack_weights(words: np.ndarray, K: int, N: int) -> np.ndarray:
    """Inverse of pack_weights."""
    C, KU = N // 64, K // 128
    w = np.asarray(words, dtype=np.uint32).reshape(C, KU, 4, 64, 4)
    q = np.empty((K, N), dtype=np.uint8)
    c, ku, nb, l, t, j = np.meshgrid(np.arange(C), np.arange(KU), np.arange(4),
                                     np.arange(64), np.arange(4), np.arange(8),
                                     indexing="ij")
    n = 64 * c + 16 * nb + (l % 16)
    k = 128 * ku + 32 * t + 8 * (l // 16) + j
    q[k, n] = ((w[c, ku, nb, l, t] >> (4 * NIBBLE_OF[j])) & 0xF).astype(np.uint8)
    return q


def pack_scales(s: np.ndarray, K: int, group) -> np.ndarray:
    """fp16 [G, N] -> fp16 flat in the packed order."""
    G, N = s.shape
    assert G == _num_groups(K, group)
    C = N // 64
    c, r, lg, nb, i = np.meshgrid(np.arange(C), np.arange(G), np.arange(4),
                                  np.arange(4), np.arange(4), indexing="ij")
    return s[r, 64 * c + 16 * nb + 4 * lg + i].reshape(-1)


def unpack_scales(sp: np.ndarray, K: int, N: int, group) -> np.ndarray:
    G = _num_groups(K, group)
    C = N // 64
    out = np.empty((G, N), dtype=sp.dtype)
    c, r, lg, nb, i = np.meshgrid(np.arange(C), np.arange(G), np.arange(4),
                                  np.arange(4), np.arange(4), indexing="ij")
    out[r, 64 * c + 16 * nb + 4 * lg + i] = np.asarray(sp).reshape(C, G, 4, 4, 4)
    return out
