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


# ---- 2:4 sparse weights (Section 4) ----

def sparse_selection(q: np.ndarray):
    """Kept rows of every group of 4 consecutive k in each column.

    Returns (pos, codes), each [K/4, 2, N]: the two kept rows (0..3,
    increasing) and their codes.  Kept rows are the first two rows whose
    code is not 8 (non-zero weight); a group with fewer is completed with
    its lowest rows of code 8 (the documented packing rule)."""
    K, N = q.shape
    qg = (q & 0xF).reshape(K // 4, 4, N)
    r = np.arange(4).reshape(1, 4, 1)
    key = np.where(qg != 8, r, 4 + r)
    first2 = np.argsort(key, axis=1, kind="stable")[:, :2, :]
    pos = np.sort(first2, axis=1)
    codes = np.take_along_axis(qg, pos, axis=1)
    return pos.astype(np.uint32), codes.astype(np.uint32)


def pack_sparse(q: np.ndarray) -> np.ndarray:
    """uint8 codes [K, N] (2:4 along K: pruned positions hold code 8) -> uint32
    words of the packed sparse layout (flat), 768 words per 64 x 128 unit."""
    K, N = q.shape
    assert K % 128 == 0 and N % 64 == 0
    C, KU = N // 64, K // 128
    pos, codes = sparse_selection(q)
    out = np.zeros((C, KU, 768), dtype=np.uint32)
    c, ku, nb, l, h = np.meshgrid(np.arange(C), np.arange(KU), np.arange(4), np.arange(64),
                                  np.arange(2), indexing="ij")
    n = 64 * c + 16 * nb + (l % 16)
    grp0 = (128 * ku + 64 * h + 16 * (l // 16)) // 4
    word = np.zeros(n.shape, dtype=np.uint32)
    meta = np.zeros(n.shape, dtype=np.uint32)
    for g in range(4):
        for t in range(2):
            j = 2 * g + t
            word |= codes[grp0 + g, t, n] << np.uint32(4 * NIBBLE_OF[j])
            meta |= pos[grp0 + g, t, n] << np.uint32(4 * g + 2 * t)
    d = 2 * nb + h
    out[c, ku, ((d >> 2) * 64 + l) * 4 + (d & 3)] = word
    m2 = np.zeros((C, KU, 4, 64), dtype=np.uint32)
    for hh in range(2):
        m2 |= meta[..., hh] << np.uint32(16 * hh)
    c2, ku2, nb2, l2 = np.meshgrid(np.arange(C), np.arange(KU), np.arange(4), np.arange(64), indexing="ij")
    out[c2, ku2, 512 + l2 * 4 + nb2] = m2
    return out.reshape(-1)


def unpack_sparse(words: np.ndarray, K: int, N: int) -> np.ndarray:
    """Inverse of pack_sparse: dense codes [K, N], code 8 at pruned rows."""
    C, KU = N // 64, K // 128
    w = np.asarray(words, dtype=np.uint32).reshape(C, KU, 768)
    q = np.full((K, N), 8, dtype=np.uint8)
    c, ku, nb, l, h = np.meshgrid(np.arange(C), np.arange(KU), np.arange(4), np.arange(64),
                                  np.arange(2), indexing="ij")
    n = 64 * c + 16 * nb + (l % 16)
    d = 2 * nb + h
    word = w[c, ku, ((d >> 2) * 64 + l) * 4 + (d & 3)]
    meta = w[c, ku, 512 + l * 4 + nb] >> np.uint32(16 * h)
    for g in range(4):
        for t in range(2):
            j = 2 * g + t
            r = (meta >> np.uint32(4 * g + 2 * t)) & 3
            k = 128 * ku + 64 * h + 16 * (l // 16) + 4 * g + r
            q[k, n] = ((word >> np.uint32(4 * NIBBLE_OF[j])) & 0xF).astype(np.uint8)
    return q
