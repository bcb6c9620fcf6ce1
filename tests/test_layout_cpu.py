"""Host-side checks of the packed layouts and of the paper's dequantisation
recipe (no GPU).

The layout reference in oracle/layout.py is checked against the header's
description by construction tests (each packed word is rebuilt from the
definition for single positions); the dequantisation recipe of Section 3.4
("Dequantization and Tensor Cores") is checked on every code in every nibble
slot with numpy's own fp16 arithmetic.
"""
import json
import os

import numpy as np
import pytest

from oracle import layout

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_constants.json")))


def test_roundtrip_random():
    rng = np.random.default_rng(3)
    for K, N in [(128, 64), (256, 128), (384, 192)]:
        q = rng.integers(0, 16, size=(K, N), dtype=np.uint8)
        w = layout.pack_weights(q)
        assert w.dtype == np.uint32 and w.size == K * N // 8
        assert np.array_equal(layout.unpack_weights(w, K, N), q)
        for g in (128, -1):
            G = 1 if g == -1 else K // g
            s = rng.standard_normal((G, N)).astype(np.float16)
            sp = layout.pack_scales(s, K, g)
            assert np.array_equal(layout.unpack_scales(sp, K, N, g).view(np.uint16), s.view(np.uint16))


def test_single_positions_follow_header():
    # a lone code 0xF at (k, n) must land in word (((c*KU+ku)*4+nb)*64+l)*4+t,
    # nibble (j>>1)+4(j&1), with c=n//64, nb=(n%64)//16, l%16=n%16,
    # ku=k//128, t=(k%128)//32, l//16=(k%32)//8, j=k%8
    K, N = 256, 128
    for (k, n) in [(0, 0), (7, 0), (8, 1), (31, 15), (32, 16), (127, 63), (128, 64), (255, 127), (77, 90)]:
        q = np.zeros((K, N), dtype=np.uint8)
        q[k, n] = 0xF
        w = layout.pack_weights(q)
        c, nb, lo = n // 64, (n % 64) // 16, n % 16
        ku, t, hi, j = k // 128, (k % 128) // 32, (k % 32) // 8, k % 8
        l = hi * 16 + lo
        idx = (((c * (K // 128) + ku) * 4 + nb) * 64 + l) * 4 + t
        nib = (j >> 1) + 4 * (j & 1)
        assert np.flatnonzero(w).tolist() == [idx]
        assert w[idx] == 0xF << (4 * nib)


def test_scale_positions_follow_header():
    K, N, g = 256, 128, 128
    G = 2
    s = np.arange(G * N, dtype=np.float16).reshape(G, N)
    sp = layout.pack_scales(s, K, g)
    for (r, n) in [(0, 0), (1, 127), (0, 21), (1, 64)]:
        c, rem = n // 64, n % 64
        nb, lg, i = rem // 16, (rem % 16) // 4, rem % 4
        assert sp[(((c * G + r) * 4 + lg) * 4 + nb) * 4 + i] == s[r, n]


def _fp16(bits):
    return np.array(bits, dtype=np.uint16).view(np.float16)


def test_paper_or_bits_give_1024():
    # the OR pattern 0110010 in the top 7 bits of an fp16 is the number 1024,
    # whose mantissa LSB has weight 1 (Section 3.4)
    top7 = int(GOLD["dequant_or_bits"]["value"], 2)
    assert top7 == 50
    base = top7 << 9
    assert base == 0x6400 and float(_fp16(base)) == 1024.0
    assert float(_fp16(base | 1)) - 1024.0 == 1.0


@pytest.mark.parametrize("slot", range(8))
def test_dequant_recipe_every_code_every_slot(slot):
    # low nibble of each 16-bit half: (x & 0x000F000F) | 0x64006400 = 1024 + q,
    # minus 1032 (the zero point 8 folded into the subtrahend) = q - 8;
    # high nibble: (x & 0x00F000F0) | 0x64006400 = 1024 + 16q, then
    # fma(., 1/16, -72) = q - 8.  Shifting by 8 reaches the other two nibbles.
    zp = GOLD["zero_point"]["value"]
    for code in range(16):
        x = np.uint32(code << (4 * slot))
        half = slot // 4          # which 16-bit half holds the code
        sub = slot % 4            # nibble within that half
        y = x >> np.uint32(8) if sub >= 2 else x
        if sub % 2 == 0:
            bits = (y & np.uint32(0x000F000F)) | np.uint32(0x64006400)
            h = np.array([bits], dtype=np.uint32).view(np.float16)
            val = (h - np.float16(1024 + zp))[half]
        else:
            bits = (y & np.uint32(0x00F000F0)) | np.uint32(0x64006400)
            h = np.array([bits], dtype=np.uint32).view(np.float16)
            val = (h[half].astype(np.float32) * np.float32(1 / 16) - np.float32(64 + zp))
            val = np.float16(val)  # one rounding, as a fused multiply-add
        assert float(val) == code - zp, (slot, code, float(val))


@pytest.mark.parametrize("slot", range(8))
def test_subnormal_operands_every_code_every_slot(slot):
    # The kernel's form of the same trick with the magic number 0: the masked
    # code alone, read as fp16, is the subnormal q * 2^-24 (lower nibble of a
    # byte) or 16 q * 2^-24 (upper nibble); the activation paired with an
    # upper nibble carries 1/16, and the zero point is the same encoding of
    # the code 8 (8 * 2^-24 or 128 * 2^-24), subtracted.  In exact arithmetic
    # w * a' - z * a' = (q - 8) * a * 2^-24 for every code in every slot.
    from fractions import Fraction
    zp = GOLD["zero_point"]["value"]
    e = Fraction(1, 1 << 24)
    half, sub = slot // 4, slot % 4
    upper = sub % 2 == 1
    zbits = 0x0080 if upper else 0x0008
    assert Fraction(float(_fp16(zbits))) == (128 if upper else 8) * e
    for code in range(16):
        x = np.uint32(code << (4 * slot))
        y = x >> np.uint32(8) if sub >= 2 else x
        mask = np.uint32(0x00F000F0) if upper else np.uint32(0x000F000F)
        h = np.array([y & mask], dtype=np.uint32).view(np.float16)[half]
        w = Fraction(float(h))
        assert w == (16 if upper else 1) * code * e, (slot, code)
        for a in (Fraction(1), Fraction(-3, 4), Fraction(1027, 1024)):
            a_scaled = a / 16 if upper else a
            assert w * a_scaled - Fraction(float(_fp16(zbits))) * a_scaled == (code - zp) * a * e


# ---- 2:4 sparse layout ----

def test_sparse_roundtrip_and_selection():
    import synth
    for K, N in [(128, 64), (256, 128)]:
        q, keep, s = synth.sparse24_weights(4, K, N, 128)
        w = layout.pack_sparse(q)
        assert w.dtype == np.uint32 and w.size == K * N * 3 // 32
        assert np.array_equal(layout.unpack_sparse(w, K, N), q)
    # at most two non-8 codes per group: exact; the kept rows are increasing
    rng = np.random.default_rng(5)
    K, N = 128, 64
    q = np.full((K, N), 8, np.uint8)
    for r in range(K // 4):
        for n in range(N):
            rows = rng.choice(4, size=rng.integers(0, 3), replace=False)
            q[4 * r + rows, n] = rng.choice([c for c in range(16) if c != 8], size=len(rows))
    pos, codes = layout.sparse_selection(q)
    assert (pos[:, 0, :] < pos[:, 1, :]).all()
    assert np.array_equal(layout.unpack_sparse(layout.pack_sparse(q), K, N), q)
    # a third non-8 code in a group is dropped, the first two are kept
    q3 = np.full((K, N), 8, np.uint8)
    q3[0:3, 0] = [1, 2, 3]
    out = layout.unpack_sparse(layout.pack_sparse(q3), K, N)
    assert list(out[0:4, 0]) == [1, 2, 8, 8]


def test_sparse_single_positions_follow_header():
    # a lone non-8 code at (k, n): codes word ((d>>2)*64 + l)*4 + (d&3) of
    # unit (c, ku), d = 2nb + h, nibble (j>>1) + 4(j&1) with j = 2g + t; the
    # index word 512 + 4l + nb holds its row at bits 16h + 4g + 2t.
    K, N = 256, 128
    KU = K // 128
    for (k, n, code) in [(0, 0, 3), (5, 17, 15), (66, 64, 0), (130, 127, 9), (255, 90, 1)]:
        q = np.full((K, N), 8, np.uint8)
        q[k, n] = code
        w = layout.pack_sparse(q).reshape(N // 64, KU, 768)
        c, nb, ku = n // 64, (n % 64) // 16, k // 128
        h, lg, g, r = (k % 128) // 64, (k % 64) // 16, (k % 16) // 4, k % 4
        l = 16 * lg + n % 16
        # the group is completed with its lowest code-8 row: (r, 1) if r == 0, else (0, r)
        t = 0 if r == 0 else 1
        j = 2 * g + t
        d = 2 * nb + h
        word = w[c, ku, ((d >> 2) * 64 + l) * 4 + (d & 3)]
        assert (word >> (4 * int(layout.NIBBLE_OF[j]))) & 0xF == code
        meta = w[c, ku, 512 + 4 * l + nb]
        assert (meta >> (16 * h + 4 * g + 2 * t)) & 3 == r
        other = 1 if r == 0 else 0
        assert (meta >> (16 * h + 4 * g + 2 * (1 - t))) & 3 == other
