"""Byte and FLOP accounting of the W4A16 GEMM, and MI355X peaks.

Algorithmic work per call (what the method must move or compute; workspace
traffic is implementation overhead and not counted):

* FLOPs: 2*M*N*K (Section 3.4, "Bound By Weight Loading": exactly M*K*N
  multiply-accumulates of 2 FLOPs each);
* bytes: the paper's 16MK + 4KN + 16MN bits (fp16 A and C, 4-bit B) plus the
  group scales, 2 bytes per scale, ceil(K/g)*N of them (the 0.125 bit per
  weight that Section 5.1 includes in its ideal 3.87x at g = 128);
* weight-stream bytes: K*N/2 + 2*ceil(K/g)*N.

The fp16 comparator (a plain fp16 GEMM of the same shape) moves
2KN + 2MK + 2MN bytes.  The roofline time of either is
max(bytes / HBM bandwidth, FLOPs / MFMA peak).
"""
from __future__ import annotations

# MI355X published peaks (dense): HBM3E bandwidth and fp16 MFMA throughput.
HBM_BYTES_PER_S = 8.0e12
FP16_MFMA_FLOPS = 2.5e15
CU_COUNT = 256
CLOCK_HZ = 2.4e9


def num_groups(K: int, g) -> int:
    if g is None or g == -1 or g >= K:
        return 1
    return -(-K // g)


def flops(M: int, N: int, K: int) -> float:
    return 2.0 * M * N * K


def paper_memory_bits(M: int, N: int, K: int) -> int:
    """The paper's count of bits touched, without scales: 16MK + 4KN + 16MN."""
    return 16 * M * K + 4 * K * N + 16 * M * N


def weight_bytes(N: int, K: int, g, bits: int = 4) -> float:
    return K * N * bits / 8.0 + 2.0 * num_groups(K, g) * N


def w4a16_bytes(M: int, N: int, K: int, g) -> float:
    return paper_memory_bits(M, N, K) / 8.0 + 2.0 * num_groups(K, g) * N


def sparse24_bytes(M: int, N: int, K: int, g) -> float:
    """2:4 sparse weights (Section 4): half the codes (K*N/4 bytes), 2-bit row
    indices per kept code (K*N/8 bytes), the same scales, A and C."""
    return K * N / 4.0 + K * N / 8.0 + 2.0 * num_groups(K, g) * N + 2.0 * M * K + 2.0 * M * N


def sparse24_flops(M: int, N: int, K: int) -> float:
    """Kept multiply-accumulates only: M*N*K/2 of 2 FLOPs each."""
    return 1.0 * M * N * K


def sparse24_t_roof(M, N, K, g, bw=HBM_BYTES_PER_S, peak=FP16_MFMA_FLOPS) -> float:
    return t_roof(sparse24_bytes(M, N, K, g), sparse24_flops(M, N, K), bw, peak)


def fp16_bytes(M: int, N: int, K: int) -> float:
    return 2.0 * K * N + 2.0 * M * K + 2.0 * M * N


def t_roof(nbytes: float, nflops: float, bw: float = HBM_BYTES_PER_S,
           peak: float = FP16_MFMA_FLOPS) -> float:
    return max(nbytes / bw, nflops / peak)


def w4a16_t_roof(M, N, K, g, bw=HBM_BYTES_PER_S, peak=FP16_MFMA_FLOPS) -> float:
    return t_roof(w4a16_bytes(M, N, K, g), flops(M, N, K), bw, peak)


def fp16_t_roof(M, N, K, bw=HBM_BYTES_PER_S, peak=FP16_MFMA_FLOPS) -> float:
    return t_roof(fp16_bytes(M, N, K), flops(M, N, K), bw, peak)


def bound(M, N, K, g, bw=HBM_BYTES_PER_S, peak=FP16_MFMA_FLOPS) -> str:
    return "hbm" if w4a16_bytes(M, N, K, g) / bw >= flops(M, N, K) / peak else "mfma"


def ideal_weight_speedup(bits: int = 4, g: int = 128, scale_bits: int = 16) -> float:
    """fp16 weight bits over quantised weight bits including scale storage."""
    return 16.0 / (bits + scale_bits / g)


def b_opt(flop_per_byte: float, bits: int = 4) -> float:
    """Batch size at which a weight-load-bound matmul turns compute-bound:
    2 FLOPs per weight per input row against bits/8 bytes per weight."""
    return flop_per_byte * (bits / 8.0) / 2.0


def ridge_m(g: int = 128, bw=HBM_BYTES_PER_S, peak=FP16_MFMA_FLOPS, bits: int = 4) -> float:
    """M at which weight bytes / bw equals 2MNK / peak (A and C ignored)."""
    per_weight = bits / 8.0 + 2.0 / g
    return (peak / bw) * per_weight / 2.0


# ---- quantiser (symmetric uniform quantisation with a clipping search) ----
# Vector issue rate: 256 CUs x 4 SIMDs x 32 fp32 lanes per clock x 2.4 GHz
# = 78.6 T lane operations/s.  The published fp32 vector peak, 157.3 TFLOP/s,
# is this rate with a fused multiply-add counted as two FLOPs.  The library
# is built without packed fp32 instructions; that an unpacked wave64
# instruction issues in two clocks, not four, is measured: on 28672 x 8192
# the quantiser issues 307 M wave instructions (SQ_INSTS_VALU) over 1024
# SIMDs in 0.94 M kernel clocks (GRBM_GUI_ACTIVE per XCD), 3.1 clocks per
# instruction and SIMD, which four-clock issue could not reach
# (profiles/quantize_g128_clip10_counters.md).
VALU_LANE_OPS = 256 * 4 * 32 * 2.4e9
FP32_VECTOR_FLOPS = 157.3e12
FP32_LANE_OPS = VALU_LANE_OPS

# Vector instructions per weight (lane operations) of the built g = 128
# quantiser kernel: 12.35 outside the search (loading, magnitude maximum,
# the final scale's reciprocal and codes) and 7.21 per clipping ratio
# (scale multiply, round, clamp, multiply back, subtract, square,
# accumulate), counted in its gfx950 assembly: 1580 + 923 per ratio, for the
# 128 weights a thread owns.  The counters give 83.7 per weight at 10 ratios
# (branches skip a few), against 84.5 by this count.
QUANT_VALU_BASE = 1580 / 128
QUANT_VALU_PER_RATIO = 923 / 128
QUANT_VALU_PER_WEIGHT_G128_10 = QUANT_VALU_BASE + 10 * QUANT_VALU_PER_RATIO


def quant_ops(K: int, N: int, n_ratios: int) -> float:
    """fp32 vector operations the quantiser must perform, K*N weights:
    per weight one max of magnitudes, then per ratio the code (scale
    multiply, round, clamp) and its error term (multiply back, subtract,
    square, accumulate): 7, and the final code (multiply, round, clamp,
    offset): 4."""
    return float(K) * N * (1 + 7 * n_ratios + 4)


def quant_lane_ops(K: int, N: int, n_ratios: int) -> float:
    """Vector lane operations the built g = 128 quantiser issues for K*N
    weights (its instruction count, which includes conversions, address
    arithmetic and the reciprocal)."""
    return float(K) * N * (QUANT_VALU_BASE + QUANT_VALU_PER_RATIO * n_ratios)


def quant_bytes(K: int, N: int, g) -> float:
    """HBM bytes: fp16 weights read, one code byte and the fp16 scales written."""
    return 2.0 * K * N + 1.0 * K * N + 2.0 * num_groups(K, g) * N
