// Weight quantiser for gfx950: fp16 W[K][N] -> 4-bit codes q[K][N] and fp16
// scales s[K/g][N] in the format the GEMM consumes, w = s * (q - 8).
//
// Uniform quantisation (Section 2.2, Eq. 1) in its symmetric form: a group of
// g consecutive weights of a column is mapped onto the range [-a, a] with 15
// steps of s = 2a / 15 and the fixed zero point 8, q = clamp(rint(v * (1/s))
// + 8, 0, 15).  The clipping threshold a = r * max|v| is searched per group over
// the caller's ratios r, keeping the one with the smallest reconstruction
// error sum (v - s(q - 8))^2 (Section 2.2; the group-wise clipping search of
// Section 3.5).  GPTQ's error feedback needs calibration data and is not
// part of this quantiser.
//
// Every decision (the rounding of each code, the choice of the ratio) is an
// fp32 computation in a fixed order: the stored fp16 scale is formed first,
// codes use its fp32 reciprocal, each thread sums its group sequentially,
// and no multiply-add is contracted, so the result is the same bits on any
// device and in any launch shape.
//
// One thread owns one (group, column): consecutive threads take consecutive
// columns, so every row of a group is one coalesced 2-byte-per-lane load.
// With g = 128 the group's values stay in registers for the whole search;
// other group sizes re-read the group (from L2) for each ratio.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "quant.h"

namespace marlin {
namespace {

struct QuantArgs {
    const uint16_t *W;
    uint8_t *q;
    uint16_t *s;
    int K, N, g;
    int n_ratios;
    float ratios[kMaxQuantRatios];
};

__device__ __forceinline__ float h2f(uint16_t bits) { return (float)__builtin_bit_cast(_Float16, bits); }

// Code offset t = q - 8 of v for the reciprocal inv of a non-zero scale.
__device__ __forceinline__ float code_of(float v, float inv)
{
    float t = __builtin_rintf(v * inv);
    return __builtin_fminf(__builtin_fmaxf(t, -8.0f), 7.0f);
}

template <int GC>  // GC = 128: the group in registers; 0: any group size
__global__ void __launch_bounds__(256) quantize_kernel(QuantArgs a)
{
#pragma clang fp contract(off)
    const int n = blockIdx.x * 256 + (int)threadIdx.x;
    if (n >= a.N) return;
    const int g = GC ? GC : a.g;
    // register-held groups are indexed by constants only (full unrolling)
    constexpr int kUnroll = GC ? GC : 8;
    const int64_t row0 = (int64_t)blockIdx.y * g;
    const uint16_t *col = a.W + row0 * a.N + n;
    float vr[GC ? GC : 1];
    auto val = [&](int k) -> float {
        if constexpr (GC != 0) return vr[k];
        else return h2f(col[(int64_t)k * a.N]);
    };

    float amax = 0.0f;
    if constexpr (GC != 0) {
#pragma unroll
        for (int k = 0; k < GC; ++k) vr[k] = h2f(col[(int64_t)k * a.N]);
    }
#pragma unroll kUnroll
    for (int k = 0; k < g; ++k) amax = __builtin_fmaxf(amax, __builtin_fabsf(val(k)));

    float best_err = __builtin_inff();
    _Float16 best = (_Float16)0.0f;
    for (int i = 0; i < a.n_ratios; ++i) {
        const float lim = a.ratios[i] * amax;
        const _Float16 s16 = (_Float16)((lim + lim) / 15.0f);
        const float sf = (float)s16;
        float err = 0.0f;
        if (sf == 0.0f) {  // every code 8: the error is the group's energy
#pragma unroll kUnroll
            for (int k = 0; k < g; ++k) {
                const float v = val(k);
                err = err + v * v;
            }
        } else {
            const float inv = 1.0f / sf;
#pragma unroll kUnroll
            for (int k = 0; k < g; ++k) {
                const float v = val(k);
                const float d = v - code_of(v, inv) * sf;
                err = err + d * d;
            }
        }
        if (err < best_err) {
            best_err = err;
            best = s16;
        }
    }

    const float sf = (float)best;
    const float inv = sf == 0.0f ? 0.0f : 1.0f / sf;
    uint8_t *qc = a.q + row0 * a.N + n;
#pragma unroll kUnroll
    for (int k = 0; k < g; ++k) {
        const float t = sf == 0.0f ? 0.0f : code_of(val(k), inv);
        qc[(int64_t)k * a.N] = (uint8_t)(int)(t + 8.0f);
    }
    a.s[(int64_t)blockIdx.y * a.N + n] = __builtin_bit_cast(uint16_t, best);
}

}  // namespace

hipError_t launch_quantize(const uint16_t *W, int K, int N, int g, const float *ratios, int n_ratios,
                           uint8_t *q, uint16_t *s, hipStream_t stream)
{
    QuantArgs a;
    a.W = W;
    a.q = q;
    a.s = s;
    a.K = K;
    a.N = N;
    a.g = g;
    a.n_ratios = n_ratios;
    for (int i = 0; i < kMaxQuantRatios; ++i) a.ratios[i] = i < n_ratios ? ratios[i] : 0.0f;
    const dim3 grid((unsigned)((N + 255) / 256), (unsigned)(K / g));
    if (g == 128)
        hipLaunchKernelGGL(quantize_kernel<128>, grid, dim3(256), 0, stream, a);
    else
        hipLaunchKernelGGL(quantize_kernel<0>, grid, dim3(256), 0, stream, a);
    return hipGetLastError();
}

}  // namespace marlin
