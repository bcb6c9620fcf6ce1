// Offline repack of int4 codes and fp16 scales into the order the GEMM
// streams them (Section 3.4: "Maximizing Loading Bandwidth",
// "Dequantization and Tensor Cores", "Groups and Instruction Ordering").
//
// Weight words (uint32), c = 64-column tile, ku = 128-row block, nb = 16-column
// block, l = lane 0..63, t = 0..3:
//   word (((c*KU + ku)*4 + nb)*64 + l)*4 + t holds column n = 64c + 16nb + l%16,
//   rows k = 128ku + 32t + 8(l/16) + j (j = 0..7), code j in nibble
//   (j >> 1) + 4(j & 1).
// The nibble order puts codes j and j+1 sixteen bits apart, so one mask (and
// an or with the magic number) yields two fp16 values at once (dequant_sub in
// gemm.hip, dequant_magic in device.h).
//
// Scales (fp16), r = scale row, lg = n-row group of the MFMA output, i = 0..3:
//   index (((c*G + r)*4 + lg)*4 + nb)*4 + i holds s[r][64c + 16nb + 4lg + i],
// so the 16 scales one output lane needs for a 64-column tile are contiguous.
#include <hip/hip_runtime.h>

#include "internal.h"

namespace marlin {
namespace {

__device__ __forceinline__ int nibble_of(int j) { return (j >> 1) + 4 * (j & 1); }

__global__ void pack_weights_kernel(const uint8_t *__restrict__ q, int K, int N,
                                    uint32_t *__restrict__ w)
{
    const int64_t words = (int64_t)K * N / 8;
    const int KU = K / 128;
    for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < words;
         idx += (int64_t)gridDim.x * blockDim.x) {
        const int t = (int)(idx & 3);
        const int l = (int)((idx >> 2) & 63);
        const int nb = (int)((idx >> 8) & 3);
        const int64_t tile = idx >> 10;  // c*KU + ku
        const int ku = (int)(tile % KU);
        const int c = (int)(tile / KU);
        const int n = 64 * c + 16 * nb + (l & 15);
        const int k0 = 128 * ku + 32 * t + 8 * (l >> 4);
        uint32_t word = 0;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const uint32_t code = q[(int64_t)(k0 + j) * N + n] & 0xFu;
            word |= code << (4 * nibble_of(j));
        }
        w[idx] = word;
    }
}

__global__ void unpack_weights_kernel(const uint32_t *__restrict__ w, int K, int N,
                                      uint8_t *__restrict__ q)
{
    const int64_t words = (int64_t)K * N / 8;
    const int KU = K / 128;
    for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < words;
         idx += (int64_t)gridDim.x * blockDim.x) {
        const int t = (int)(idx & 3);
        const int l = (int)((idx >> 2) & 63);
        const int nb = (int)((idx >> 8) & 3);
        const int64_t tile = idx >> 10;
        const int ku = (int)(tile % KU);
        const int c = (int)(tile / KU);
        const int n = 64 * c + 16 * nb + (l & 15);
        const int k0 = 128 * ku + 32 * t + 8 * (l >> 4);
        const uint32_t word = w[idx];
#pragma unroll
        for (int j = 0; j < 8; ++j)
            q[(int64_t)(k0 + j) * N + n] = (uint8_t)((word >> (4 * nibble_of(j))) & 0xFu);
    }
}

// dir = 0: natural [G][N] -> packed; dir = 1: packed -> natural.
__global__ void permute_scales_kernel(const uint16_t *__restrict__ src, int N, int G, int dir,
                                      uint16_t *__restrict__ dst)
{
    const int64_t total = (int64_t)G * N;
    for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
         idx += (int64_t)gridDim.x * blockDim.x) {
        const int i = (int)(idx & 3);
        const int nb = (int)((idx >> 2) & 3);
        const int lg = (int)((idx >> 4) & 3);
        const int64_t cr = idx >> 6;  // c*G + r
        const int r = (int)(cr % G);
        const int c = (int)(cr / G);
        const int64_t nat = (int64_t)r * N + 64 * c + 16 * nb + 4 * lg + i;
        if (dir == 0)
            dst[idx] = src[nat];
        else
            dst[nat] = src[idx];
    }
}

// ---- 2:4 sparse weights (Section 4) ----
// Unit (c, ku) = 64-column tile c, 128-row block ku, at word (c*KU + ku)*768:
//   codes, 512 words: word ((d >> 2)*64 + l)*4 + (d & 3), d = 2*nb + h, holds
//     the 8 kept codes of column n = 64c + 16nb + l%16 in rows
//     128ku + 64h + 16(l/16) + [0, 16): group g = 0..3 of 4 rows keeps codes
//     j = 2g and 2g + 1 (in increasing row order), code j in nibble
//     (j >> 1) + 4(j & 1);
//   metadata, 256 words: word 512 + l*4 + nb holds, at bits 16h + 4g + 2t,
//     the row (0..3) within group g of kept code 2g + t.
// Kept rows are the first two rows of the group whose code is not 8 (weight
// not zero); a group with fewer is completed with its lowest rows of code 8,
// and the pair is kept in increasing row order.
__global__ void pack_sparse_kernel(const uint8_t *__restrict__ q, int K, int N, uint32_t *__restrict__ w)
{
    const int64_t items = (int64_t)K * N / 32;  // (unit, lane, column block)
    const int KU = K / 128;
    for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < items;
         idx += (int64_t)gridDim.x * blockDim.x) {
        const int nb = (int)(idx & 3);
        const int l = (int)((idx >> 2) & 63);
        const int64_t unit = idx >> 8;  // c*KU + ku
        const int ku = (int)(unit % KU);
        const int c = (int)(unit / KU);
        const int n = 64 * c + 16 * nb + (l & 15);
        uint32_t meta = 0;
        uint32_t *uw = w + unit * 768;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            uint32_t word = 0;
            const int kbase = 128 * ku + 64 * h + 16 * (l >> 4);
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                uint32_t code[4];
#pragma unroll
                for (int r = 0; r < 4; ++r) code[r] = q[(int64_t)(kbase + 4 * g + r) * N + n] & 0xFu;
                int p[2] = {-1, -1}, np = 0;
                for (int r = 0; r < 4 && np < 2; ++r)
                    if (code[r] != 8u) p[np++] = r;
                for (int r = 0; r < 4 && np < 2; ++r)
                    if (r != p[0]) p[np++] = r;
                if (p[0] > p[1]) {
                    const int t = p[0];
                    p[0] = p[1];
                    p[1] = t;
                }
#pragma unroll
                for (int t = 0; t < 2; ++t) {
                    const int j = 2 * g + t;
                    word |= code[p[t]] << (4 * nibble_of(j));
                    meta |= (uint32_t)p[t] << (16 * h + 4 * g + 2 * t);
                }
            }
            const int d = 2 * nb + h;
            uw[((d >> 2) * 64 + l) * 4 + (d & 3)] = word;
        }
        uw[512 + l * 4 + nb] = meta;
    }
}

__global__ void unpack_sparse_kernel(const uint32_t *__restrict__ w, int K, int N, uint8_t *__restrict__ q)
{
    const int64_t items = (int64_t)K * N / 32;
    const int KU = K / 128;
    for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < items;
         idx += (int64_t)gridDim.x * blockDim.x) {
        const int nb = (int)(idx & 3);
        const int l = (int)((idx >> 2) & 63);
        const int64_t unit = idx >> 8;
        const int ku = (int)(unit % KU);
        const int c = (int)(unit / KU);
        const int n = 64 * c + 16 * nb + (l & 15);
        const uint32_t *uw = w + unit * 768;
        const uint32_t meta = uw[512 + l * 4 + nb];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int d = 2 * nb + h;
            const uint32_t word = uw[((d >> 2) * 64 + l) * 4 + (d & 3)];
            const int kbase = 128 * ku + 64 * h + 16 * (l >> 4);
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                uint8_t out[4] = {8, 8, 8, 8};
#pragma unroll
                for (int t = 0; t < 2; ++t) {
                    const int j = 2 * g + t;
                    const int r = (int)((meta >> (16 * h + 4 * g + 2 * t)) & 3u);
                    out[r] = (uint8_t)((word >> (4 * nibble_of(j))) & 0xFu);
                }
#pragma unroll
                for (int r = 0; r < 4; ++r) q[(int64_t)(kbase + 4 * g + r) * N + n] = out[r];
            }
        }
    }
}

int blocks_for(int64_t work, int threads)
{
    int64_t b = (work + threads - 1) / threads;
    if (b > 65536) b = 65536;
    return (int)(b < 1 ? 1 : b);
}

}  // namespace

hipError_t launch_pack(const uint8_t *q, const uint16_t *s, int K, int N, int G,
                       uint32_t *w_packed, uint16_t *s_packed, hipStream_t stream)
{
    const int threads = 256;
    const int64_t words = (int64_t)K * N / 8;
    hipLaunchKernelGGL(pack_weights_kernel, dim3(blocks_for(words, threads)), dim3(threads), 0,
                       stream, q, K, N, w_packed);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(permute_scales_kernel, dim3(blocks_for((int64_t)G * N, threads)),
                       dim3(threads), 0, stream, s, N, G, 0, s_packed);
    return hipGetLastError();
}

hipError_t launch_unpack(const uint32_t *w_packed, const uint16_t *s_packed, int K, int N,
                         int G, uint8_t *q, uint16_t *s, hipStream_t stream)
{
    const int threads = 256;
    const int64_t words = (int64_t)K * N / 8;
    hipLaunchKernelGGL(unpack_weights_kernel, dim3(blocks_for(words, threads)), dim3(threads), 0,
                       stream, w_packed, K, N, q);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(permute_scales_kernel, dim3(blocks_for((int64_t)G * N, threads)),
                       dim3(threads), 0, stream, s_packed, N, G, 1, s);
    return hipGetLastError();
}

hipError_t launch_pack_sparse(const uint8_t *q, const uint16_t *s, int K, int N, int G, uint32_t *w_packed,
                              uint16_t *s_packed, hipStream_t stream)
{
    const int threads = 256;
    const int64_t items = (int64_t)K * N / 32;
    hipLaunchKernelGGL(pack_sparse_kernel, dim3(blocks_for(items, threads)), dim3(threads), 0, stream, q, K, N,
                       w_packed);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(permute_scales_kernel, dim3(blocks_for((int64_t)G * N, threads)), dim3(threads), 0, stream,
                       s, N, G, 0, s_packed);
    return hipGetLastError();
}

hipError_t launch_unpack_sparse(const uint32_t *w_packed, const uint16_t *s_packed, int K, int N, int G,
                                uint8_t *q, uint16_t *s, hipStream_t stream)
{
    const int threads = 256;
    const int64_t items = (int64_t)K * N / 32;
    hipLaunchKernelGGL(unpack_sparse_kernel, dim3(blocks_for(items, threads)), dim3(threads), 0, stream, w_packed,
                       K, N, q);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(permute_scales_kernel, dim3(blocks_for((int64_t)G * N, threads)), dim3(threads), 0, stream,
                       s_packed, N, G, 1, s);
    return hipGetLastError();
}

}  // namespace marlin
