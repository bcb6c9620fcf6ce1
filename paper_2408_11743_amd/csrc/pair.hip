// W4A16 GEMM for gfx950 with 64-row groups and two waves per SIMD:
// C[M,N] = A[M,K] * (s * (q - 8)), fp32 accumulation.
//
// The tiles, units, partition and combination are the stream kernel's with
// four 16-row blocks (64 rows x 128 columns per tile, gemm.hip); the work of
// a stage is split differently.  Eight waves form four pairs; pair k takes
// 128-row block k of the stage (the waves of a work-group split K in four),
// and the two waves of a pair take one packed 64-column tile each, 64 x 64
// outputs per wave.  A pair shares its block's 64 activation rows: each wave
// brings half of them into the pair's LDS ring slot by direct-to-LDS loads,
// and the pair meets at a barrier before reading them and again before the
// slot is refilled.  Waves w and w + 4 run on one SIMD, so one wave's code
// conversion overlaps the other's MFMAs (with one wave per SIMD the two run
// in turn).  Codes are converted with the magic number (exact q - 8) and the
// group scale multiplies the fp16 weights (Section 3.4, "Dequantization and
// Tensor Cores", "Groups and Instruction Ordering"); the four waves of a
// column half meet in LDS when a tile segment ends (Algorithm 1's
// reduction over the waves that share an output tile).
#include <hip/hip_runtime.h>
#include <stdio.h>

#include "device.h"
#include "internal.h"

namespace marlin {
namespace {

using namespace dev;

// Eight fp16 weights times one scale (in both halves of s2), one rounding each.
__device__ __forceinline__ half8_t scale_weights(half8_t w, half2_t s2)
{
    const u32x4_t u = __builtin_bit_cast(u32x4_t, w);
    return __builtin_bit_cast(half8_t, u32x4_t{as_u32(as_h2(u[0]) * s2), as_u32(as_h2(u[1]) * s2),
                                               as_u32(as_h2(u[2]) * s2), as_u32(as_h2(u[3]) * s2)});
}

template <bool PER_CHANNEL>
__global__ void __launch_bounds__(512, 1) w4a16_pair_kernel(GemmProblem p)
{
    constexpr int KS = 4;               // 128-row blocks of K per stage (one per pair)
    constexpr int D = 2;                // ring depth
    constexpr int MB = 4;               // 16-row blocks per wave (all 64 rows)
    constexpr int NBW = 4;              // 16-column blocks per wave (one packed tile)
    constexpr int kOwn = 4;             // blocks a wave holds after the reduction
    constexpr int kAStage = 64 * 256;   // one block's 64 rows x 128 k, bytes
    constexpr int kADma = 8;            // this wave's half of the block's 16 one-KiB loads
    constexpr int kWL = NBW;            // weight loads per stage
    constexpr int kSL = PER_CHANNEL ? 0 : 2;
    constexpr int kLoads = kADma + kWL + kSL;
    static_assert((D - 1) * kLoads + kWL + kSL < 64, "vmcnt range");
    __shared__ __attribute__((aligned(16))) uint8_t a_lds[KS * D * kAStage];  // 128 KiB
    __shared__ int flags[2];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int ks = wave & 3;    // the pair: 128-row block of the stage
    const int hf = wave >> 2;   // packed 64-column tile of the column tile (column half)
    const int lg = lane >> 4;
    const int KU = p.KU;
    const int grid = gridDim.x;
    const int wg = xcd_local_wg(blockIdx.x, grid);
    const int u0 = range_start(p, wg, grid);
    const int u1 = range_start(p, wg + 1, grid);
    const int c_first = tile_of(p, u0);
    const int c_last = tile_of(p, u1 - 1);
    const int k0 = u0 - c_first * KU;
    const int k1 = u1 - c_last * KU;

    // Tile c: column tile c / rg (128 columns, packed tiles 2 (c / rg) and
    // 2 (c / rg) + 1), row group c % rg (64 rows).
    const uint32_t RG = (uint32_t)p.rg;
    auto col_of = [&](int c) -> uint32_t { return RG == 1 ? (uint32_t)c : (uint32_t)c / RG; };
    auto ptile_of = [&](int c) -> uint32_t { return col_of(c) * 2u + (uint32_t)hf; };
    auto w_tile = [&](int c) -> uint32_t { return ptile_of(c) * (uint32_t)KU * 4096u; };
    auto s_tile = [&](int c) -> uint32_t { return (ptile_of(c) * (uint32_t)p.G) << 7; };
    auto row0_of = [&](int c) -> int { return RG == 1 ? 0 : (int)((uint32_t)c - col_of(c) * RG) * 64; };
    auto rows_of = [&](int c) -> int {
        const int r = p.M - row0_of(c);
        return r < 64 ? r : 64;
    };

    const uint32_t w_lane = (uint32_t)ks * 4096u + (uint32_t)lane * 16u;
    // Scale runs: lane group g of the packed 128-byte row holds, for each
    // 16-column block, the scales of columns 4g .. 4g + 3; the weight operand's
    // column is lane % 16, so a lane loads run (lane % 16) / 4 and keeps
    // element lane % 4 of it (one v_perm per block).
    const uint32_t s_lane = (uint32_t)((lane & 15) >> 2) * 32u;
    const uint32_t s_sel = 0x01000100u + (uint32_t)(lane & 3) * 0x02020202u;
    // Direct-to-LDS loads: load i of the block (0..15) brings rows 4i .. 4i + 3,
    // lane l row 4i + l/16, 16-byte chunk (l % 16) ^ row (XOR swizzle); this
    // wave issues loads 8 hf .. 8 hf + 7, and loads q, q + 4 are 16 rows
    // apart with the same swizzle.
    uint32_t a_dma[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int r = 4 * (8 * hf + q) + lg;
        a_dma[q] = (uint32_t)(r * p.K + (((lane & 15) ^ (r & 15)) * 8)) * 2u + (uint32_t)ks * 256u;
    }
    const uint32_t a_rows16 = (uint32_t)p.K * 32u;
    const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint8_t *)a_lds;
    const uint32_t lds_pair = lds0 + (uint32_t)(ks * D * kAStage);  // the pair's ring
    // Operand reads, k-step t: row mb*16 + l%16, chunk (4t + l/16) ^ (l%16);
    // the slot and the row block are instruction offsets.
    uint32_t a_rd[4];
#pragma unroll
    for (int t = 0; t < 4; ++t)
        a_rd[t] = lds_pair + (uint32_t)((lane & 15) * 256) + (uint32_t)(((4 * t + lg) ^ (lane & 15)) << 4);
    const uint32_t w_bytes = (uint32_t)p.K * (uint32_t)(p.N / 2);
    const uint32_t s_bytes = (uint32_t)p.G * (uint32_t)p.N * 2u;

    u32x4_t wr[D][NBW];
    half8_t sr[D][2];

    // ---- load cursor (work-group uniform) ----
    int ld_c = c_first, ld_ku = k0;
    int ld_end = (c_first == c_last) ? k1 : KU;
    uint32_t ld_w = w_tile(ld_c) + (uint32_t)ld_ku * 4096u;
    uint32_t ld_s = s_tile(ld_c);
    const uint16_t *ld_a = p.A + (int64_t)row0_of(ld_c) * p.K;
    uint32_t a_bytes = (uint32_t)rows_of(ld_c) * (uint32_t)p.K * 2u;

    auto issue = [&](int j) {
        const int my = ld_ku + ks;
        const bool on = my < ld_end;
        {  // first, so a stage's LDS rows are its oldest loads
            const __amdgpu_buffer_rsrc_t rd =
                __builtin_amdgcn_make_buffer_rsrc((void *)ld_a, (short)0, on ? a_bytes : 0u, kBufferFlags);
            uint32_t slot = lds_pair;
            asm volatile("" : "+s"(slot));
            slot += (uint32_t)(j * kAStage + hf * 8192);
            uint32_t dma[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                dma[q] = a_dma[q];
                asm volatile("" : "+v"(dma[q]));  // formed per stage, not held
            }
#pragma unroll
            for (int q = 0; q < kADma; ++q)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(
                    rd, (__attribute__((address_space(3))) void *)(uintptr_t)(slot + (uint32_t)(q * 1024)), 16,
                    (int)(dma[q & 3] + (uint32_t)(q >> 2) * a_rows16), ld_ku * 256, 0, 0);
        }
        issue_order_point();
        const __amdgpu_buffer_rsrc_t rw =
            __builtin_amdgcn_make_buffer_rsrc((void *)p.W, (short)0, on ? w_bytes : 0u, kBufferFlags);
#pragma unroll
        for (int b = 0; b < NBW; ++b)
            wr[j][b] = __builtin_bit_cast(
                u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rw, w_lane + b * 1024, ld_w, kAuxNonTemporal));
        if constexpr (!PER_CHANNEL) {
            const __amdgpu_buffer_rsrc_t rs =
                __builtin_amdgcn_make_buffer_rsrc((void *)p.S, (short)0, on ? s_bytes : 0u, kBufferFlags);
            const uint32_t s_off = ld_s + ((uint32_t)scale_row_of(my, p) << 7);
#pragma unroll
            for (int i = 0; i < 2; ++i)
                sr[j][i] = __builtin_bit_cast(half8_t, __builtin_amdgcn_raw_buffer_load_b128(rs, s_lane + i * 16,
                                                                                             s_off, 0));
        }
        issue_order_point();  // stages do not interleave
    };
    auto advance_ld = [&]() {
        ld_ku += KS;
        ld_w += KS * 4096u;
        if (ld_ku >= ld_end) {  // next segment
            ld_c += 1;
            ld_ku = 0;
            ld_end = (ld_c < c_last) ? KU : (ld_c == c_last) ? k1 : 0;
            ld_w = w_tile(ld_c);
            ld_s = s_tile(ld_c);
            if (RG > 1 && ld_end > 0) {
                ld_a = p.A + (int64_t)row0_of(ld_c) * p.K;
                a_bytes = (uint32_t)rows_of(ld_c) * (uint32_t)p.K * 2u;
            }
        }
    };

#pragma unroll
    for (int j = 0; j < D; ++j) {
        issue(j);
        advance_ld();
    }

    const int n_st = (c_first == c_last)
                         ? (k1 - k0 + KS - 1) / KS
                         : (KU - k0 + KS - 1) / KS + (c_last - c_first - 1) * ((KU + KS - 1) / KS) +
                               (k1 + KS - 1) / KS;

    float4_t acc[NBW][MB];
#pragma unroll
    for (int b = 0; b < NBW; ++b)
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) acc[b][mb] = float4_t{0.f, 0.f, 0.f, 0.f};
    const float4_t zero4 = {0.f, 0.f, 0.f, 0.f};
    const DequantConsts dq = dequant_consts();

    // One stage (ring slot j, `later` stages issued after it).  Every wave
    // passes both barriers, also one whose block lies past the segment.
    auto compute = [&](int j, int later, bool active) {
        // this wave's rows of the stage have landed (the loads issued after
        // them are the stage's weight and scale loads and `later` stages);
        // the barrier waits for the partner's
        wait_vmcnt_n(later * kLoads + kWL + kSL);
        __builtin_amdgcn_s_barrier();
        u32x4_t v[4 * MB];
        if (active) {
#pragma unroll
            for (int mb = 0; mb < MB; ++mb)
#pragma unroll
                for (int t = 0; t < 4; ++t)
                    asm volatile("ds_read_b128 %0, %1 offset:%2"
                                 : "=v"(v[mb * 4 + t])
                                 : "v"(a_rd[t]), "i"(j * kAStage + mb * 4096));
            asm volatile("s_waitcnt lgkmcnt(0)"
                         : "+v"(v[0]), "+v"(v[1]), "+v"(v[2]), "+v"(v[3]), "+v"(v[4]), "+v"(v[5]), "+v"(v[6]),
                           "+v"(v[7]), "+v"(v[8]), "+v"(v[9]), "+v"(v[10]), "+v"(v[11]), "+v"(v[12]),
                           "+v"(v[13]), "+v"(v[14]), "+v"(v[15])::"memory");
        }
        // both waves of the pair have their rows: the slot may be refilled
        __builtin_amdgcn_s_barrier();
        if (!active) return;
        half2_t s2[NBW];
        if constexpr (!PER_CHANNEL) {
#pragma unroll
            for (int b = 0; b < NBW; ++b) {
                const u32x4_t u = __builtin_bit_cast(u32x4_t, sr[j][b >> 1]);
                s2[b] = as_h2(__builtin_amdgcn_perm(u[2 * (b & 1) + 1], u[2 * (b & 1)], s_sel));
            }
        }
#pragma unroll
        for (int t = 0; t < 4; ++t) {
#pragma unroll
            for (int b = 0; b < NBW; ++b) {
                half8_t w = dequant_magic(wr[j][b][t], dq);
                if constexpr (!PER_CHANNEL) w = scale_weights(w, s2[b]);
#pragma unroll
                for (int mb = 0; mb < MB; ++mb)
                    acc[b][mb] = mfma(w, __builtin_bit_cast(half8_t, v[mb * 4 + t]), acc[b][mb]);
            }
        }
    };

    // After the reduction wave (ks, hf) holds row block ks of the column
    // blocks of its half hf: tile block (4 hf + j) * MB + ks for j = 0..3.
    auto own = [&](int j) { return (4 * hf + j) * MB + ks; };
    auto store_c = [&](int c, const float4_t *out) {
        const int r0 = row0_of(c), rows = rows_of(c);
        const int col = (int)col_of(c);
#pragma unroll
        for (int j = 0; j < kOwn; ++j) {
            const int blk = own(j);
            const int b = blk / MB, mb = blk % MB;
            const int m = mb * 16 + (lane & 15);
            if (m < rows) {
                const int nbg = col * 8 + b;
                float4_t v = out[j];
                if constexpr (PER_CHANNEL) {
                    const half4_t s4 = *(const half4_t *)(p.S + (int64_t)(nbg >> 2) * 64 + lg * 16 + (nbg & 3) * 4);
#pragma unroll
                    for (int i = 0; i < 4; ++i) v[i] *= (float)s4[i];
                }
                const half4_t h = {(_Float16)v[0], (_Float16)v[1], (_Float16)v[2], (_Float16)v[3]};
                *(half4_t *)(p.C + (int64_t)(r0 + m) * p.N + nbg * 16 + lg * 4) = h;
            }
        }
    };

    constexpr int kSlotFloats = 2 * NBW * MB * 256;  // the tile's 32 blocks
    float *const my_slots = p.partials + (int64_t)wg * 2 * kSlotFloats;
    bool has_first = false, has_last = false;
    float4_t last_out[kOwn];
#pragma unroll
    for (int j = 0; j < kOwn; ++j) last_out[j] = zero4;

    int cp_c = c_first, cp_ku = k0, cp_begin = k0;
    int cp_end = (c_first == c_last) ? k1 : KU;

    // A segment is complete: the four waves of each column half sum their
    // tiles in ring slot j, which every pair has read (its refill is issued
    // after the last barrier here; the other slot may be receiving the next
    // stage).  Wave (ks, hf) writes into the half of the pair's slot its
    // own loads fill, in two rounds of eight blocks (column blocks 2r, 2r + 1).
    auto finish_segment = [&](int j) {
        float4_t out[kOwn];
        const auto area = [&](int k2, int h2) {
            return reinterpret_cast<float4_t *>(a_lds + (k2 * D + j) * kAStage + h2 * 8192);
        };
        float4_t *const mine = area(ks, hf);
#pragma unroll
        for (int r = 0; r < 2; ++r) {
#pragma unroll
            for (int c = 0; c < 2; ++c)
#pragma unroll
                for (int mb = 0; mb < MB; ++mb) mine[(c * MB + mb) * 64 + lane] = acc[2 * r + c][mb];
            lds_barrier();
#pragma unroll
            for (int c = 0; c < 2; ++c) {
                const int at = (c * MB + ks) * 64 + lane;
                float4_t s = area(0, hf)[at];
#pragma unroll
                for (int k2 = 1; k2 < KS; ++k2) s += area(k2, hf)[at];
                out[2 * r + c] = s;
            }
            lds_barrier();
        }
#pragma unroll
        for (int b = 0; b < NBW; ++b)
#pragma unroll
            for (int mb = 0; mb < MB; ++mb) acc[b][mb] = zero4;
        if (cp_begin == 0 && cp_end == KU) {
            store_c(cp_c, out);
        } else if (cp_c == c_last) {
            has_last = true;
#pragma unroll
            for (int j2 = 0; j2 < kOwn; ++j2) last_out[j2] = out[j2];
        } else {
            has_first = true;
#pragma unroll
            for (int j2 = 0; j2 < kOwn; ++j2) store_partial(my_slots, own(j2), lane, out[j2]);
        }
    };

    auto step = [&](int j, int st, int later) {
        if (st < n_st) {
            compute(j, later, cp_ku + ks < cp_end);
            if (cp_ku + KS >= cp_end) {
                if (cp_c != c_last) {  // the last segment is closed after the loop
                    finish_segment(j);
                    cp_c += 1;
                    cp_ku = 0;
                    cp_begin = 0;
                    cp_end = (cp_c < c_last) ? KU : k1;
                }
            } else {
                cp_ku += KS;
            }
        }
    };
    const int st_last = (n_st - 1) / D * D;
    for (int st0 = 0; st0 < st_last; st0 += D) {
#pragma unroll
        for (int j = 0; j < D; ++j) {
            step(j, st0 + j, D - 1);
            issue(j);
            advance_ld();
        }
    }
#pragma unroll
    for (int j = 0; j < D; ++j) step(j, st_last + j, D - 1 - j);
    // Stages past the range were issued (through empty descriptors) but never
    // waited for: each wave drains its own before the ring is reused (a wave
    // writes only where its own loads land).
    wait_vmcnt<0>();
    finish_segment(0);

    auto own_slot = [&](int j) { return own(j); };
    combine_tiles<kOwn>(p, flags, wg, grid, kSlotFloats, lane, has_first, c_first, has_last, c_last, last_out,
                        own_slot, store_c);
}

}  // namespace

hipError_t launch_pair_gemm(const GemmConfig &cfg, const GemmProblem &p, hipStream_t stream)
{
    if (cfg.sparse || cfg.mb != 4 || cfg.nb != 8) return hipErrorInvalidValue;
    GemmProblem arg = p;
    void *args[] = {&arg};
    const void *fn = p.group_units == 0 ? (const void *)&w4a16_pair_kernel<true>
                                        : (const void *)&w4a16_pair_kernel<false>;
    return hipLaunchKernel(fn, dim3(cfg.grid), dim3(512), args, 0, stream);
}

void pair_kernel_name(bool per_channel, char *buf, size_t n)
{
    snprintf(buf, n, "w4a16_pair_kernel<%s>", per_channel ? "true" : "false");
}

}  // namespace marlin
