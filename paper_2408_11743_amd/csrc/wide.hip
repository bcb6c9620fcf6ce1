// W4A16 GEMM for gfx950 at batches of 33 rows and more, where every
// dequantized weight must feed many rows of A:
// C[M,N] = A[M,K] * (s * (q - 8)), fp32 accumulation.
//
//  * A work-group of four waves (one per SIMD) owns a tile of 16*MBW rows x
//    4*16*NBW columns; each wave owns 16*MBW rows x 16*NBW columns, 32
//    16x16 accumulator blocks (MBW * NBW = 32).  The accumulators are touched
//    by the MFMAs only (no per-stage fp32 fold), so the compiler may keep
//    them in the accumulation registers and every dequantized weight feeds
//    MBW MFMAs.
//  * Group scales multiply the dequantized fp16 weights: (q - 8) is exact
//    (the paper's magic number, Section 3.4 "Dequantization and Tensor
//    Cores": the code ORed into 1024.0, minus 1032; the upper nibble gives
//    1024 + 16q, fixed by one exact fma), then one fp16 multiply by s per two
//    weights, rounded once ("Groups and Instruction Ordering": scales applied
//    to the weights before the matrix product).  Per-channel scales multiply
//    the final fp32 sums.
//  * Weights stream from HBM straight into a P-deep register ring per wave
//    (16-byte non-temporal loads; a wave's weights are its own, so nothing
//    is gained by staging them in LDS).  The activation block of a stage
//    (16*MBW rows x 128 k) and the stage's group scales arrive by gfx950
//    direct-to-LDS loads in a P-deep LDS ring shared by the four waves, one
//    barrier per stage (Section 3.4 "Memory Load Pipelining"); the
//    activation rows are XOR-swizzled so that the MFMA-operand reads of 16
//    rows hit 16 bank groups.
//  * Partition (whole tiles or Stream-K ranges of 128-row blocks) and the
//    combination of shared tiles are the other kernels' (device.h).
#include <hip/hip_runtime.h>
#include <stdio.h>

#include "device.h"
#include "internal.h"

namespace marlin {
namespace {

using namespace dev;

template <int MBW, int NBW, int P>
struct WideShape {
    static constexpr int NW = 4;                   // waves per work-group, all along N
    static constexpr int TR = 16 * MBW;            // rows of A per tile
    static constexpr int kABytes = TR * 256;       // one block of A: TR rows x 128 k x 2 B
    static constexpr int kSBytes = NW * 1024;      // the stage's group scales: 1 KiB per wave
    static constexpr int kStage = kABytes + kSBytes;
    static constexpr int kDmaA = TR / (4 * NW);    // 1 KiB direct-to-LDS A loads per wave and stage
    static_assert(MBW * NBW == 32, "32 accumulator blocks per wave");
    static_assert(NBW == 4 || NBW == 8, "one or two packed 64-column tiles per wave");
    static_assert(kDmaA >= 1, "activation rows per wave");
    static_assert(P >= 3 && P * kStage <= 160 * 1024 - 64, "LDS ring");
};

// Eight codes of one word -> the fp16 weights s * (q - 8), element order
// j = 0..7 (code j in nibble (j >> 1) + 4 (j & 1)): q - 8 exactly by the
// magic number, then one rounding of the product with the scale.
__device__ __forceinline__ half8_t dequant_scaled(uint32_t x, half2_t s2, const DequantConsts &k)
{
    const half2_t sub = {(_Float16)1032.0f, (_Float16)1032.0f};
    const half2_t mul = {(_Float16)0.0625f, (_Float16)0.0625f};
    const half2_t add = {(_Float16)-72.0f, (_Float16)-72.0f};
    const uint32_t y = x >> 8;
    const half2_t r0 = (as_h2((x & k.lo) | k.ex) - sub) * s2;
    const half2_t r1 = __builtin_elementwise_fma(as_h2((x & k.hi) | k.ex), mul, add) * s2;
    const half2_t r2 = (as_h2((y & k.lo) | k.ex) - sub) * s2;
    const half2_t r3 = __builtin_elementwise_fma(as_h2((y & k.hi) | k.ex), mul, add) * s2;
    return half8_t{r0.x, r0.y, r1.x, r1.y, r2.x, r2.y, r3.x, r3.y};
}

// One quarter (codes 2q and 2q + 1) of dequant_scaled (SCALED), or of the
// exact magic-number conversion alone (per-channel scales multiply the sums).
template <bool SCALED>
__device__ __forceinline__ half2_t convert_quarter(uint32_t x, int q, half2_t s2, const DequantConsts &k)
{
    const half2_t sub = {(_Float16)1032.0f, (_Float16)1032.0f};
    const half2_t mul = {(_Float16)0.0625f, (_Float16)0.0625f};
    const half2_t add = {(_Float16)-72.0f, (_Float16)-72.0f};
    const uint32_t y = (q >> 1) ? x >> 8 : x;
    const half2_t r = (q & 1) == 0 ? as_h2((y & k.lo) | k.ex) - sub
                                   : __builtin_elementwise_fma(as_h2((y & k.hi) | k.ex), mul, add);
    return SCALED ? r * s2 : r;
}

template <int MBW, int NBW, int P, bool PER_CHANNEL>
__global__ void __launch_bounds__(256, 1) w4a16_wide_kernel(GemmProblem p)
{
    using S = WideShape<MBW, NBW, P>;
    constexpr int NW = S::NW;
    constexpr int TR = S::TR;
    constexpr int kABytes = S::kABytes;
    constexpr int kStage = S::kStage;
    constexpr int kDmaA = S::kDmaA;
    constexpr int kSL = PER_CHANNEL ? 0 : 1;           // direct-to-LDS scale loads per wave and stage
    constexpr int kLoads = kDmaA + kSL + NBW;          // vector-memory ops per wave and stage
    static_assert(NBW + (P - 2) * kLoads <= 63, "vmcnt range");
    constexpr int kBlocks = NBW * MBW;                 // 16x16 output blocks per wave
    __shared__ __attribute__((aligned(16))) uint8_t ring[P * kStage];
    __shared__ int flags[2];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int lg = lane >> 4;
    const DequantConsts dq = dequant_consts();
    const int KU = p.KU;
    const int grid = gridDim.x;
    const int wg = xcd_local_wg(blockIdx.x, grid);
    const int u0 = range_start(p, wg, grid);
    const int u1 = range_start(p, wg + 1, grid);
    const int c_first = tile_of(p, u0);
    const int c_last = tile_of(p, u1 - 1);
    const int k0 = u0 - c_first * KU;
    const int k1 = u1 - c_last * KU;
    const int n_st = (c_first == c_last) ? (k1 - k0) : (KU - k0) + (c_last - c_first - 1) * KU + k1;

    // Tile c: column group c / rg (64 * NBW * NW columns), row group c % rg (TR rows).
    const uint32_t RG = (uint32_t)p.rg;
    auto cg_of = [&](int c) -> uint32_t { return RG == 1 ? (uint32_t)c : (uint32_t)c / RG; };
    auto row0_of = [&](int c) -> int { return RG == 1 ? 0 : (int)((uint32_t)c - cg_of(c) * RG) * TR; };
    auto rows_of = [&](int c) -> int {
        const int r = p.M - row0_of(c);
        return r < TR ? r : TR;
    };
    // this wave's first packed 64-column tile (NBW / 4 of them)
    auto ptile_of = [&](int c) -> uint32_t { return (cg_of(c) * NW + (uint32_t)wave) * (uint32_t)(NBW / 4); };

    // ---- per-lane address parts ----
    const uint32_t w_lane = (uint32_t)lane * 16u;
    const uint32_t w_next = (uint32_t)KU * 4096u;  // the next packed tile's weights
    const uint32_t w_bytes = (uint32_t)p.K * (uint32_t)(p.N / 2);
    const uint32_t s_bytes = (uint32_t)p.G * (uint32_t)p.N * 2u;
    // A: load i of this wave brings rows r = wave*TR/4 + 4i + lg, lane chunk
    // (lane % 16) of row r holding the global chunk (lane % 16) ^ (r % 16)
    uint32_t a_dma[kDmaA];
#pragma unroll
    for (int i = 0; i < kDmaA; ++i) {
        const int r = wave * (TR / NW) + 4 * i + lg;
        a_dma[i] = (uint32_t)(r * p.K + (((lane & 15) ^ (r & 15)) * 8)) * 2u;
    }
    // scales: lane L % 16 brings 16 bytes of its wave's scale run: packed tile
    // (L % 16) / 8 (NBW = 8; else 0), chunk L % 8 of the 128-byte row; the
    // other lanes repeat those loads
    const uint32_t s_lane =
        (NBW == 8 ? (uint32_t)((lane & 15) >> 3) * (uint32_t)p.G * 128u : 0u) + (uint32_t)(lane & 7) * 16u;
    const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint8_t *)ring;
    // MFMA operand reads: row mb*16 + (lane % 16), chunk (4t + lg) ^ (lane % 16)
    uint32_t a_rd[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) a_rd[t] = lds0 + (uint32_t)((lane & 15) * 256 + (((4 * t + lg) ^ (lane & 15)) << 4));
    // this lane's column scale of block nb: packed tile nb / 4, byte
    // (cn / 4) * 32 + ((nb % 4) * 4 + cn % 4) * 2 of its 128-byte row, cn = lane % 16
    const uint32_t s_rd = lds0 + (uint32_t)(kABytes + wave * 1024 + ((lane & 15) >> 2) * 32 + (lane & 3) * 2);

    u32x4_t wr[P][NBW];

    // ---- load cursor ----
    int ld_c = c_first, ld_ku = k0;
    int ld_end = (c_first == c_last) ? k1 : KU;
    uint32_t ld_w = (ptile_of(ld_c) * (uint32_t)KU + (uint32_t)ld_ku) << 12;
    uint32_t ld_s = ptile_of(ld_c) * (uint32_t)p.G * 128u;
    const uint16_t *ld_a = p.A + (int64_t)row0_of(ld_c) * p.K;
    uint32_t a_bytes = (uint32_t)rows_of(ld_c) * (uint32_t)p.K * 2u;
    const uint32_t a_dst0 = lds0 + (uint32_t)(wave * (TR / NW) * 256);
    const uint32_t s_dst0 = lds0 + (uint32_t)(kABytes + wave * 1024);

    auto issue = [&](int j) {
        const bool on = ld_ku < ld_end;
        uint32_t a_base = a_dst0, s_base = s_dst0;
        asm volatile("" : "+s"(a_base), "+s"(s_base));
        {  // activation rows, then the scales: the stage's direct-to-LDS loads
            const __amdgpu_buffer_rsrc_t ra =
                __builtin_amdgcn_make_buffer_rsrc((void *)ld_a, (short)0, on ? a_bytes : 0u, kBufferFlags);
            const uint32_t dst = a_base + (uint32_t)(j * kStage);
#pragma unroll
            for (int i = 0; i < kDmaA; ++i)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(
                    ra, (__attribute__((address_space(3))) void *)(uintptr_t)(dst + (uint32_t)(i * 1024)), 16,
                    (int)a_dma[i], ld_ku * 256, 0, 0);
            if constexpr (!PER_CHANNEL) {
                const __amdgpu_buffer_rsrc_t rs =
                    __builtin_amdgcn_make_buffer_rsrc((void *)p.S, (short)0, on ? s_bytes : 0u, kBufferFlags);
                const uint32_t s_off = ld_s + ((uint32_t)scale_row_of(ld_ku, p) << 7);
                __builtin_amdgcn_raw_ptr_buffer_load_lds(
                    rs, (__attribute__((address_space(3))) void *)(uintptr_t)(s_base + (uint32_t)(j * kStage)), 16,
                    (int)s_lane, (int)s_off, 0, 0);
            }
        }
        issue_order_point();  // the direct-to-LDS loads are the stage's oldest
        const __amdgpu_buffer_rsrc_t rw =
            __builtin_amdgcn_make_buffer_rsrc((void *)p.W, (short)0, on ? w_bytes : 0u, kBufferFlags);
#pragma unroll
        for (int b = 0; b < NBW; ++b)
            wr[j][b] = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(
                                                       rw, w_lane + (b & 3) * 1024, ld_w + (b >> 2) * w_next,
                                                       kAuxNonTemporal));
        issue_order_point();  // stages do not interleave
    };
    auto advance_ld = [&]() {
        ld_ku += 1;
        ld_w += 4096u;
        if (ld_ku >= ld_end) {  // next tile
            ld_c += 1;
            ld_ku = 0;
            ld_end = (ld_c < c_last) ? KU : (ld_c == c_last) ? k1 : 0;  // 0: past the range
            ld_w = (ptile_of(ld_c) * (uint32_t)KU) << 12;
            ld_s = ptile_of(ld_c) * (uint32_t)p.G * 128u;
            if (ld_end > 0) {
                ld_a = p.A + (int64_t)row0_of(ld_c) * p.K;
                a_bytes = (uint32_t)rows_of(ld_c) * (uint32_t)p.K * 2u;
            }
        }
    };

#pragma unroll
    for (int j = 0; j < P - 1; ++j) {
        issue(j);
        advance_ld();
    }

    float4_t acc[NBW][MBW];
    const float4_t zero4 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int b = 0; b < NBW; ++b)
#pragma unroll
        for (int mb = 0; mb < MBW; ++mb) acc[b][mb] = zero4;

    // One stage (ring slot j): the column scales first (group scales), then
    // per k-step the MBW activation operands (read one k-step ahead) and, per
    // column block, one dequantized word feeding MBW MFMAs.
    auto compute = [&](int j) {
        uint32_t sv[PER_CHANNEL ? 1 : NBW];
        if constexpr (!PER_CHANNEL) {
#pragma unroll
            for (int b = 0; b < NBW; ++b)
                asm volatile("ds_read_u16 %0, %1 offset:%2"
                             : "=v"(sv[b])
                             : "v"(s_rd + (uint32_t)(j * kStage)), "i"((b >> 2) * 128 + (b & 3) * 8));
        }
        u32x4_t a[2][MBW];
        auto read_a = [&](int t, u32x4_t (&dst)[MBW]) {
#pragma unroll
            for (int mb = 0; mb < MBW; ++mb)
                asm volatile("ds_read_b128 %0, %1 offset:%2"
                             : "=v"(dst[mb])
                             : "v"(a_rd[t] + (uint32_t)(j * kStage)), "i"(mb * 4096));
        };
        read_a(0, a[0]);
        half2_t s2[NBW] = {};  // group scales (unused with per-channel scales)
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            u32x4_t(&cur)[MBW] = a[t & 1];
            // this k-step's operands (and at t = 0 the scales) are complete;
            // the next step's reads are issued before its MFMAs so that they
            // overlap them.  The empty asm "redefines" what the wait made
            // available, so no use is scheduled before it.
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
            for (int mb = 0; mb < MBW; ++mb) asm volatile("" : "+v"(cur[mb]));
            if constexpr (!PER_CHANNEL) {
                if (t == 0) {
#pragma unroll
                    for (int b = 0; b < NBW; ++b) {
                        asm volatile("" : "+v"(sv[b]));
                        s2[b] = as_h2(sv[b] | (sv[b] << 16));
                    }
                }
            }
            if (t < 3) read_a(t + 1, a[(t + 1) & 1]);
            // Column block b's MFMAs are interleaved with the conversion of
            // block b + 1's word, one quarter after every other MFMA: the
            // conversion does not depend on the MFMAs, so the SIMD issues
            // it while the matrix core works (the wave issues in order, so
            // a run of MFMAs would hold back the conversion behind them).
            half2_t nx[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) nx[q] = convert_quarter<!PER_CHANNEL>(wr[j][0][t], q, s2[0], dq);
#pragma unroll
            for (int b = 0; b < NBW; ++b) {
                const half8_t w = {nx[0].x, nx[0].y, nx[1].x, nx[1].y, nx[2].x, nx[2].y, nx[3].x, nx[3].y};
#pragma unroll
                for (int mb = 0; mb < MBW; ++mb) {
                    acc[b][mb] = mfma(w, __builtin_bit_cast(half8_t, cur[mb]), acc[b][mb]);
                    constexpr int kStep = MBW / 4;  // MFMAs per quarter
                    if (b + 1 < NBW && mb % kStep == 0)
                        nx[mb / kStep] = convert_quarter<!PER_CHANNEL>(wr[j][b + 1][t], mb / kStep,
                                                                       s2[b + 1], dq);
                    __builtin_amdgcn_sched_barrier(0);
                }
            }
        }
    };

    // block j of this wave = column block j / MBW, row block j % MBW; slot index wave*kBlocks + j
    auto own = [&](int j) { return wave * kBlocks + j; };
    auto store_c = [&](int c, const float4_t *out) {
        const int r0 = row0_of(c), rows = rows_of(c);
        const uint32_t pt = ptile_of(c);
        half8_t cs[NBW / 4][2];
        if constexpr (PER_CHANNEL) {
            // the output lane's 16 column scales of each packed tile (32 bytes)
#pragma unroll
            for (int i = 0; i < NBW / 4; ++i) {
                const _Float16 *src = (const _Float16 *)p.S + (int64_t)(pt + i) * 64 + lg * 16;
                cs[i][0] = *(const half8_t *)src;
                cs[i][1] = *(const half8_t *)(src + 8);
            }
        }
#pragma unroll
        for (int jb = 0; jb < kBlocks; ++jb) {
            const int b = jb / MBW, mb = jb % MBW;
            const int m = mb * 16 + (lane & 15);
            if (m < rows) {
                float4_t vv = out[jb];
                if constexpr (PER_CHANNEL) {
                    const int e = (b & 3) * 4;
#pragma unroll
                    for (int i = 0; i < 4; ++i) vv[i] *= (float)cs[b >> 2][e >> 3][(e & 7) + i];
                }
                const half4_t h = {(_Float16)vv[0], (_Float16)vv[1], (_Float16)vv[2], (_Float16)vv[3]};
                *(half4_t *)(p.C + (int64_t)(r0 + m) * p.N + (int64_t)(pt * 64 + b * 16 + lg * 4)) = h;
            }
        }
    };

    const int slot_floats = NW * kBlocks * 256;
    float *const my_slots = p.partials + (int64_t)wg * 2 * slot_floats;  // slot 0; slot 1 follows
    bool has_first = false, has_last = false;

    int cp_c = c_first, cp_ku = k0, cp_begin = k0;
    int cp_end = (c_first == c_last) ? k1 : KU;
    // A segment is complete: write C (whole tile) or slot 0 (shared first
    // tile).  A shared last tile stays in acc; it is combined after the loop.
    auto finish_segment = [&]() {
        const bool partial = cp_begin != 0 || cp_end != KU;
        if (partial && cp_c == c_last) {
            has_last = true;
            return;
        }
        float4_t out[kBlocks];
#pragma unroll
        for (int jb = 0; jb < kBlocks; ++jb) {
            out[jb] = acc[jb / MBW][jb % MBW];
            acc[jb / MBW][jb % MBW] = zero4;
        }
        if (partial) {
            has_first = true;
#pragma unroll
            for (int jb = 0; jb < kBlocks; ++jb) store_partial(my_slots, own(jb), lane, out[jb]);
        } else {
            store_c(cp_c, out);
        }
    };

    // Stage st (ring slot j) with `later` stages issued after it; `refill`:
    // the slot of stage st - 1 takes stage st + P - 1.  The wait covers this
    // wave's direct-to-LDS loads of the stage (issued before its own weight
    // loads and the later stages'; vector-memory operations complete in
    // order); the barrier makes every wave's loads of the stage visible and
    // frees the slot of stage st - 1.  Loads are issued unconditionally (past
    // the range through empty descriptors, into a slot no wave reads again)
    // so that every stage has the same load pattern.
    auto step = [&](int j, int st, int later, bool refill) {
        const bool live = st < n_st;
        if (live) {
            wait_vmcnt_n(NBW + later * kLoads);
            __builtin_amdgcn_s_barrier();
            asm volatile("" ::: "memory");
        }
        if (refill) {
            issue((j + P - 1) % P);
            advance_ld();
        }
        if (live) {
            compute(j);
            if (cp_ku + 1 >= cp_end) {
                finish_segment();
                cp_c += 1;
                cp_ku = 0;
                cp_begin = 0;
                cp_end = (cp_c < c_last) ? KU : k1;
            } else {
                cp_ku += 1;
            }
        }
    };
    const int st_last = (n_st - 1) / P * P;
    for (int st0 = 0; st0 < st_last; st0 += P) {
#pragma unroll
        for (int j = 0; j < P; ++j) step(j, st0 + j, P - 2, true);
    }
#pragma unroll
    for (int j = 0; j < P; ++j) step(j, st_last + j, j == 0 ? P - 2 : P - 1 - j, j == 0);

    float4_t last_out[kBlocks];
#pragma unroll
    for (int jb = 0; jb < kBlocks; ++jb) last_out[jb] = acc[jb / MBW][jb % MBW];
    auto own_slot = [&](int jb) { return own(jb); };
    combine_tiles<kBlocks>(p, flags, wg, grid, slot_floats, lane, has_first, c_first, has_last, c_last, last_out,
                           own_slot, store_c);
}

template <int MBW, int NBW, int P>
hipError_t launch_wide(const GemmConfig &cfg, const GemmProblem &p, hipStream_t stream)
{
    GemmProblem arg = p;
    void *args[] = {&arg};
    const void *fn = (p.group_units == 0) ? (const void *)&w4a16_wide_kernel<MBW, NBW, P, true>
                                          : (const void *)&w4a16_wide_kernel<MBW, NBW, P, false>;
    return hipLaunchKernel(fn, dim3(cfg.grid), dim3(256), args, 0, stream);
}

// Ring depth per shape: what the LDS holds (64-row tiles: 20 KiB per stage;
// 128-row tiles: 36 KiB) and the register ring affords (NBW words of 16
// bytes per lane and stage).
template <int MBW, int NBW>
constexpr int wide_depth()
{
    return MBW == 4 ? 3 : 4;
}

}  // namespace

hipError_t launch_wide_gemm(const GemmConfig &cfg, const GemmProblem &p, hipStream_t stream)
{
    switch (cfg.mb * 10 + cfg.nb) {
    case 48: return launch_wide<4, 8, wide_depth<4, 8>()>(cfg, p, stream);
    case 84: return launch_wide<8, 4, wide_depth<8, 4>()>(cfg, p, stream);
    default: return hipErrorInvalidValue;
    }
}

void wide_kernel_name(const GemmConfig &cfg, bool per_channel, char *buf, size_t n)
{
    int d = 0;
    switch (cfg.mb * 10 + cfg.nb) {
    case 48: d = wide_depth<4, 8>(); break;
    case 84: d = wide_depth<8, 4>(); break;
    default: break;
    }
    if (!d) {
        if (n) buf[0] = 0;
        return;
    }
    snprintf(buf, n, "w4a16_wide_kernel<%d, %d, %d, %s>", cfg.mb, cfg.nb, d, per_channel ? "true" : "false");
}

}  // namespace marlin
