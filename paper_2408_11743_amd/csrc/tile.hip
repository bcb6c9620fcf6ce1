// W4A16 GEMM for gfx950 at larger batches (tiles of 16 to 128 rows of A):
// C[M,N] = A[M,K] * (s * (q - 8)), fp32 accumulation.
//
// Where the stream kernel is bound by its per-weight VALU work (it serves at
// most 32 rows per dequantized weight), this kernel gives every wave a 64 x 64
// output tile: each dequantized weight feeds four MFMAs, and the work is
// bound by the matrix cores.
//  * A work-group of four waves owns a tile of 64*WN columns x 64*WM rows
//    (WN x WM waves, each 64 columns x 64 rows) over a range of 128-row blocks
//    of K (whole tiles or a Stream-K split, as for the stream kernel).
//  * The activation tile of a 128-row block (64*WM rows) is shared by the WN
//    waves of a row: gfx950's direct-to-LDS buffer loads stage it in a P-deep
//    LDS ring (each wave loads a quarter; one barrier per stage), XOR-swizzled
//    so that the MFMA-operand reads of 16 rows hit 16 bank groups ("Memory
//    Load Pipelining" of Section 3.4, with CDNA's direct-to-LDS loads in the
//    role of cp.async).
//  * Each wave streams its own 64 columns of packed weights (4 KiB per block)
//    with non-temporal direct-to-LDS loads into its own part of the ring
//    (registers are the scarce resource here: the 64x64 accumulators, the
//    activation operands and the fold's temporaries fill them) and reads them
//    back after the stage barrier.
//  * int4 -> fp16 with the paper's magic number ("Dequantization and Tensor
//    Cores"): the code ORed into the low mantissa bits of 1024.0 is 1024 + q,
//    minus 1032 gives q - 8; the next nibble gives 1024 + 16q, fixed by one
//    fma (x/16 - 72).  Exact, 9 VALU per 8 weights, no extra MFMA.
//  * Group scales multiply each 128-row fp32 product (v_fma_mix_f32); per-
//    channel scales multiply the final sum ("Groups and Instruction
//    Ordering").
//  * Tiles shared by work-groups are combined as in the stream kernel.
#include <hip/hip_runtime.h>
#include <stdio.h>

#include "device.h"
#include "internal.h"

namespace marlin {
namespace {

using namespace dev;

// One work-group stage covers KS consecutive 128-row blocks of K of one tile
// (fewer at the end of a segment: the blocks past it load zeros, which add
// exactly nothing).  Ring depth: stages that fit in LDS (activation rows,
// then each wave's weights, per block), capped so that the loads of the
// stages in flight stay within the vmcnt range.
template <int WN, int WM, int MBW, int NBW, int KS>
struct TileShape {
    static constexpr int NW = WN * WM;                    // waves per work-group
    static constexpr int TR = 16 * MBW * WM;              // rows of A per tile
    static constexpr int kABlock = TR * 256;              // one block of A (TR rows x 128 k x 2 B)
    static constexpr int kAStage = KS * kABlock;
    static constexpr int kWBlock = WN * NBW * 1024;       // the tile's weights for one block
    static constexpr int kWStage = KS * kWBlock;
    static constexpr int kStage = kAStage + kWStage;
    static constexpr int kDmaB = TR / (4 * NW);           // 1-KiB direct-to-LDS A loads per wave and block
    static constexpr int kWDma = NBW / WM;                // 1-KiB weight loads per wave and block (the
                                                          // WM waves of a column group share them)
    static constexpr int kScratch = (kDmaB + kWDma) * 1024;  // target of the loads issued past the end
    static constexpr int kSLB = NBW == 4 ? 2 : 1;         // scale loads per wave and block
    static constexpr int kLoads = KS * (kDmaB + kWDma + kSLB);  // vector-memory ops per wave per stage
    static_assert(kDmaB >= 1 && TR % (4 * NW) == 0, "activation rows per wave");
    static_assert(kWDma >= 1 && NBW % WM == 0, "weight blocks per wave");
    static constexpr int kSL = KS * kSLB;
    static constexpr int kLdsBudget = 160 * 1024 - 64;
    static constexpr int kByLds = (kLdsBudget - kScratch) / kStage;
    static constexpr int kByVm = (63 - kSL) / kLoads + 2;  // kSL + (P - 2) * kLoads <= 63
    static constexpr int kCap = 12;
    static constexpr int P = kByLds < kByVm ? (kByLds < kCap ? kByLds : kCap) : (kByVm < kCap ? kByVm : kCap);
    static_assert(P >= 3, "ring too shallow");
};

// This lane's column scales of one block: NBW column blocks x 4 values
// (element 4b + i: block b, output column 4 * (lane / 16) + i of the block).
template <int NBW>
struct ScaleFrag {
    half8_t v[2];
    __device__ __forceinline__ _Float16 at(int e) const { return v[e >> 3][e & 7]; }
};
template <>
struct ScaleFrag<1> {
    half4_t v;
    __device__ __forceinline__ _Float16 at(int e) const { return v[e & 3]; }
};

template <int WN, int WM, int MBW, int NBW, int KS, bool PER_CHANNEL>
__global__ void __launch_bounds__(64 * WN * WM, 1) w4a16_tile_kernel(GemmProblem p)
{
    static_assert(WN * WM == 4 || WN * WM == 8, "four or eight waves");
    static_assert(NBW == 1 || NBW == 2 || NBW == 4, "column blocks per wave");
    static_assert(MBW >= 1 && MBW <= 4, "row blocks per wave");
    static_assert(KS >= 1 && KS <= 4, "blocks per stage");
    using S = TileShape<WN, WM, MBW, NBW, KS>;
    constexpr int P = S::P;
    constexpr int TR = S::TR;
    constexpr int kABlock = S::kABlock;
    constexpr int kAStage = S::kAStage;
    constexpr int kWBlock = S::kWBlock;
    constexpr int kDmaB = S::kDmaB;
    constexpr int kWDma = S::kWDma;
    constexpr int NW = S::NW;
    constexpr int kStage = S::kStage;
    // Scale loads per wave and stage: one row per block, or (per-channel
    // scales, the same row for every block) one row per stage.  The ring
    // depth was sized with one row per block, an upper bound.
    constexpr int kSL = PER_CHANNEL ? S::kSLB : S::kSL;
    constexpr int kLoads = KS * (kDmaB + kWDma) + kSL;
    static_assert(kSL + (P - 2) * kLoads <= 63, "vmcnt range");
    constexpr int kBlocks = NBW * MBW;  // 16x16 output blocks per wave
    __shared__ __attribute__((aligned(16))) uint8_t a_lds[P * kStage + S::kScratch];
    __shared__ int flags[2];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int wn = wave % WN, wm = wave / WN;
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
    // stages: ceil(segment length / KS) per segment
    const int n_st = (c_first == c_last) ? (k1 - k0 + KS - 1) / KS
                                         : (KU - k0 + KS - 1) / KS + (c_last - c_first - 1) * ((KU + KS - 1) / KS) +
                                               (k1 + KS - 1) / KS;

    // Tile c: column group c / rg (16*NBW*WN columns), row group c % rg (TR rows).
    const uint32_t RG = (uint32_t)p.rg;
    auto cg_of = [&](int c) -> uint32_t { return RG == 1 ? (uint32_t)c : (uint32_t)c / RG; };
    auto row0_of = [&](int c) -> int { return RG == 1 ? 0 : (int)((uint32_t)c - cg_of(c) * RG) * TR; };
    auto rows_of = [&](int c) -> int {
        const int r = p.M - row0_of(c);
        return r < TR ? r : TR;
    };
    // this wave's first 16-column block; its NBW blocks lie in one 64-column
    // tile of the packed layout
    auto nbg_of = [&](int c) -> uint32_t { return (cg_of(c) * WN + (uint32_t)wn) * NBW; };
    auto w_tile = [&](int c) -> uint32_t {
        const uint32_t nbg = nbg_of(c);
        return ((nbg >> 2) * (uint32_t)KU * 4u + (nbg & 3u)) << 10;
    };
    auto s_tile = [&](int c) -> uint32_t {
        const uint32_t nbg = nbg_of(c);
        return (((nbg >> 2) * (uint32_t)p.G) << 7) + (nbg & 3u) * 8u;
    };

    // Per-lane address parts.
    const uint32_t w_lane = (uint32_t)lane * 16u;
    const uint32_t s_lane = (uint32_t)lg * 32u;
    uint32_t a_dma[kDmaB];  // this wave loads rows [wave*TR/4, (wave+1)*TR/4) of each block
#pragma unroll
    for (int i = 0; i < kDmaB; ++i) {
        const int r = wave * (TR / NW) + 4 * i + lg;
        a_dma[i] = (uint32_t)(r * p.K + (((lane & 15) ^ (r & 15)) * 8)) * 2u;
    }
    const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint8_t *)a_lds;
    // row wm*16*MBW + (lane & 15) (+ 16 mb via the offset field), chunk 4t + lg
    uint32_t a_rd[4];
#pragma unroll
    for (int t = 0; t < 4; ++t)
        a_rd[t] = lds0 + (uint32_t)((wm * 16 * MBW + (lane & 15)) * 256 + (((4 * t + lg) ^ (lane & 15)) << 4));
    // this wave's weights, this lane's 16 bytes (+ 1 KiB per column block)
    const uint32_t w_rd = lds0 + (uint32_t)(kAStage + wn * NBW * 1024 + lane * 16);
    const uint32_t w_bytes = (uint32_t)p.K * (uint32_t)(p.N / 2);
    const uint32_t s_bytes = (uint32_t)p.G * (uint32_t)p.N * 2u;

    ScaleFrag<NBW> sr[P][KS];

    // ---- load cursor: KS 128-row blocks per stage ----
    int ld_c = c_first, ld_ku = k0;
    int ld_end = (c_first == c_last) ? k1 : KU;
    uint32_t ld_w = w_tile(ld_c) + ((uint32_t)ld_ku << 12);
    uint32_t ld_s = s_tile(ld_c);
    const uint16_t *ld_a = p.A + (int64_t)row0_of(ld_c) * p.K;
    uint32_t a_bytes = (uint32_t)rows_of(ld_c) * (uint32_t)p.K * 2u;

    // LDS destinations of this wave's direct-to-LDS loads: slot 0's, and the
    // scratch area that takes the loads issued past the end.  The issue forms
    // each destination from these (through an opaque copy) so that the
    // compiler does not hold every slot's and block's address in a scalar
    // register across the loop.
    const uint32_t a_dst0 = lds0 + (uint32_t)(wave * (kABlock / NW));
    const uint32_t w_dst0 = lds0 + (uint32_t)(kAStage + (wn * NBW + wm * kWDma) * 1024);
    const uint32_t scratch = lds0 + (uint32_t)(P * kStage);

    auto issue = [&](int j) {
        const bool on = ld_ku < ld_end;  // the stage's first block is in range
        uint32_t a_base = a_dst0, w_base = w_dst0, x_base = scratch;
        asm volatile("" : "+s"(a_base), "+s"(w_base), "+s"(x_base));
        // Activation rows first (oldest loads of the stage), then this wave's
        // weights, then its scales.  Past the end the direct-to-LDS loads go
        // to the scratch area: other waves may still read every ring slot.
        // A block past the segment end loads through an empty buffer
        // descriptor (no memory is touched; zeros return, which add nothing).
#pragma unroll
        for (int kb = 0; kb < KS; ++kb) {
            const bool in = ld_ku + kb < ld_end;
            const __amdgpu_buffer_rsrc_t ra =
                __builtin_amdgcn_make_buffer_rsrc((void *)ld_a, (short)0, in ? a_bytes : 0u, kBufferFlags);
            const uint32_t dst = on ? a_base + (uint32_t)(j * kStage + kb * kABlock) : x_base;
#pragma unroll
            for (int i = 0; i < kDmaB; ++i)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (__attribute__((address_space(3))) void *)(uintptr_t)(dst + (uint32_t)(i * 1024)), 16, (int)a_dma[i],
                                                         (ld_ku + kb) * 256, 0, 0);
        }
#pragma unroll
        for (int kb = 0; kb < KS; ++kb) {
            const bool in = ld_ku + kb < ld_end;
            const __amdgpu_buffer_rsrc_t rw =
                __builtin_amdgcn_make_buffer_rsrc((void *)p.W, (short)0, in ? w_bytes : 0u, kBufferFlags);
            // this wave's share of its column group's blocks: wm*kWDma ..
            const uint32_t wdst = on ? w_base + (uint32_t)(j * kStage + kb * kWBlock) : x_base + kDmaB * 1024u;
#pragma unroll
            for (int b = 0; b < kWDma; ++b)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(rw, (__attribute__((address_space(3))) void *)(uintptr_t)(wdst + (uint32_t)(b * 1024)), 16,
                                                         (int)(w_lane + (wm * kWDma + b) * 1024),
                                                         (int)(ld_w + kb * 4096u), 0, kAuxNonTemporal);
        }
        issue_order_point();  // the direct-to-LDS loads precede the stage's scale loads
#pragma unroll
        for (int kb = 0; kb < (PER_CHANNEL ? 1 : KS); ++kb) {
            const bool in = ld_ku + kb < ld_end;
            const __amdgpu_buffer_rsrc_t rs =
                __builtin_amdgcn_make_buffer_rsrc((void *)p.S, (short)0, in ? s_bytes : 0u, kBufferFlags);
            const uint32_t soff = PER_CHANNEL ? ld_s : ld_s + ((uint32_t)scale_row_of(ld_ku + kb, p) << 7);
            if constexpr (NBW == 1) {
                sr[j][kb].v =
                    __builtin_bit_cast(half4_t, __builtin_amdgcn_raw_buffer_load_b64(rs, s_lane, soff, 0));
            } else {
#pragma unroll
                for (int i = 0; i < NBW / 2; ++i)
                    sr[j][kb].v[i] = __builtin_bit_cast(
                        half8_t, __builtin_amdgcn_raw_buffer_load_b128(rs, s_lane + i * 16, soff, 0));
            }
        }
        issue_order_point();  // stages do not interleave
    };
    auto advance_ld = [&]() {
        ld_ku += KS;
        ld_w += KS * 4096u;
        if (ld_ku >= ld_end) {  // next tile (rare)
            ld_c += 1;
            ld_ku = 0;
            ld_end = (ld_c < c_last) ? KU : (ld_c == c_last) ? k1 : 0;  // 0: past the range
            ld_w = w_tile(ld_c);
            ld_s = s_tile(ld_c);
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

    float4_t acc[NBW][MBW];  // [column block][row block]
    const float4_t zero4 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int b = 0; b < NBW; ++b)
#pragma unroll
        for (int mb = 0; mb < MBW; ++mb) acc[b][mb] = zero4;

    // One stage (ring slot j): every operand of the KS blocks is read first,
    // then per block the column blocks, each dequantized word feeding the MBW
    // row blocks.
    // LDS reads of one stage, in the order the MFMAs use them: per block,
    // column block 0's weights, the activation operands k-step by k-step,
    // then the other column blocks' weights.  LDS reads complete in order, so
    // each group of MFMAs waits only for the reads it needs (by counting the
    // reads issued after them) and the rest of the stage's reads overlap the
    // first column block's MFMAs.  Each wait "redefines" the registers it
    // makes available, so that no use is scheduled before it.
    constexpr int kRB = NBW + 4 * MBW;  // reads per block
    constexpr int kR = KS * kRB;        // reads per stage
    auto reads_after = [](int idx) { return kR - 1 - idx; };
    auto compute = [&](int j) {
        u32x4_t wv[KS][NBW];     // [block][column block] this lane's packed weights
        u32x4_t v[KS][MBW][4];   // [block][row block][k-step] activation operands
#pragma unroll
        for (int kb = 0; kb < KS; ++kb) {
            const uint32_t wj = w_rd + j * kStage + kb * kWBlock;
            asm volatile("ds_read_b128 %0, %1" : "=v"(wv[kb][0]) : "v"(wj));
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                const uint32_t aj = a_rd[t] + j * kStage + kb * kABlock;
#pragma unroll
                for (int mb = 0; mb < MBW; ++mb)
                    asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(v[kb][mb][t]) : "v"(aj), "i"(mb * 4096));
            }
#pragma unroll
            for (int b = 1; b < NBW; ++b)
                asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(wv[kb][b]) : "v"(wj), "i"(b * 1024));
        }
#pragma unroll
        for (int kb = 0; kb < KS; ++kb) {
#pragma unroll
            for (int b = 0; b < NBW; ++b) {
                if (b > 0) {
                    wait_lgkmcnt_n(reads_after(kb * kRB + 4 * MBW + b));
                    asm volatile("" : "+v"(wv[kb][b]));
                }
                // k-step t of column block 0 waits for the step's activation
                // operands (and, at t = 0, the block's first weights)
                auto ready_step = [&](int t) {
                    if (b == 0) {
                        wait_lgkmcnt_n(reads_after(kb * kRB + t * MBW + MBW));
                        if (t == 0) asm volatile("" : "+v"(wv[kb][0]));
#pragma unroll
                        for (int mb = 0; mb < MBW; ++mb) asm volatile("" : "+v"(v[kb][mb][t]));
                    }
                };
                if constexpr (PER_CHANNEL) {
#pragma unroll
                    for (int t = 0; t < 4; ++t) {
                        ready_step(t);
                        const half8_t w = dequant_magic(wv[kb][b][t], dq);
#pragma unroll
                        for (int mb = 0; mb < MBW; ++mb)
                            acc[b][mb] = mfma(w, __builtin_bit_cast(half8_t, v[kb][mb][t]), acc[b][mb]);
                    }
                } else {
                    float4_t tmp[MBW];
#pragma unroll
                    for (int t = 0; t < 4; ++t) {
                        ready_step(t);
                        const half8_t w = dequant_magic(wv[kb][b][t], dq);
#pragma unroll
                        for (int mb = 0; mb < MBW; ++mb)
                            tmp[mb] = mfma(w, __builtin_bit_cast(half8_t, v[kb][mb][t]), t == 0 ? zero4 : tmp[mb]);
                    }
#pragma unroll
                    for (int mb = 0; mb < MBW; ++mb)
#pragma unroll
                        for (int i = 0; i < 4; ++i)
                            acc[b][mb][i] = __builtin_fmaf(tmp[mb][i], (float)sr[j][kb].at(b * 4 + i), acc[b][mb][i]);
                }
            }
        }
    };

    // block j of this wave = column block j / MBW, row block j % MBW; slot index wave*kBlocks + j
    auto own = [&](int j) { return wave * kBlocks + j; };
    // Tile c's C from full sums (per-channel scales from cs).
    auto store_c_scaled = [&](int c, const float4_t *out, const ScaleFrag<NBW> &cs) {
        const int r0 = row0_of(c) + wm * 16 * MBW, rows = rows_of(c) - wm * 16 * MBW;
        const uint32_t col0 = nbg_of(c) * 16u;
#pragma unroll
        for (int j = 0; j < kBlocks; ++j) {
            const int b = j / MBW, mb = j % MBW;
            const int m = mb * 16 + (lane & 15);
            if (m < rows) {
                float4_t vv = out[j];
                if constexpr (PER_CHANNEL) {
#pragma unroll
                    for (int i = 0; i < 4; ++i) vv[i] *= (float)cs.at(b * 4 + i);
                }
                const half4_t h = {(_Float16)vv[0], (_Float16)vv[1], (_Float16)vv[2], (_Float16)vv[3]};
                *(half4_t *)(p.C + (int64_t)(r0 + m) * p.N + col0 + b * 16 + lg * 4) = h;
            }
        }
    };

    const int slot_floats = NW * kBlocks * 256;
    float *const my_slots = p.partials + (int64_t)wg * 2 * slot_floats;  // slot 0; slot 1 follows
    bool has_first = false, has_last = false;

    int cp_c = c_first, cp_ku = k0, cp_begin = k0;
    int cp_end = (c_first == c_last) ? k1 : KU;
    // A segment is complete: write C (whole tile) or slot 0 (shared first
    // tile).  A shared last tile stays in acc: it is the range's final
    // segment, combined after the loop.  Per-channel scales of the tile came
    // with the stage's first block.
    auto finish_segment = [&](int j_stage) {
        const bool partial = cp_begin != 0 || cp_end != KU;
        if (partial && cp_c == c_last) {
            has_last = true;
            return;
        }
        float4_t out[kBlocks];
#pragma unroll
        for (int j = 0; j < kBlocks; ++j) {
            out[j] = acc[j / MBW][j % MBW];
            acc[j / MBW][j % MBW] = zero4;
        }
        if (partial) {
            has_first = true;
#pragma unroll
            for (int j = 0; j < kBlocks; ++j) store_partial(my_slots, own(j), lane, out[j]);
        } else {
            store_c_scaled(cp_c, out, sr[j_stage][0]);
        }
    };

    // Stage st: wait for this wave's direct-to-LDS loads of the stage (loads
    // issued after them: the stage's scales and the P - 2 stages issued later;
    // vector-memory operations complete in order), meet at the barrier (now
    // the whole stage is in LDS, and every wave is done with the slot of stage
    // st - 1), refill that slot with stage st + P - 1, compute.  Loads are
    // issued unconditionally (past the range into the scratch area, through
    // empty descriptors) so that every stage has the same load pattern and the
    // compiler's own vmcnt waits (for the scale registers) stay static.
    // Stage st (ring slot j) with `later` stages issued after it; `refill`:
    // the slot of stage st - 1 takes stage st + P - 1.
    auto step = [&](int j, int st, int later, bool refill) {
        const bool live = st < n_st;
        if (live) {
            wait_vmcnt_n(kSL + later * kLoads);
            __builtin_amdgcn_s_barrier();
            asm volatile("" ::: "memory");
        }
        if (refill) {
            issue((j + P - 1) % P);
            advance_ld();
        }
        if (live) {
            compute(j);
            if (cp_ku + KS >= cp_end) {
                finish_segment(j);
                cp_c += 1;
                cp_ku = 0;
                cp_begin = 0;
                cp_end = (cp_c < c_last) ? KU : k1;
            } else {
                cp_ku += KS;
            }
        }
    };
    // Groups of P stages.  In the last group only the first step has a stage
    // left to load (the group's last); the others issue nothing, and stage j
    // of the group waits with the P - 1 - j stages issued after it behind it.
    const int st_last = (n_st - 1) / P * P;
    for (int st0 = 0; st0 < st_last; st0 += P) {
#pragma unroll
        for (int j = 0; j < P; ++j) step(j, st0 + j, P - 2, true);
    }
#pragma unroll
    for (int j = 0; j < P; ++j) step(j, st_last + j, j == 0 ? P - 2 : P - 1 - j, j == 0);

    float4_t last_out[kBlocks];
#pragma unroll
    for (int j = 0; j < kBlocks; ++j) last_out[j] = acc[j / MBW][j % MBW];
    auto own_slot = [&](int j) { return own(j); };
    // After the loop nothing is in flight to wait behind: load the column
    // scales directly.
    auto store_c = [&](int c, const float4_t *out) {
        ScaleFrag<NBW> cs{};
        if constexpr (PER_CHANNEL) {
            const _Float16 *src = (const _Float16 *)p.S + (int64_t)(nbg_of(c) >> 2) * 64 + lg * 16 + (nbg_of(c) & 3u) * 4;
            if constexpr (NBW == 1) {
                cs.v = *(const half4_t *)src;
            } else {
#pragma unroll
                for (int i = 0; i < NBW / 2; ++i) cs.v[i] = *(const half8_t *)(src + 8 * i);
            }
        }
        store_c_scaled(c, out, cs);
    };
    combine_tiles<kBlocks>(p, flags, wg, grid, slot_floats, lane, has_first, c_first, has_last, c_last, last_out,
                           own_slot, store_c);
}

}  // namespace

template <int WN, int WM, int MBW, int NBW, int KS>
hipError_t launch_tile(const GemmConfig &cfg, const GemmProblem &p, hipStream_t stream)
{
    GemmProblem arg = p;
    void *args[] = {&arg};
    const void *fn = (p.group_units == 0) ? (const void *)&w4a16_tile_kernel<WN, WM, MBW, NBW, KS, true>
                                          : (const void *)&w4a16_tile_kernel<WN, WM, MBW, NBW, KS, false>;
    return hipLaunchKernel(fn, dim3(cfg.grid), dim3(64 * WN * WM), args, 0, stream);
}

// Instantiated shapes (waves along M, row blocks per wave, column blocks per
// wave, 128-row blocks per stage): 64 x 64 per wave for large batches; for
// up to 32 rows, 16 or 32 rows per wave over 2 or 4 blocks per stage.  One
// case per entry of kTileConfigs (plan.h), which the planner chooses from.
hipError_t launch_tile_gemm(const GemmConfig &cfg, const GemmProblem &p, hipStream_t stream)
{
    switch (cfg.tile_nw * 10000 + cfg.tile_wm * 1000 + cfg.mb * 100 + cfg.nb * 10 + cfg.tile_ks) {
    case 41441: return launch_tile<4, 1, 4, 4, 1>(cfg, p, stream);
    case 42441: return launch_tile<2, 2, 4, 4, 1>(cfg, p, stream);
    case 82441: return launch_tile<4, 2, 4, 4, 1>(cfg, p, stream);
    case 82241: return launch_tile<4, 2, 2, 4, 1>(cfg, p, stream);
    case 41142: return launch_tile<4, 1, 1, 4, 2>(cfg, p, stream);
    case 41124: return launch_tile<4, 1, 1, 2, 4>(cfg, p, stream);
    case 41222: return launch_tile<4, 1, 2, 2, 2>(cfg, p, stream);
    case 41214: return launch_tile<4, 1, 2, 1, 4>(cfg, p, stream);
    default: return hipErrorInvalidValue;
    }
}

void tile_kernel_name(const GemmConfig &cfg, bool per_channel, char *buf, size_t n)
{
    snprintf(buf, n, "w4a16_tile_kernel<%d, %d, %d, %d, %d, %s>", cfg.tile_nw / cfg.tile_wm, cfg.tile_wm, cfg.mb,
             cfg.nb, cfg.tile_ks, per_channel ? "true" : "false");
}

}  // namespace marlin
