// W4A16 GEMM for gfx950: C[M,N] = A[M,K] * (s * (q - 8)), fp32 accumulation.
//
// Design (the paper's Section 3.4 ideas, re-derived for CDNA4):
//  * Transposed product, as the paper does for its sparse kernel (Section 4):
//    each v_mfma_f32_16x16x32_f16 multiplies a 16(n) x 32(k) block of W^T
//    (first operand) by a 32(k) x 16(m) block of A^T.  A lane's first operand
//    is 8 consecutive k of one column n: exactly one packed 32-bit word of
//    codes, so one 16-byte load feeds four MFMA steps ("Maximizing Loading
//    Bandwidth", "Dequantization and Tensor Cores").
//  * Weights and activations reach LDS through gfx950's direct-to-LDS loads
//    (global_load_lds_dwordx4), the CDNA counterpart of cp.async, with the
//    non-temporal bit on the weight stream (the paper's evict_first).  P stages
//    are in flight; the kernel waits on vmcnt per stage with static counts
//    ("Memory Load Pipelining").
//  * int4 -> fp16 by bit operations: mask the code into the low mantissa bits
//    of the fp16 number 1024 (0x6400) and subtract 1032 exactly; codes in the
//    next nibble become 1024 + 16q and are fixed by one fma (x/16 - 72).  Two
//    codes per 32-bit register at a time ("Dequantization and Tensor Cores").
//  * Group scales multiply each 128-row fp32 partial product (one group or
//    part of one); per-channel scales multiply the final sum once
//    ("Groups and Instruction Ordering").
//  * Waves of a work-group split N (sharing the activation tile in LDS) or K
//    (each with its own tile, reduced in LDS at the end: Algorithm 1's layout).
//  * Stream-K style striped partitioning over a persistent grid: work-group w
//    owns the contiguous range [w*T/grid, (w+1)*T/grid) of (column tile,
//    128-row block) units, column-major, wrapping into the next column
//    ("Striped Partitioning").  Columns split across work-groups are combined
//    through fp32 partial slots in the workspace; the last work-group to
//    arrive (an agent-scope acq_rel counter) sums the slots in a fixed order
//    and writes C, then resets the counter.  No work-group ever waits on
//    another, so no co-residency is assumed.
#include <hip/hip_runtime.h>

#include "internal.h"

namespace marlin {
namespace {

typedef _Float16 half2_t __attribute__((ext_vector_type(2)));
typedef _Float16 half4_t __attribute__((ext_vector_type(4)));
typedef _Float16 half8_t __attribute__((ext_vector_type(8)));
typedef float float4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

#define LDS_PTR(p) ((__attribute__((address_space(3))) void *)(p))

constexpr int kLdsBytes = 160 * 1024;
constexpr int kAuxNonTemporal = 2;  // cache-policy bit: non-temporal (streamed once)
// Word 3 of a gfx9 buffer descriptor for raw (untyped) dword access.
constexpr int kBufferFlags = 0x00020000;

// s_waitcnt immediate for gfx9: vmcnt[3:0] | expcnt[6:4] | lgkmcnt[11:8] | vmcnt[5:4]<<14.
template <int V>
__device__ __forceinline__ void wait_vmcnt()
{
    static_assert(V >= 0 && V < 64, "vmcnt out of range");
    __builtin_amdgcn_s_waitcnt((V & 15) | (7 << 4) | (15 << 8) | ((V >> 4) << 14));
    asm volatile("" ::: "memory");
}

__device__ __forceinline__ void wait_lgkmcnt0()
{
    __builtin_amdgcn_s_waitcnt(63 | (7 << 4) | (0 << 8) | (3 << 14));
    asm volatile("" ::: "memory");
}

// Work-group barrier that does not wait for outstanding global loads.
__device__ __forceinline__ void lds_barrier()
{
    wait_lgkmcnt0();
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

__device__ __forceinline__ half2_t as_h2(uint32_t x) { return __builtin_bit_cast(half2_t, x); }

// Masks of the int4 -> fp16 conversion.  They are made opaque once per
// kernel (an empty asm that "redefines" them in vector registers) so that
// (x & m) | o selects the single v_and_or_b32 with register operands instead
// of an and/or pair with literal constants.
struct DequantConsts {
    uint32_t lo, hi, ex;
};

__device__ __forceinline__ DequantConsts dequant_consts()
{
    DequantConsts k{0x000F000Fu, 0x00F000F0u, 0x64006400u};
    asm volatile("" : "+v"(k.lo), "+v"(k.hi), "+v"(k.ex));
    return k;
}

// Eight codes of one packed word -> the eight fp16 values q - 8 in element
// order j = 0..7 (code j sits in nibble (j >> 1) + 4 (j & 1)).  Low nibbles
// of each 16-bit half land in the low mantissa bits of 1024.0 (0x6400):
// 1024 + q, minus 1032 gives q - 8 exactly.  The next nibble lands 4 bits
// higher: 1024 + 16q, and (1024 + 16q) / 16 - 72 = q - 8 in one fma.  A shift
// by 8 brings the other two nibbles of each half into the same positions.
__device__ __forceinline__ half8_t dequant8(uint32_t x, const DequantConsts &k)
{
    const half2_t sub = {(_Float16)1032.0f, (_Float16)1032.0f};
    const half2_t mul = {(_Float16)0.0625f, (_Float16)0.0625f};
    const half2_t add = {(_Float16)-72.0f, (_Float16)-72.0f};
    const uint32_t y = x >> 8;
    const half2_t r0 = as_h2((x & k.lo) | k.ex) - sub;
    const half2_t r1 = __builtin_elementwise_fma(as_h2((x & k.hi) | k.ex), mul, add);
    const half2_t r2 = as_h2((y & k.lo) | k.ex) - sub;
    const half2_t r3 = __builtin_elementwise_fma(as_h2((y & k.hi) | k.ex), mul, add);
    return half8_t{r0.x, r0.y, r1.x, r1.y, r2.x, r2.y, r3.x, r3.y};
}

// Multiply eight fp16 weights by one fp16 scale (four packed multiplies).
__device__ __forceinline__ half8_t scale8(half8_t b, half2_t s)
{
    half2_t r0 = half2_t{b[0], b[1]} * s, r1 = half2_t{b[2], b[3]} * s;
    half2_t r2 = half2_t{b[4], b[5]} * s, r3 = half2_t{b[6], b[7]} * s;
    return half8_t{r0.x, r0.y, r1.x, r1.y, r2.x, r2.y, r3.x, r3.y};
}

template <int MB, int NW, int KW, bool PER_CHANNEL>
struct Geo {
    static constexpr int kWaves = NW * KW;
    static constexpr int kThreads = 64 * kWaves;
    static constexpr int kAFrags = 4 * MB;                 // 1 KiB fragments per kw per stage
    static constexpr int kAFragsPerWave = kAFrags / NW;
    static constexpr int kABytes = KW * kAFrags * 1024;
    static constexpr int kWBytes = KW * NW * 4 * 1024;
    static constexpr int kSBytes = PER_CHANNEL ? 0 : KW * NW * 128;
    static constexpr int kStageBytes = kABytes + kWBytes + kSBytes;
    static constexpr int kBlocks = 4 * MB;                 // 16x16 output blocks per wave
    static constexpr int kOwnBlocks = kBlocks / KW;        // blocks a wave owns after reduction
    static constexpr int kRedBytes = (KW > 1) ? KW * NW * kBlocks * 1024 : 0;
    static constexpr int kFlagBytes = 64;
    static constexpr int kLoadsPerStage = 4 + kAFragsPerWave + (PER_CHANNEL ? 0 : 1);
    // Stages: as many as fit in LDS, at most 4, and few enough that the loads
    // issued after a stage stay within the 6-bit vmcnt counter.
    static constexpr int kStagesFit = (kLdsBytes - kRedBytes - kFlagBytes) / kStageBytes;
    static constexpr int kStagesCnt = 2 + 63 / kLoadsPerStage;
    static constexpr int P0 = kStagesFit < kStagesCnt ? kStagesFit : kStagesCnt;
    static constexpr int P = P0 > 4 ? 4 : P0;
    static constexpr int kSmemBytes = P * kStageBytes + kRedBytes + kFlagBytes;
    static constexpr int kSlotFloats = NW * kBlocks * 256;  // one partial tile, register layout
    // Group scales: fp32 fold of each 128-row product for small M (cheapest
    // in VALU there); fp16 scaling of the weights for larger M (no extra
    // accumulators).
    static constexpr bool kFold = !PER_CHANNEL && MB <= 2;
    static_assert(kAFrags % NW == 0, "A fragments must split evenly over N-waves");
    static_assert(kBlocks % KW == 0, "output blocks must split evenly over K-waves");
    static_assert(P >= 2, "at least two pipeline stages must fit in LDS");
    static_assert((P - 2) * kLoadsPerStage < 64, "vmcnt range");
};

// Position of a work-group in its range of units.  A stage covers up to KW
// consecutive 128-row blocks of one column tile.
struct Cursor {
    int c;          // column tile
    int ku;         // first 128-row block of the stage
    int ku_end;     // end of the segment (this work-group's part of column c)
    int seg_begin;  // first block of the segment
    int64_t u_end;  // end of the work-group's unit range
    bool done;
};

__device__ __forceinline__ void cursor_init(Cursor &cu, int64_t u0, int64_t u1, int KU)
{
    cu.u_end = u1;
    cu.done = (u0 >= u1);
    cu.c = (int)(u0 / KU);
    cu.ku = (int)(u0 - (int64_t)cu.c * KU);
    cu.seg_begin = cu.ku;
    const int64_t rem = u1 - (int64_t)cu.c * KU;
    cu.ku_end = rem < KU ? (int)rem : KU;
}

template <int KW>
__device__ __forceinline__ void cursor_next(Cursor &cu, int KU)
{
    cu.ku += KW;
    if (cu.ku >= cu.ku_end) {
        cu.c += 1;
        cu.ku = 0;
        cu.seg_begin = 0;
        const int64_t rem = cu.u_end - (int64_t)cu.c * KU;
        cu.done = rem <= 0;
        cu.ku_end = rem < KU ? (int)rem : KU;
    }
}

// Scale row of 128-row block ku: ku / group_units, by a shift when the group
// is a power-of-two number of blocks, else by a multiply with the rounded-up
// reciprocal 2^32 / group_units (exact for ku, group_units < 2^16).
__device__ __forceinline__ int scale_row_of(int ku, const GemmProblem &p)
{
    return p.gshift >= 0 ? (ku >> p.gshift) : (int)__umulhi((uint32_t)ku, p.gmagic);
}

__device__ __forceinline__ int64_t range_start(int w, int64_t total, int grid)
{
    return ((int64_t)w * total) / grid;
}

// Work-group that owns unit u: the largest w with range_start(w) <= u.
__device__ __forceinline__ int unit_owner(int64_t u, int64_t total, int grid)
{
    return (int)(((u + 1) * grid - 1) / total);
}

// ---- cross-work-group partial tiles ----
// A work-group that covers a column tile only in part writes its fp32 tile to
// one of its two workspace slots (0: its first column, 1: its last), in
// structure-of-arrays order so every store instruction covers 256 contiguous
// bytes: float index ((blk*4 + i)*64 + lane), blk = nw*kBlocks + b.  Those
// bytes are written and read with relaxed agent-scope atomics, which the
// compiler emits as ordinary vector stores / loads carrying the
// device-coherence bit, so they bypass the per-XCD L2 non-coherence without a
// whole-cache writeback or invalidate.  Ordering: each wave waits for its
// stores to complete (vmcnt 0) before the work-group barrier that precedes
// the arrival counter's atomic increment, and the last arriver issues its
// loads only after that increment has returned.
__device__ __forceinline__ void store_partial(float *slot, int blk, int lane, float4_t v)
{
    float *d = slot + blk * 256 + lane;
#pragma unroll
    for (int i = 0; i < 4; ++i) __hip_atomic_store(d + i * 64, v[i], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ float4_t load_partial(const float *slot, int blk, int lane)
{
    const float *s = slot + blk * 256 + lane;
    float4_t v;
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = __hip_atomic_load(s + i * 64, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return v;
}

// After the main loop: announce this work-group's partial columns (at most
// two); the work-group whose arrival completes a column's count sums the
// column's slots in work-group order (a fixed order: results are bitwise
// reproducible) and stores C.  `own(j)` gives the partial-tile block index of
// the j-th block this wave owns; `store_c(c, out)` writes C.
template <int KOWN, typename OwnFn, typename StoreFn>
__device__ __forceinline__ void publish_and_reduce(const GemmProblem &p, const int (&pcol)[2], int *flags,
                                                   int wg, int KU, int64_t total, int grid,
                                                   int slot_floats, int lane, OwnFn own, StoreFn store_c)
{
    if (pcol[0] < 0 && pcol[1] < 0) return;  // uniform across the work-group
    wait_vmcnt<0>();                          // this wave's partial stores are complete
    lds_barrier();
    if (threadIdx.x == 0) {
#pragma unroll
        for (int which = 0; which < 2; ++which) {
            int last = 0;
            const int c = pcol[which];
            if (c >= 0) {
                const int wf = unit_owner((int64_t)c * KU, total, grid);
                const int wl = unit_owner((int64_t)c * KU + KU - 1, total, grid);
                const uint32_t old = __hip_atomic_fetch_add(p.counters + c, 1u, __ATOMIC_RELAXED,
                                                            __HIP_MEMORY_SCOPE_AGENT);
                if (old == (uint32_t)(wl - wf)) {
                    last = 1;
                    __hip_atomic_store(p.counters + c, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                }
            }
            flags[which] = last;
        }
    }
    lds_barrier();
#pragma unroll
    for (int which = 0; which < 2; ++which) {
        const int c = pcol[which];
        if (c < 0 || !flags[which]) continue;
        const int wf = unit_owner((int64_t)c * KU, total, grid);
        const int wl = unit_owner((int64_t)c * KU + KU - 1, total, grid);
        float4_t out[KOWN];
        for (int w = wf; w <= wl; ++w) {
            const int wcol = (int)(range_start(w, total, grid) / KU);
            const float *slot = p.partials + ((int64_t)w * 2 + ((c == wcol) ? 0 : 1)) * slot_floats;
#pragma unroll
            for (int j = 0; j < KOWN; ++j) {
                const float4_t v = load_partial(slot, own(j), lane);
                out[j] = (w == wf) ? v : out[j] + v;
            }
        }
        store_c(c, out);
    }
    (void)wg;
}

// ---------------------------------------------------------------------------
// Kernel 1 (decode batches, M <= 32): register streaming.
//
// A work-group owns a column tile of 16*NB columns (NB 16-column blocks) over
// a range of 128-row blocks of K (the striped partition); its KW waves take
// consecutive 128-row blocks of each stage (waves split K), so no weight or
// activation byte is shared between waves: each lane loads exactly its MFMA
// operands (16-byte non-temporal buffer loads of the pre-shuffled weights,
// 16-byte loads of the activation rows, which hit L2) straight into a D-deep
// ring of registers.  The loop is unrolled over the ring so register slots
// are static and the compiler's vmcnt waits keep D-1 stages in flight.  Waves
// meet only at the end of a column segment, where their fp32 tiles are summed
// in LDS (Algorithm 1's reduction across waves that share an output tile).
// Narrow tiles (NB = 1) give enough whole columns to occupy every compute unit
// without splitting K across work-groups on small layers.
template <int MB, int NB, int KW, int D, int OCC, bool PER_CHANNEL>
__global__ void __launch_bounds__(64 * KW, OCC) w4a16_stream_kernel(GemmProblem p)
{
    constexpr int kBlocks = NB * MB;               // 16x16 output blocks per wave
    constexpr int kOwn = (kBlocks + KW - 1) / KW;  // blocks a wave owns after the LDS reduction
    constexpr int kSLoads = (NB + 1) / 2;          // 16-byte scale loads per stage
    __shared__ float4_t red[KW * kBlocks * 64];
    __shared__ int flags[2];

    const int lane = threadIdx.x & 63;
    const DequantConsts dq = dequant_consts();
    // wave index as a scalar: all cursor and address arithmetic below is uniform
    const int kw = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int lg = lane >> 4;
    const int KU = p.K >> 7;
    const int cols = p.N / (16 * NB);
    const int total = cols * KU;  // < 2^31 (host checks K * N)
    const int grid = gridDim.x;
    const int wg = blockIdx.x;
    const int u0 = (int)range_start(wg, total, grid);
    const int u1 = (int)range_start(wg + 1, total, grid);
    const int first_col = u0 / KU;

    // Stages of this work-group: each segment (its part of one column) takes
    // ceil(length / KW) stages.
    int n_st = 0;
    for (int u = u0; u < u1;) {
        const int e = (u / KU + 1) * KU < u1 ? (u / KU + 1) * KU : u1;
        n_st += (e - u + KW - 1) / KW;
        u = e;
    }

    // Stage cursors (wave-uniform): column tile c, first 128-row block ku of
    // the stage, segment [begin, end) within the column.
    struct Cur {
        int c, ku, begin, end;
    };
    auto cur_init = [&](Cur &q) {
        q.c = first_col;
        q.ku = u0 - q.c * KU;
        q.begin = q.ku;
        q.end = (u1 - q.c * KU) < KU ? (u1 - q.c * KU) : KU;
    };
    auto cur_next = [&](Cur &q) {
        q.ku += KW;
        if (q.ku >= q.end) {
            q.c += 1;
            q.ku = 0;
            q.begin = 0;
            q.end = (u1 - q.c * KU) < KU ? (u1 - q.c * KU) : KU;
        }
    };
    Cur ld, cp;
    cur_init(ld);
    cp = ld;

    // Loads are buffer loads: a fixed per-lane byte offset in one VGPR, the
    // per-stage offset in a scalar register, so the stream costs no vector
    // address arithmetic.  Past the end of the range a stage uses an empty
    // descriptor: its loads are out of range, touch no memory and return 0,
    // which keeps the pattern of loads per stage static.  Activation rows are
    // loaded only by lanes whose row exists (the other lanes' MFMA columns are
    // never stored).
    const uint32_t w_lane = lane * 16;
    const int arow = lane & 15;
    uint32_t a_lane[MB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) a_lane[mb] = (uint32_t)((mb * 16 + arow) * p.K + 8 * lg) * 2;
    const uint32_t s_lane = lg * 32;
    const int w_bytes = (int)((uint32_t)p.K * (uint32_t)(p.N / 2));
    const int a_bytes = p.M * p.K * 2;
    const int s_bytes = p.G * p.N * 2;

    u32x4_t wr[D][NB];
    half8_t ar[D][4 * MB];
    half8_t sr[D][kSLoads];
#pragma unroll
    for (int j = 0; j < D; ++j)
#pragma unroll
        for (int i = 0; i < 4 * MB; ++i) ar[j][i] = half8_t{};

    auto issue = [&](int j, const Cur &cu, bool valid) {
        int ku = cu.ku + kw;
        ku = ku < cu.end ? ku : cu.ku;  // idle wave: any valid block, result unused
        const int nbg = cu.c * NB;      // first global 16-column block of the tile
        const __amdgpu_buffer_rsrc_t rw =
            __builtin_amdgcn_make_buffer_rsrc((void *)p.W, (short)0, valid ? w_bytes : 0, kBufferFlags);
        const int w_off = (((nbg >> 2) * KU + ku) * 4 + (nbg & 3)) << 10;
#pragma unroll
        for (int b = 0; b < NB; ++b)
            wr[j][b] = __builtin_bit_cast(
                u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rw, w_lane + b * 1024, w_off, kAuxNonTemporal));
        const __amdgpu_buffer_rsrc_t ra =
            __builtin_amdgcn_make_buffer_rsrc((void *)p.A, (short)0, valid ? a_bytes : 0, kBufferFlags);
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
            if (mb * 16 + arow < p.M) {
#pragma unroll
                for (int t = 0; t < 4; ++t)
                    ar[j][mb * 4 + t] = __builtin_bit_cast(
                        half8_t, __builtin_amdgcn_raw_buffer_load_b128(ra, a_lane[mb] + t * 64, ku << 8, 0));
            }
        }
        if constexpr (!PER_CHANNEL) {
            const __amdgpu_buffer_rsrc_t rs =
                __builtin_amdgcn_make_buffer_rsrc((void *)p.S, (short)0, valid ? s_bytes : 0, kBufferFlags);
            const int s_off = (((nbg >> 2) * p.G + scale_row_of(ku, p)) << 7) + (nbg & 3) * 8;
#pragma unroll
            for (int i = 0; i < kSLoads; ++i)
                sr[j][i] = __builtin_bit_cast(
                    half8_t, __builtin_amdgcn_raw_buffer_load_b128(rs, s_lane + i * 16, s_off, 0));
        }
    };

    float4_t acc[NB][MB];
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) acc[b][mb] = float4_t{0.f, 0.f, 0.f, 0.f};

    // MFMA order: k-step outer, column block inner, so consecutive MFMAs are
    // independent; group scales fold in after the stage's last MFMA.
    auto compute = [&](int j) {
        if constexpr (!PER_CHANNEL) {
            float4_t tmp[NB][MB];
#pragma unroll
            for (int t = 0; t < 4; ++t)
#pragma unroll
                for (int b = 0; b < NB; ++b) {
                    const half8_t w = dequant8(wr[j][b][t], dq);
#pragma unroll
                    for (int mb = 0; mb < MB; ++mb)
                        tmp[b][mb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(
                            w, ar[j][mb * 4 + t], t == 0 ? float4_t{0.f, 0.f, 0.f, 0.f} : tmp[b][mb], 0, 0, 0);
                }
#pragma unroll
            for (int b = 0; b < NB; ++b) {
                // scales of block b: halves 4b .. 4b+3 of this lane's run
                const half8_t sv = sr[j][b >> 1];
#pragma unroll
                for (int mb = 0; mb < MB; ++mb)
#pragma unroll
                    for (int i = 0; i < 4; ++i) acc[b][mb][i] += tmp[b][mb][i] * (float)sv[(b & 1) * 4 + i];
            }
        } else {
#pragma unroll
            for (int t = 0; t < 4; ++t)
#pragma unroll
                for (int b = 0; b < NB; ++b) {
                    const half8_t w = dequant8(wr[j][b][t], dq);
#pragma unroll
                    for (int mb = 0; mb < MB; ++mb)
                        acc[b][mb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(w, ar[j][mb * 4 + t], acc[b][mb], 0, 0, 0);
                }
        }
    };

    // block index blk = b*MB + mb; wave kw owns blk = kw + j*KW (< kBlocks)
    auto own = [&](int j) { return kw + j * KW; };
    auto store_c = [&](int c, const float4_t *out) {
#pragma unroll
        for (int j = 0; j < kOwn; ++j) {
            const int blk = kw + j * KW;
            if (blk >= kBlocks) break;
            const int b = blk / MB, mb = blk % MB;
            const int m = mb * 16 + arow;
            if (m < p.M) {
                const int nbg = c * NB + b;
                float4_t v = out[j];
                if constexpr (PER_CHANNEL) {
                    const half4_t s4 = *(const half4_t *)(p.S + (int64_t)(nbg >> 2) * 64 + lg * 16 + (nbg & 3) * 4);
#pragma unroll
                    for (int i = 0; i < 4; ++i) v[i] *= (float)s4[i];
                }
                const half4_t h = {(_Float16)v[0], (_Float16)v[1], (_Float16)v[2], (_Float16)v[3]};
                *(half4_t *)(p.C + (int64_t)m * p.N + nbg * 16 + lg * 4) = h;
            }
        }
    };

    int pcol[2] = {-1, -1};
    const int slot_floats = kBlocks * 256;
    auto finish_segment = [&](const Cur &cu) {
        float4_t out[kOwn];
        if constexpr (KW > 1) {
#pragma unroll
            for (int b = 0; b < NB; ++b)
#pragma unroll
                for (int mb = 0; mb < MB; ++mb) red[(kw * kBlocks + b * MB + mb) * 64 + lane] = acc[b][mb];
            lds_barrier();
#pragma unroll
            for (int j = 0; j < kOwn; ++j) {
                const int blk = own(j);
                if (blk < kBlocks) {
                    float4_t s = red[blk * 64 + lane];
#pragma unroll
                    for (int k2 = 1; k2 < KW; ++k2) s += red[(k2 * kBlocks + blk) * 64 + lane];
                    out[j] = s;
                }
            }
            lds_barrier();
        } else {
#pragma unroll
            for (int j = 0; j < kOwn; ++j) out[j] = acc[j / MB][j % MB];
        }
#pragma unroll
        for (int b = 0; b < NB; ++b)
#pragma unroll
            for (int mb = 0; mb < MB; ++mb) acc[b][mb] = float4_t{0.f, 0.f, 0.f, 0.f};
        if (cu.begin == 0 && cu.end == KU) {
            store_c(cu.c, out);
        } else {
            const int which = (cu.c == first_col) ? 0 : 1;
            pcol[which] = cu.c;
            float *slot = p.partials + ((int64_t)wg * 2 + which) * slot_floats;
#pragma unroll
            for (int j = 0; j < kOwn; ++j)
                if (own(j) < kBlocks) store_partial(slot, own(j), lane, out[j]);
        }
    };

#pragma unroll
    for (int j = 0; j < D; ++j) {
        issue(j, ld, j < n_st);
        cur_next(ld);
    }
    const int iters = (n_st + D - 1) / D;
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int j = 0; j < D; ++j) {
            const int st = it * D + j;
            if (st < n_st) {
                if (cp.ku + kw < cp.end) compute(j);
                if (cp.ku + KW >= cp.end) finish_segment(cp);
                cur_next(cp);
            }
            issue(j, ld, st + D < n_st);
            cur_next(ld);
        }
    }
    auto own_valid = [&](int j) { return own(j) < kBlocks ? own(j) : 0; };
    publish_and_reduce<kOwn>(p, pcol, flags, wg, KU, (int64_t)total, grid, slot_floats, lane, own_valid,
                             store_c);
}

// ---------------------------------------------------------------------------
// Kernel 2 (larger batches, M > 32): LDS pipeline.
template <int MB, int NW, int KW, bool PER_CHANNEL>
__global__ void __launch_bounds__(64 * NW * KW, 1)
    w4a16_lds_kernel(GemmProblem p)
{
    using Gm = Geo<MB, NW, KW, PER_CHANNEL>;
    constexpr int P = Gm::P;
    constexpr int L = Gm::kLoadsPerStage;
    __shared__ __attribute__((aligned(1024))) uint8_t smem[Gm::kSmemBytes];

    const int lane = threadIdx.x & 63;
    const DequantConsts dq = dequant_consts();
    const int wave = threadIdx.x >> 6;
    const int nw = (NW == 1) ? 0 : wave % NW;
    const int kw = (KW == 1) ? 0 : wave / NW;
    const int lg = lane >> 4;

    const int KU = p.K >> 7;
    const int cols = p.N / (64 * NW);
    const int64_t total = (int64_t)cols * KU;
    const int grid = gridDim.x;
    const int wg = blockIdx.x;
    const int64_t u0 = range_start(wg, total, grid);
    const int64_t u1 = range_start(wg + 1, total, grid);
    const int first_col = (int)(u0 / KU);

    Cursor ld, cp;
    cursor_init(ld, u0, u1, KU);
    cp = ld;

    uint8_t *const red = smem + P * Gm::kStageBytes;
    int *const flags = (int *)(smem + P * Gm::kStageBytes + Gm::kRedBytes);

    // ---- stage loader: every wave issues exactly L loads per stage ----
    auto issue = [&](const Cursor &cu, int slot) {
        int ku = cu.ku + kw;
        if (ku >= cu.ku_end) ku = cu.ku;  // idle wave: reload a valid block, result unused
        uint8_t *base = smem + slot * Gm::kStageBytes;
        const int c64 = cu.c * NW + nw;
        const uint32_t *wsrc = p.W + ((int64_t)(c64 * KU + ku) * 4) * 256 + lane * 4;
        uint8_t *wdst = base + Gm::kABytes + (kw * NW + nw) * 4096;
#pragma unroll
        for (int nb = 0; nb < 4; ++nb)
            __builtin_amdgcn_global_load_lds((const void *)(wsrc + nb * 256), LDS_PTR(wdst + nb * 1024),
                                             16, 0, kAuxNonTemporal);
#pragma unroll
        for (int i = 0; i < Gm::kAFragsPerWave; ++i) {
            const int f = nw + i * NW;
            const int mb = f >> 2, t = f & 3;
            int row = mb * 16 + (lane & 15);
            row = row < p.M ? row : p.M - 1;
            const uint16_t *asrc = p.A + (int64_t)row * p.K + ku * 128 + 32 * t + 8 * lg;
            __builtin_amdgcn_global_load_lds((const void *)asrc,
                                             LDS_PTR(base + (kw * Gm::kAFrags + f) * 1024), 16, 0, 0);
        }
        if constexpr (!PER_CHANNEL) {
            const int r = scale_row_of(ku, p);
            const uint16_t *ssrc = p.S + ((int64_t)c64 * p.G + r) * 64 + (lane & 31) * 2;
            if (lane < 32)
                __builtin_amdgcn_global_load_lds((const void *)ssrc,
                                                 LDS_PTR(base + Gm::kABytes + Gm::kWBytes + (kw * NW + nw) * 128),
                                                 4, 0, 0);
        }
    };

    float4_t acc[4][MB];
#pragma unroll
    for (int nb = 0; nb < 4; ++nb)
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) acc[nb][mb] = float4_t{0.f, 0.f, 0.f, 0.f};

    // Partial segments of this work-group: head (its first column) and tail.
    int pcol[2] = {-1, -1};

    // ---- output helpers (register layout: block b = nb*MB + mb; lane holds
    //      rows n = 16nb + 4lg + i, column m = 16mb + lane%16) ----
    auto store_c = [&](int c, const float4_t *out) {
        const int c64 = c * NW + nw;
#pragma unroll
        for (int j = 0; j < Gm::kOwnBlocks; ++j) {
            const int b = kw + j * KW;
            const int nb = b / MB, mb = b % MB;
            const int m = mb * 16 + (lane & 15);
            if (m < p.M) {
                float4_t v = out[j];
                if constexpr (PER_CHANNEL) {
                    const half4_t s4 = *(const half4_t *)(p.S + (int64_t)c64 * 64 + lg * 16 + nb * 4);
#pragma unroll
                    for (int i = 0; i < 4; ++i) v[i] *= (float)s4[i];
                }
                const half4_t h = {(_Float16)v[0], (_Float16)v[1], (_Float16)v[2], (_Float16)v[3]};
                const int n = c64 * 64 + nb * 16 + lg * 4;
                *(half4_t *)(p.C + (int64_t)m * p.N + n) = h;
            }
        }
    };

    // ---- segment end: reduce over K-waves, then write C or a partial slot ----
    auto finish_segment = [&](const Cursor &cu) {
        float4_t out[Gm::kOwnBlocks];
        if constexpr (KW > 1) {
            float4_t *r = (float4_t *)red;
#pragma unroll
            for (int nb = 0; nb < 4; ++nb)
#pragma unroll
                for (int mb = 0; mb < MB; ++mb)
                    r[((kw * NW + nw) * Gm::kBlocks + nb * MB + mb) * 64 + lane] = acc[nb][mb];
            lds_barrier();
#pragma unroll
            for (int j = 0; j < Gm::kOwnBlocks; ++j) {
                const int b = kw + j * KW;
                float4_t s = r[((0 * NW + nw) * Gm::kBlocks + b) * 64 + lane];
#pragma unroll
                for (int k2 = 1; k2 < KW; ++k2) s += r[((k2 * NW + nw) * Gm::kBlocks + b) * 64 + lane];
                out[j] = s;
            }
            lds_barrier();
        } else {
#pragma unroll
            for (int j = 0; j < Gm::kOwnBlocks; ++j) out[j] = acc[j / MB][j % MB];
        }
#pragma unroll
        for (int nb = 0; nb < 4; ++nb)
#pragma unroll
            for (int mb = 0; mb < MB; ++mb) acc[nb][mb] = float4_t{0.f, 0.f, 0.f, 0.f};

        if (cu.seg_begin == 0 && cu.ku_end == KU) {
            store_c(cu.c, out);
        } else {
            const int which = (cu.c == first_col) ? 0 : 1;
            pcol[which] = cu.c;
            float *slot = p.partials + ((int64_t)wg * 2 + which) * Gm::kSlotFloats;
#pragma unroll
            for (int j = 0; j < Gm::kOwnBlocks; ++j) store_partial(slot, nw * Gm::kBlocks + kw + j * KW, lane, out[j]);
        }
    };

    // ---- main pipeline ----
    int issued = 0, computed = 0;
#pragma unroll
    for (int s = 0; s < P - 1; ++s) {
        if (!ld.done) {
            issue(ld, s);
            cursor_next<KW>(ld, KU);
            ++issued;
        }
    }
    int slot = 0, ld_slot = P - 1;
    while (!cp.done) {
        const int ahead = issued - computed - 1;  // stages issued after the one to compute
        if constexpr (P >= 4) {
            if (ahead >= 2) wait_vmcnt<2 * L>();
            else if (ahead == 1) wait_vmcnt<L>();
            else wait_vmcnt<0>();
        } else if constexpr (P == 3) {
            if (ahead >= 1) wait_vmcnt<L>();
            else wait_vmcnt<0>();
        } else {
            wait_vmcnt<0>();
        }
        if constexpr (NW > 1) lds_barrier();
        if (!ld.done) {
            issue(ld, ld_slot);
            cursor_next<KW>(ld, KU);
            ++issued;
            ld_slot = (ld_slot + 1 == P) ? 0 : ld_slot + 1;
        }

        // ---- compute one stage ----
        if (cp.ku + kw < cp.ku_end) {
            const uint8_t *base = smem + slot * Gm::kStageBytes;
            const half8_t *abase = (const half8_t *)(base + kw * Gm::kAFrags * 1024);
            const u32x4_t *wbase = (const u32x4_t *)(base + Gm::kABytes + (kw * NW + nw) * 4096);
            const uint8_t *sbase = base + Gm::kABytes + Gm::kWBytes + (kw * NW + nw) * 128;
            if constexpr (Gm::kFold) {
                // fp32 fold: each 128-row product is scaled once per output.
                half8_t a[MB][4];
#pragma unroll
                for (int mb = 0; mb < MB; ++mb)
#pragma unroll
                    for (int t = 0; t < 4; ++t) a[mb][t] = abase[(mb * 4 + t) * 64 + lane];
                float sc[16];
                const half8_t *sp = (const half8_t *)(sbase + lg * 32);
                const half8_t s0 = sp[0], s1 = sp[1];
#pragma unroll
                for (int i = 0; i < 8; ++i) { sc[i] = (float)s0[i]; sc[8 + i] = (float)s1[i]; }
#pragma unroll
                for (int nb = 0; nb < 4; ++nb) {
                    const u32x4_t wv = wbase[nb * 64 + lane];
                    float4_t tmp[MB];
#pragma unroll
                    for (int t = 0; t < 4; ++t) {
                        const half8_t b = dequant8(wv[t], dq);
#pragma unroll
                        for (int mb = 0; mb < MB; ++mb)
                            tmp[mb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(
                                b, a[mb][t], t == 0 ? float4_t{0.f, 0.f, 0.f, 0.f} : tmp[mb], 0, 0, 0);
                    }
#pragma unroll
                    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
                        for (int i = 0; i < 4; ++i) acc[nb][mb][i] += tmp[mb][i] * sc[nb * 4 + i];
                }
            } else {
                // Per-channel scales (applied at the end), or group scales
                // multiplied into the fp16 weights of column n = 16nb + lane%16.
                u32x4_t wv[4];
#pragma unroll
                for (int nb = 0; nb < 4; ++nb) wv[nb] = wbase[nb * 64 + lane];
                half2_t s2[4];
                if constexpr (!PER_CHANNEL) {
                    const _Float16 *sh = (const _Float16 *)sbase;
                    const int col = lane & 15;
#pragma unroll
                    for (int nb = 0; nb < 4; ++nb) {
                        const _Float16 v = sh[16 * (col >> 2) + 4 * nb + (col & 3)];
                        s2[nb] = half2_t{v, v};
                    }
                }
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    half8_t a[MB];
#pragma unroll
                    for (int mb = 0; mb < MB; ++mb) a[mb] = abase[(mb * 4 + t) * 64 + lane];
#pragma unroll
                    for (int nb = 0; nb < 4; ++nb) {
                        half8_t b = dequant8(wv[nb][t], dq);
                        if constexpr (!PER_CHANNEL) b = scale8(b, s2[nb]);
#pragma unroll
                        for (int mb = 0; mb < MB; ++mb)
                            acc[nb][mb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(b, a[mb], acc[nb][mb], 0, 0, 0);
                    }
                }
            }
        }
        ++computed;

        if (cp.ku + KW >= cp.ku_end) finish_segment(cp);
        cursor_next<KW>(cp, KU);
        slot = (slot + 1 == P) ? 0 : slot + 1;
    }

    auto own = [&](int j) { return nw * Gm::kBlocks + kw + j * KW; };
    publish_and_reduce<Gm::kOwnBlocks>(p, pcol, flags, wg, KU, total, grid, Gm::kSlotFloats, lane, own,
                                       store_c);
}

template <int MB, int NW, int KW>
hipError_t launch_variant(const GemmConfig &cfg, const GemmProblem &p, hipStream_t stream)
{
    const bool per_channel = (p.group_units == 0);
    GemmProblem arg = p;
    void *args[] = {&arg};
    if (per_channel) {
        using Gm = Geo<MB, NW, KW, true>;
        return hipLaunchKernel((const void *)&w4a16_lds_kernel<MB, NW, KW, true>, dim3(cfg.grid),
                               dim3(Gm::kThreads), args, 0, stream);
    }
    using Gm = Geo<MB, NW, KW, false>;
    return hipLaunchKernel((const void *)&w4a16_lds_kernel<MB, NW, KW, false>, dim3(cfg.grid),
                           dim3(Gm::kThreads), args, 0, stream);
}

}  // namespace

int slot_floats(const GemmConfig &cfg)
{
    return cfg.kind == kKindStream ? cfg.nb * cfg.mb * 256 : cfg.nw * 4 * cfg.mb * 256;
}

template <int MB, int NB>
hipError_t launch_stream(const GemmConfig &cfg, const GemmProblem &p, hipStream_t stream)
{
    constexpr int KW = kStreamWaves, OCC = kStreamOcc;
    constexpr int D = (MB == 1) ? (NB == 4 ? 3 : NB == 2 ? 4 : 6) : (NB == 4 ? 2 : 4);
    GemmProblem arg = p;
    void *args[] = {&arg};
    const void *fn = (p.group_units == 0) ? (const void *)&w4a16_stream_kernel<MB, NB, KW, D, OCC, true>
                                          : (const void *)&w4a16_stream_kernel<MB, NB, KW, D, OCC, false>;
    return hipLaunchKernel(fn, dim3(cfg.grid), dim3(64 * KW), args, 0, stream);
}

hipError_t launch_gemm(const GemmConfig &cfg, const GemmProblem &p, hipStream_t stream)
{
    if (cfg.kind == kKindStream) {
        switch (cfg.mb * 10 + cfg.nb) {
        case 11: return launch_stream<1, 1>(cfg, p, stream);
        case 12: return launch_stream<1, 2>(cfg, p, stream);
        case 14: return launch_stream<1, 4>(cfg, p, stream);
        case 21: return launch_stream<2, 1>(cfg, p, stream);
        case 22: return launch_stream<2, 2>(cfg, p, stream);
        case 24: return launch_stream<2, 4>(cfg, p, stream);
        default: return hipErrorInvalidValue;
        }
        return hipErrorInvalidValue;
    }
    const int key = cfg.mb * 100 + cfg.nw * 10 + cfg.kw;
    switch (key) {
    case 441: return launch_variant<4, 4, 1>(cfg, p, stream);
    case 421: return launch_variant<4, 2, 1>(cfg, p, stream);
    case 411: return launch_variant<4, 1, 1>(cfg, p, stream);
    case 841: return launch_variant<8, 4, 1>(cfg, p, stream);
    case 821: return launch_variant<8, 2, 1>(cfg, p, stream);
    case 811: return launch_variant<8, 1, 1>(cfg, p, stream);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace marlin
