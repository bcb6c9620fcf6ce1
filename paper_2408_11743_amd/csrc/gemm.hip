// W4A16 GEMM for gfx950: C[M,N] = A[M,K] * (s * (q - 8)), fp32 accumulation.
//
// Design (the ideas of the paper's Section 3.4, re-derived for CDNA4):
//  * Transposed product, as the paper does for its sparse kernel (Section 4):
//    each v_mfma_f32_16x16x32_f16 multiplies a 16(n) x 32(k) block of W^T
//    (first operand) by a 32(k) x 16(m) block of A^T.  A lane's first operand
//    is 8 consecutive k of one column n: exactly one packed 32-bit word of
//    codes, so one 16-byte load feeds four MFMA steps ("Maximizing Loading
//    Bandwidth", "Dequantization and Tensor Cores").
//  * int4 -> fp16 by bit operations only.  A code masked into the low bits of
//    a zero-exponent fp16 number IS the fp16 value q * 2^-24 (a subnormal,
//    which the matrix cores consume exactly); the code one nibble higher is
//    16 q * 2^-24.  So one AND yields two operands, and a word of eight codes
//    costs one shift and four ANDs.  The factor 16 of the upper nibbles is
//    moved to the activations (their elements 2, 3, 6, 7 are multiplied by
//    1/16, exact for normal fp16), the zero point to one extra MFMA per
//    k-step against the codes 8 (shared by all column blocks, subtracted),
//    and 2^24 into the final conversion.  This is the magic-number idea of
//    the "Dequantization and Tensor Cores" paragraph with the magic number 0:
//    no subtraction is needed per weight at all.  (Row groups of 64 rows use
//    the paper's magic number itself, below.)
//  * Group scales multiply each 128-row fp32 partial product once, fused
//    with the bias add (v_fma_mix_f32 reads the fp16 scale directly), or,
//    with 64-row groups, the fp16 weights before the product; per-channel
//    scales multiply the final sum ("Groups and Instruction Ordering").
//  * The waves of a work-group (four; eight, two per SIMD, with a single
//    16-row block of A or a single 16-column block, so that one wave's
//    dependent MFMA chain and LDS latency overlap the other's) take
//    consecutive 128-row blocks of one column tile per stage and meet in LDS
//    when a tile segment ends (Algorithm 1's reduction over waves that share
//    an output tile).
//  * Stream-K style striped partitioning over a persistent grid: work-group w
//    owns the contiguous range [w*T/grid, (w+1)*T/grid) of (column tile,
//    128-row block) units, column-major, wrapping into the next column
//    ("Striped Partitioning").  A column tile shared by several work-groups
//    is combined through fp32 partial slots in the workspace; whichever
//    work-group completes the tile's arrival count sums the slots in
//    work-group order (bitwise reproducible) and writes C.  No work-group
//    ever waits for another, so no co-residency is assumed.
#include <hip/hip_runtime.h>
#include <stdio.h>

#include "device.h"
#include "internal.h"

namespace marlin {
namespace {

using namespace dev;

constexpr float kTwo24 = 16777216.0f;  // undoes the 2^-24 of the subnormal operands

// Eight codes of one packed word -> eight MFMA operands in element order
// j = 0..7 (code j sits in nibble (j >> 1) + 4 (j & 1)).  Elements 0, 1, 4, 5
// are q * 2^-24, elements 2, 3, 6, 7 are 16 q * 2^-24.
__device__ __forceinline__ half8_t dequant_sub(uint32_t x)
{
    const uint32_t y = x >> 8;
    return __builtin_bit_cast(half8_t, u32x4_t{x & 0x000F000Fu, x & 0x00F000F0u, y & 0x000F000Fu,
                                               y & 0x00F000F0u});
}

// Eight fp16 weights times one scale (in both halves of s2), one rounding each.
__device__ __forceinline__ half8_t scale_pairs(half8_t w, half2_t s2)
{
    const u32x4_t u = __builtin_bit_cast(u32x4_t, w);
    return __builtin_bit_cast(half8_t, u32x4_t{as_u32(as_h2(u[0]) * s2), as_u32(as_h2(u[1]) * s2),
                                               as_u32(as_h2(u[2]) * s2), as_u32(as_h2(u[3]) * s2)});
}

// Activation operand matching dequant_sub: elements 2, 3, 6, 7 times 1/16.
__device__ __forceinline__ half8_t prescale(half8_t a)
{
    const u32x4_t u = __builtin_bit_cast(u32x4_t, a);
    const half2_t r = {(_Float16)0.0625f, (_Float16)0.0625f};
    return __builtin_bit_cast(half8_t, u32x4_t{u[0], as_u32(as_h2(u[1]) * r), u[2], as_u32(as_h2(u[3]) * r)});
}

// Zero-point operand: the codes 8 in the same encoding, 8 * 2^-24 in the
// elements paired with unscaled activations and 128 * 2^-24 where the
// activation carries 1/16.  Against the prescaled activations it yields
// 8 * sum_k A_k * 2^-24 for every column n, which is subtracted.  Because it
// is exactly the operand of a column whose codes are all 8, such a column's
// two products are the same computation and cancel exactly (the matrix
// cores' fp32 rounding is not symmetric under negation, so the constant is
// subtracted rather than added negated).
__device__ __forceinline__ half8_t bias_operand()
{
    return __builtin_bit_cast(half8_t, u32x4_t{0x00080008u, 0x00800080u, 0x00080008u, 0x00800080u});
}

// One stage of 2:4 sparse weights for NB column blocks: per block, two words
// of kept codes (rows 0..63 and 64..127 of the 128-row block) and one word of
// row indices (16 bits per half).  Loaded with the narrowest loads that cover
// them: NB = 4 two 16-byte code loads and one 16-byte index load; NB = 2 one
// 16-byte and one 8-byte; NB = 1 one 8-byte and one 4-byte.
template <int NB>
struct SparseWords {
    u32x4_t c[NB == 4 ? 2 : 1];
    u32x4_t m;
    __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t r, uint32_t lane_off, uint32_t codes_off,
                                         uint32_t meta_off, uint32_t next = 0)
    {
        (void)next;
        if constexpr (NB == 4) {
            c[0] = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(r, lane_off, codes_off, kAuxNonTemporal));
            c[1] = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(r, lane_off + 1024, codes_off, kAuxNonTemporal));
            m = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(r, lane_off, meta_off, kAuxNonTemporal));
        } else if constexpr (NB == 2) {
            c[0] = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(r, lane_off, codes_off, kAuxNonTemporal));
            const uint64_t v = __builtin_bit_cast(uint64_t, __builtin_amdgcn_raw_buffer_load_b64(r, lane_off, meta_off, kAuxNonTemporal));
            m = u32x4_t{(uint32_t)v, (uint32_t)(v >> 32), 0u, 0u};
        } else {
            const uint64_t v = __builtin_bit_cast(uint64_t, __builtin_amdgcn_raw_buffer_load_b64(r, lane_off, codes_off, kAuxNonTemporal));
            c[0] = u32x4_t{(uint32_t)v, (uint32_t)(v >> 32), 0u, 0u};
            m = u32x4_t{__builtin_amdgcn_raw_buffer_load_b32(r, lane_off, meta_off, kAuxNonTemporal), 0u, 0u, 0u};
        }
    }
    // kept codes of column block b, rows 64h .. 64h + 63
    __device__ __forceinline__ uint32_t code(int b, int h) const { return c[(2 * b + h) >> 2][(2 * b + h) & 3]; }
    __device__ __forceinline__ uint32_t meta(int b) const { return m[b]; }
};

// NB = 8 (two packed 64-column units, the second `next` bytes on): the
// NB = 4 loads of each, six per stage.
template <>
struct SparseWords<8> {
    SparseWords<4> u[2];
    __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t r, uint32_t lane_off, uint32_t codes_off,
                                         uint32_t meta_off, uint32_t next)
    {
        u[0].load(r, lane_off, codes_off, meta_off);
        u[1].load(r, lane_off, codes_off + next, meta_off + next);
    }
    __device__ __forceinline__ uint32_t code(int b, int h) const { return u[b >> 2].code(b & 3, h); }
    __device__ __forceinline__ uint32_t meta(int b) const { return u[b >> 2].meta(b & 3); }
};

// Sparse product of one column block and one 16-row block over 128 rows of
// K: two smfmac steps (rows 0..63, 64..127), each taking the activation
// operands of two dense k-steps.
__device__ __forceinline__ float4_t smfmac2(half8_t w0, half8_t w1, const half8_t *a, uint32_t idx, float4_t c)
{
    typedef _Float16 half16_t __attribute__((ext_vector_type(16)));
    const half16_t b0 = __builtin_shufflevector(a[0], a[1], 0, 1, 2, 3, 4, 5, 6, 7, 8, 9, 10, 11, 12, 13, 14, 15);
    const half16_t b1 = __builtin_shufflevector(a[2], a[3], 0, 1, 2, 3, 4, 5, 6, 7, 8, 9, 10, 11, 12, 13, 14, 15);
    c = __builtin_amdgcn_smfmac_f32_16x16x64_f16(w0, b0, c, (int)idx, 0, 0);
    return __builtin_amdgcn_smfmac_f32_16x16x64_f16(w1, b1, c, (int)idx, 0, 1);
}

// ---------------------------------------------------------------------------
// Register-streaming kernel.
//
// A work-group owns a column tile of 16*NB columns (NB 16-column blocks; NB = 8
// spans two 64-column tiles of the packed layout) of one row group (16*MB
// rows: MB = 1, 2, or 4 with 128-column dense tiles) over a range of 128-row
// blocks of K (the striped partition); its KW waves take consecutive 128-row
// blocks of each stage (waves split K), so no weight or activation byte is
// shared between waves: each lane loads exactly its MFMA weight operands
// (16-byte non-temporal buffer loads of the pre-shuffled weights) into a
// D-deep ring of registers, and the stage's activation rows (which hit L2)
// arrive by direct-to-LDS loads in a D-deep per-wave LDS ring.  The loop is
// unrolled over the ring so register slots are static and the vmcnt waits
// keep D-1 stages in flight while one is computed.  A wave whose block lies
// past the end of a segment loads through an empty buffer descriptor (no
// memory is touched, zeros return) and skips the stage's arithmetic.
//
// Codes become MFMA operands as subnormal fp16 numbers with a separate
// zero-point product and the group scale applied to each 128-row fp32
// partial product (MB <= 2), or, with four row blocks, by the magic number
// with the group scale on the fp16 weights: that path touches no fp32 value
// per stage, so its 128 accumulators stay with the matrix cores.
//
// Cross-work-group combination, at the end: the work-group's first tile (if
// shared) was written to slot 0 when its segment ended; its last tile (if
// shared) is written to slot 1 now; it then arrives at both tiles' counters,
// and whoever completes a count sums the slots (device.h, combine_tiles).
//
// 2:4 sparse weights (SPARSE, Section 4): the same schedule with the sparse
// packed layout (per 64 x 128 unit: 2 KiB of kept codes, 1 KiB of 2-bit row
// indices) and v_smfmac_f32_16x16x64_f16, whose first operand is the
// compressed weights (two kept values of every 4 rows, row indices in a
// VGPR) and whose second is the dense activations.  With the transposed
// product the sparse operand is the weights, as the paper's 2:4 kernel does.
// The activation reads are the dense path's (one smfmac takes the operands of
// two 16x16x32 steps); codes are converted with the magic number (exact
// q - 8, no zero-point product: the zero point of a pruned row would depend
// on the row indices).
template <int MB, int NB, int D, int AR, int KW, bool PER_CHANNEL, bool SPARSE>
__device__ __forceinline__ void stream_body(const GemmProblem &p)
{
    constexpr int kBlocks = NB * MB;               // 16x16 output blocks per wave
    constexpr int kOwn = (kBlocks + KW - 1) / KW;  // blocks a wave owns after the LDS reduction
    constexpr int kSLoads = (NB + 1) / 2;          // 16-byte scale loads per stage
    constexpr int kSL = PER_CHANNEL ? 0 : kSLoads;
    // weight loads per stage: NB 16-byte words (dense), or codes and row
    // indices (sparse: 2 + 1 for NB = 4, else 1 + 1)
    constexpr int kWL = SPARSE ? (NB == 8 ? 6 : NB == 4 ? 3 : 2) : NB;
    constexpr uint32_t kUnitBytes = SPARSE ? 3072u : 4096u;  // per 64 x 128 unit
    // Four row blocks (dense) convert codes with the magic number too (exact
    // q - 8, group scales on the fp16 weights; see compute)
    constexpr bool kMagic = SPARSE || MB == 4;
    constexpr float kOutScale = kMagic ? 1.0f : kTwo24;      // subnormal operands carry 2^-24
    // Activation rows through LDS (one or two 16-row blocks): the 4*AR rows of
    // the tile's row group for the stage's 128-row block land in a per-wave
    // LDS ring by AR direct-to-LDS loads (only real rows are fetched; the
    // register ring holds weights and scales only).
    constexpr int kARows = 4 * AR;
    constexpr int kAStage = kARows * 256;            // bytes per wave and stage
    constexpr int kLoads = AR + kWL + kSL;           // vector-memory ops per stage
    static_assert(KW == 4 || (KW == 8 && (MB == 1 || NB == 1)), "four waves, or eight with one row block or column block");
    static_assert(MB <= 2 || (MB == 4 && NB == 8 && KW == 4 && !SPARSE),
                  "one or two row blocks; four only with 128-column dense tiles and four waves");
    // Tiles too large for a reduction buffer beside the activation ring (64 x
    // 128 per wave) meet in the ring slot of the stage that ends the segment;
    // that configuration also loads every row of its group, and holds fewer
    // activation addresses.
    static_assert(AR >= 1 && kARows <= 16 * MB, "at least 4 rows");
    static_assert((D - 1) * kLoads + kWL + kSL < 64, "vmcnt range");
    // The waves' tiles meet in LDS: in a buffer of their own up to two row
    // blocks; with four (64 x 128 per wave, 32 KiB of fp32, beside a 128 KiB
    // activation ring) in the ring slot of the stage that ends the segment.
    constexpr bool kRingRed = MB == 4;
    static_assert(!kRingRed || (kARows == 16 * MB && (kAStage / 1024) % KW == 0 && kBlocks % (kAStage / 1024) == 0),
                  "ring-slot reduction: whole row groups, rounds of whole slots");
    __shared__ float4_t red[kRingRed ? 1 : KW * kBlocks * 64];
    __shared__ __attribute__((aligned(16))) uint8_t a_lds[KW * D * kAStage + 256];
    __shared__ int flags[2];

    const int lane = threadIdx.x & 63;
    const int kw = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave index, scalar
    const int lg = lane >> 4;
    const int KU = p.KU;
    const int grid = gridDim.x;
    const int wg = xcd_local_wg(blockIdx.x, grid);
    const int u0 = range_start(p, wg, grid);
    const int u1 = range_start(p, wg + 1, grid);
    const int c_first = tile_of(p, u0);
    const int c_last = tile_of(p, u1 - 1);
    const int k0 = u0 - c_first * KU;  // first block in the first tile
    const int k1 = u1 - c_last * KU;   // end block in the last tile (1..KU)

    // A tile c is column tile c / rg and row group c % rg (rows 16*MB*(c % rg)
    // onwards when M exceeds 16*MB; one group otherwise).  Byte offsets of tile
    // c's block 0: weights (4 KiB per (64 columns x 128 rows) block, 1 KiB per
    // 16 columns; sparse: 3 KiB per block, this column block's codes at
    // 1 KiB * (q/2) + 8 * (q%2) for column block q of the 64) and scale rows
    // (128 B per 64 columns).
    const uint32_t RG = (uint32_t)p.rg;
    auto col_of = [&](int c) -> uint32_t { return RG == 1 ? (uint32_t)c : (uint32_t)c / RG; };
    auto w_tile = [&](int c) -> uint32_t {
        const uint32_t nbg = col_of(c) * NB;
        if constexpr (SPARSE)
            return (nbg >> 2) * (uint32_t)KU * kUnitBytes + ((nbg & 3u) >> 1) * 1024u + (nbg & 1u) * 8u;
        return ((nbg >> 2) * (uint32_t)KU * 4u + (nbg & 3u)) << 10;
    };
    // sparse: the row indices of column block q lie 2 KiB + 4q past the unit
    // start, i.e. this much past the codes
    auto meta_delta = [&](int c) -> uint32_t {
        const uint32_t q = (col_of(c) * NB) & 3u;
        return 2048u + 4u * q - (q >> 1) * 1024u - (q & 1u) * 8u;
    };
    auto s_tile = [&](int c) -> uint32_t {
        const uint32_t nbg = col_of(c) * NB;
        return (((nbg >> 2) * (uint32_t)p.G) << 7) + (nbg & 3u) * 8u;
    };
    // First row of tile c's row group, and the rows it has (1 .. 16*MB).
    auto row0_of = [&](int c) -> int { return RG == 1 ? 0 : (int)((uint32_t)c - col_of(c) * RG) * (16 * MB); };
    auto rows_of = [&](int c) -> int {
        const int r = p.M - row0_of(c);
        return r < 16 * MB ? r : 16 * MB;
    };

    // Per-lane parts of the load addresses (fixed for the whole kernel).
    const uint32_t w_lane = (uint32_t)kw * kUnitBytes + (uint32_t)lane * 16u;
    // Scale runs: lane group g of the packed 128-byte row holds, for each
    // 16-column block, the scales of columns 4g .. 4g + 3 (the accumulator
    // columns of lanes 16g .. 16g + 15, which the subnormal path scales); the
    // magic path scales the weight operand, whose column is lane % 16, so a
    // lane loads run (lane % 16) / 4 and keeps element lane % 4 of it.
    const uint32_t s_lane = (MB == 4 ? (uint32_t)((lane & 15) >> 2) : (uint32_t)lg) * 32u;
    const uint32_t s_sel = 0x01000100u + (uint32_t)(lane & 3) * 0x02020202u;  // v_perm: that half, twice
    (void)s_sel;
    // Direct-to-LDS activation loads: load i, lane l fetches row r = 4i + l/16,
    // 16-byte chunk (l % 16) ^ r of the block (an XOR swizzle, so that the
    // MFMA-operand reads of 16 rows hit 16 different bank groups).
    // The MFMA operands are read back with ds_read_b128 at per-lane LDS
    // addresses fixed for each ring slot; lanes of rows past the 4*AR loaded
    // ones read a zero row (the 256 bytes after the ring) instead.
    // Four row blocks: rows r and r + 16 share the swizzle, so loads i >= 4
    // add 16 rows to the offset of load i % 4 when they are issued, and the
    // operand reads take the ring slot and row block as instruction offsets
    // from one address per k-step (fewer registers held across the loop).
    constexpr int kADma = kRingRed ? 4 : AR;
    uint32_t a_dma[kADma];
    uint32_t a_rd[kRingRed ? 1 : D][kRingRed ? 1 : MB][4];
#pragma unroll
    for (int i = 0; i < kADma; ++i) {
        const int r = 4 * i + lg;
        a_dma[i] = (uint32_t)(r * p.K + (((lane & 15) ^ (r & 15)) * 8)) * 2u + (uint32_t)kw * 256u;
    }
    const uint32_t a_rows16 = (uint32_t)p.K * 32u;  // 16 rows of A, bytes
    const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint8_t *)a_lds;
    const uint32_t zero_row = lds0 + KW * D * kAStage;
    const uint32_t lds_wave = lds0 + (uint32_t)(kw * D * kAStage);  // this wave's ring
    // Rows of A past M lie past the end of the A buffer: their loads return 0.
    const uint32_t w_bytes = SPARSE ? (uint32_t)p.K / 8u * (uint32_t)p.N * 3u : (uint32_t)p.K * (uint32_t)(p.N / 2);

    const uint32_t s_bytes = (uint32_t)p.G * (uint32_t)p.N * 2u;
    // NB = 8: the wave's column blocks 4..7 lie in the next 64-column tile of
    // the packed layout, KU * 4 KiB further on (weights) and G * 128 bytes
    // further on (scales)
    const uint32_t w_next = (uint32_t)KU * kUnitBytes;
    const uint32_t s_next = (uint32_t)p.G * 128u;

    u32x4_t wr[SPARSE ? 1 : D][NB];   // dense weights
    SparseWords<NB> sw[SPARSE ? D : 1];  // sparse codes and row indices
    half8_t sr[D][kSLoads];

    // ---- load cursor: wave-uniform, advanced once per stage ----
    int ld_c = c_first, ld_ku = k0;
    int ld_end = (c_first == c_last) ? k1 : KU;
    uint32_t ld_w = w_tile(ld_c) + (uint32_t)ld_ku * kUnitBytes;
    uint32_t ld_s = s_tile(ld_c);
    uint32_t ld_md = SPARSE ? meta_delta(ld_c) : 0u;
    // The tile's activation rows as their own buffer: rows past M read 0.
    const uint16_t *ld_a = p.A + (int64_t)row0_of(ld_c) * p.K;
    uint32_t a_bytes = (uint32_t)rows_of(ld_c) * (uint32_t)p.K * 2u;

    auto issue = [&](int j) {
        const int my = ld_ku + kw;
        const bool on = my < ld_end;
        {  // first, so a stage's LDS rows are its oldest loads
            const __amdgpu_buffer_rsrc_t rd =
                __builtin_amdgcn_make_buffer_rsrc((void *)ld_a, (short)0, on ? a_bytes : 0u, kBufferFlags);
            // The slot's LDS address is formed here from one per-wave base
            // (the opaque copy keeps the compiler from holding all D * AR
            // destination addresses in scalar registers across the loop).
            uint32_t slot = lds_wave;
            asm volatile("" : "+s"(slot));
            slot += (uint32_t)(j * kAStage);
            uint32_t dma[kADma];
#pragma unroll
            for (int i = 0; i < kADma; ++i) {
                dma[i] = a_dma[i];
                if constexpr (kRingRed) asm volatile("" : "+v"(dma[i]));  // formed per stage, not held
            }
#pragma unroll
            for (int i = 0; i < AR; ++i)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(
                    rd, (__attribute__((address_space(3))) void *)(uintptr_t)(slot + (uint32_t)(i * 1024)), 16,
                    (int)(dma[i % kADma] + (uint32_t)(i / kADma) * a_rows16), ld_ku * 256, 0, 0);
        }
        issue_order_point();  // the rows are the stage's oldest loads
        const __amdgpu_buffer_rsrc_t rw =
            __builtin_amdgcn_make_buffer_rsrc((void *)p.W, (short)0, on ? w_bytes : 0u, kBufferFlags);
        if constexpr (SPARSE) {
            sw[j].load(rw, w_lane, ld_w, ld_w + ld_md, w_next);
        } else {
#pragma unroll
            for (int b = 0; b < NB; ++b)
                wr[j][b] = __builtin_bit_cast(
                    u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rw, w_lane + (b & 3) * 1024,
                                                                   ld_w + (b >> 2) * w_next, kAuxNonTemporal));
        }
        if constexpr (!PER_CHANNEL) {
            const __amdgpu_buffer_rsrc_t rs =
                __builtin_amdgcn_make_buffer_rsrc((void *)p.S, (short)0, on ? s_bytes : 0u, kBufferFlags);
            const uint32_t s_off = ld_s + ((uint32_t)scale_row_of(my, p) << 7);
            if constexpr (NB == 1) {
                // four scales: an 8-byte load (a 16-byte one would leave half
                // of its destination dead, and the compiler would wait for the
                // load before reusing those registers)
                const uint64_t v = __builtin_bit_cast(
                    uint64_t, __builtin_amdgcn_raw_buffer_load_b64(rs, s_lane, s_off, 0));
                sr[j][0] = __builtin_bit_cast(half8_t, u32x4_t{(uint32_t)v, (uint32_t)(v >> 32), 0u, 0u});
            } else {
#pragma unroll
                for (int i = 0; i < kSLoads; ++i)
                    sr[j][i] = __builtin_bit_cast(
                        half8_t, __builtin_amdgcn_raw_buffer_load_b128(rs, s_lane + (i & 1) * 16,
                                                                       s_off + (i >> 1) * s_next, 0));
            }
        }
        issue_order_point();  // stages do not interleave
    };
    auto advance_ld = [&]() {
        ld_ku += KW;
        ld_w += KW * kUnitBytes;
        if (ld_ku >= ld_end) {  // next segment (rare)
            ld_c += 1;
            ld_ku = 0;
            ld_end = (ld_c < c_last) ? KU : (ld_c == c_last) ? k1 : 0;  // 0: past the range
            ld_w = w_tile(ld_c);
            ld_s = s_tile(ld_c);
            if constexpr (SPARSE) ld_md = meta_delta(ld_c);
            if (RG > 1 && ld_end > 0) {
                ld_a = p.A + (int64_t)row0_of(ld_c) * p.K;
                a_bytes = (uint32_t)rows_of(ld_c) * (uint32_t)p.K * 2u;
            }
        }
    };

    // Issue the first D stages before anything else.
#pragma unroll
    for (int j = 0; j < D; ++j) {
        issue(j);
        advance_ld();
    }
    // While they are on their way: the LDS read addresses and, where some of
    // the 16*MB operand rows are not loaded, the zero row (written by an
    // instruction of its own, so that the compiler's tracking of the
    // direct-to-LDS writes in flight adds no wait) and the barrier that
    // publishes it before any wave reads it.  No wave waits for the others
    // before issuing its loads.
    if constexpr (kARows < 16 * MB) {
        if (threadIdx.x < 16)
            asm volatile("ds_write_b128 %0, %1" ::"v"(zero_row + threadIdx.x * 16u), "v"(u32x4_t{0u, 0u, 0u, 0u})
                         : "memory");
    }
#pragma unroll
    for (int j = 0; j < (kRingRed ? 1 : D); ++j)
#pragma unroll
        for (int mb = 0; mb < (kRingRed ? 1 : MB); ++mb)
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                const int am = mb * 16 + (lane & 15);
                const uint32_t chunk = (uint32_t)(((4 * t + lg) ^ (am & 15)) << 4);
                a_rd[j][mb][t] = (am < kARows) ? lds0 + (uint32_t)((kw * D + j) * kAStage + am * 256) + chunk
                                               : zero_row + chunk;
            }
    // With one row block the barrier also lines the waves up before the
    // first stage, which measured faster even where no row is zero; with
    // two it measured slower and is kept only for the zero row.
    if constexpr (kARows < 16 * MB || MB == 1) lds_barrier();

    // Stages of this work-group: ceil(segment length / KW) per segment.
    const int n_st = (c_first == c_last)
                         ? (k1 - k0 + KW - 1) / KW
                         : (KU - k0 + KW - 1) / KW + (c_last - c_first - 1) * ((KU + KW - 1) / KW) +
                               (k1 + KW - 1) / KW;

    float4_t acc[NB][MB];
    float4_t bacc[PER_CHANNEL ? MB : 1];  // per-channel: zero-point sum, chained like acc
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) acc[b][mb] = float4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int mb = 0; mb < (PER_CHANNEL ? MB : 1); ++mb) bacc[mb] = float4_t{0.f, 0.f, 0.f, 0.f};

    half8_t kb = bias_operand();
    asm volatile("" : "+v"(kb));  // keep the constant in vector registers
    const float4_t zero4 = {0.f, 0.f, 0.f, 0.f};
    const DequantConsts dq = dequant_consts();  // sparse codes: magic-number conversion
    (void)dq;

    // One stage: for each 16-row block of A, four MFMA steps per column block
    // plus four for the zero point.  Group scales: the stage's zero-point
    // product is subtracted from each column block's 128-row product, and the
    // difference scaled and accumulated in one fused multiply-add per value.
    auto compute = [&](int j, int later) {
        half8_t a[4 * MB];
        {
            // Wait for this stage's direct-to-LDS rows: the loads issued
            // after them are the stage's own weight and scale loads and
            // `later` stages (vector-memory ops complete in order).  The
            // reads are written as assembly, with their own lgkmcnt wait, so
            // that the compiler's conservative tracking of direct-to-LDS
            // writes does not add waits for the whole ring.
            wait_vmcnt_n(later * kLoads + kWL + kSL);
            u32x4_t v[4 * MB];
#pragma unroll
            for (int mb = 0; mb < MB; ++mb)
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    if constexpr (kRingRed)  // slot j, row block mb: kAStage and 4 KiB from the k-step's address
                        asm volatile("ds_read_b128 %0, %1 offset:%2"
                                     : "=v"(v[mb * 4 + t])
                                     : "v"(a_rd[0][0][t]), "i"(j * kAStage + mb * 4096));
                    else
                        asm volatile("ds_read_b128 %0, %1" : "=v"(v[mb * 4 + t]) : "v"(a_rd[j][mb][t]));
                }
            // The wait "redefines" the results, so no use of them can be
            // scheduled before the data has arrived.
            if constexpr (MB == 1) {
                asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(v[0]), "+v"(v[1]), "+v"(v[2]), "+v"(v[3])::"memory");
            } else if constexpr (MB == 4) {
                asm volatile("s_waitcnt lgkmcnt(0)"
                             : "+v"(v[0]), "+v"(v[1]), "+v"(v[2]), "+v"(v[3]), "+v"(v[4]), "+v"(v[5]), "+v"(v[6]),
                               "+v"(v[7]), "+v"(v[8]), "+v"(v[9]), "+v"(v[10]), "+v"(v[11]), "+v"(v[12]),
                               "+v"(v[13]), "+v"(v[14]), "+v"(v[15])::"memory");
            } else {
                asm volatile("s_waitcnt lgkmcnt(0)"
                             : "+v"(v[0]), "+v"(v[1]), "+v"(v[2]), "+v"(v[3]), "+v"(v[4]), "+v"(v[5]), "+v"(v[6]),
                               "+v"(v[7])::"memory");
            }
#pragma unroll
            for (int i = 0; i < 4 * MB; ++i)
                a[i] = kMagic ? __builtin_bit_cast(half8_t, v[i]) : prescale(__builtin_bit_cast(half8_t, v[i]));
        }
        if constexpr (MB == 4) {
            // Four row blocks: q - 8 exactly by the magic number, times the
            // group scale in fp16 (one rounding per weight, the scale applied
            // to the weights before the product: Section 3.4, "Groups and
            // Instruction Ordering"), straight into the MFMA chains, which
            // run over the whole segment; each converted weight feeds four
            // MFMAs and no fp32 value is touched per stage.
            half2_t s2[NB];
            if constexpr (!PER_CHANNEL) {
#pragma unroll
                for (int b = 0; b < NB; ++b) {
                    const u32x4_t v = __builtin_bit_cast(u32x4_t, sr[j][b >> 1]);
                    s2[b] = as_h2(__builtin_amdgcn_perm(v[2 * (b & 1) + 1], v[2 * (b & 1)], s_sel));
                }
            }
#pragma unroll
            for (int t = 0; t < 4; ++t) {
#pragma unroll
                for (int b = 0; b < NB; ++b) {
                    half8_t w = dequant_magic(wr[j][b][t], dq);
                    if constexpr (!PER_CHANNEL) w = scale_pairs(w, s2[b]);
#pragma unroll
                    for (int mb = 0; mb < MB; ++mb) acc[b][mb] = mfma(w, a[mb * 4 + t], acc[b][mb]);
                }
            }
        } else if constexpr (SPARSE) {
#pragma unroll
            for (int b = 0; b < NB; ++b) {
                const half8_t w0 = dequant_magic(sw[j].code(b, 0), dq);
                const half8_t w1 = dequant_magic(sw[j].code(b, 1), dq);
                if constexpr (PER_CHANNEL) {
#pragma unroll
                    for (int mb = 0; mb < MB; ++mb) acc[b][mb] = smfmac2(w0, w1, a + mb * 4, sw[j].meta(b), acc[b][mb]);
                } else {
                    // scales of block b: halves 4b .. 4b+3 of this lane's run
                    const half8_t sv = sr[j][b >> 1];
#pragma unroll
                    for (int mb = 0; mb < MB; ++mb) {
                        const float4_t t4 = smfmac2(w0, w1, a + mb * 4, sw[j].meta(b), zero4);
#pragma unroll
                        for (int i = 0; i < 4; ++i)
                            acc[b][mb][i] = __builtin_fmaf(t4[i], (float)sv[(b & 1) * 4 + i], acc[b][mb][i]);
                    }
                }
            }
        } else if constexpr (PER_CHANNEL) {
#pragma unroll
            for (int t = 0; t < 4; ++t) {
#pragma unroll
                for (int mb = 0; mb < MB; ++mb) bacc[mb] = mfma(kb, a[mb * 4 + t], bacc[mb]);
#pragma unroll
                for (int b = 0; b < NB; ++b) {
                    const half8_t w = dequant_sub(wr[j][b][t]);
#pragma unroll
                    for (int mb = 0; mb < MB; ++mb) acc[b][mb] = mfma(w, a[mb * 4 + t], acc[b][mb]);
                }
            }
        } else {
            // k-step outer, column block inner: consecutive MFMAs are
            // independent.  Column blocks go in passes of at most four (NB = 8:
            // two passes), which bounds the temporaries; the zero-point
            // product of the first pass serves both.
            constexpr int kCB = NB < 4 ? NB : 4;
            float4_t tb[MB];
#pragma unroll
            for (int c0 = 0; c0 < NB; c0 += kCB) {
                float4_t tmp[kCB][MB];
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    if (c0 == 0) {
#pragma unroll
                        for (int mb = 0; mb < MB; ++mb) tb[mb] = mfma(kb, a[mb * 4 + t], t == 0 ? zero4 : tb[mb]);
                    }
#pragma unroll
                    for (int b = 0; b < kCB; ++b) {
                        const half8_t w = dequant_sub(wr[j][c0 + b][t]);
#pragma unroll
                        for (int mb = 0; mb < MB; ++mb)
                            tmp[b][mb] = mfma(w, a[mb * 4 + t], t == 0 ? zero4 : tmp[b][mb]);
                    }
                }
#pragma unroll
                for (int b = 0; b < kCB; ++b) {
                    // scales of block c0 + b: halves 4(c0 + b) .. +3 of this lane's runs
                    const half8_t sv = sr[j][(c0 + b) >> 1];
#pragma unroll
                    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
                        for (int i = 0; i < 4; ++i)
                            acc[c0 + b][mb][i] = __builtin_fmaf(tmp[b][mb][i] - tb[mb][i],
                                                                (float)sv[((c0 + b) & 1) * 4 + i], acc[c0 + b][mb][i]);
                }
            }
        }
    };

    // block index blk = b*MB + mb; wave kw owns blk = kw + j*KW (< kBlocks)
    auto own = [&](int j) { return kw + j * KW; };
    auto store_c = [&](int c, const float4_t *out) {
        const int r0 = row0_of(c), rows = rows_of(c);
        const int col = (int)col_of(c);
#pragma unroll
        for (int j = 0; j < kOwn; ++j) {
            const int blk = own(j);
            if (blk >= kBlocks) break;
            const int b = blk / MB, mb = blk % MB;
            const int m = mb * 16 + (lane & 15);
            if (m < rows) {
                const int nbg = col * NB + b;
                float4_t v = out[j];
                if constexpr (PER_CHANNEL) {
                    const half4_t s4 = *(const half4_t *)(p.S + (int64_t)(nbg >> 2) * 64 + lg * 16 + (nbg & 3) * 4);
#pragma unroll
                    for (int i = 0; i < 4; ++i) v[i] *= (float)s4[i] * kOutScale;
                } else {
#pragma unroll
                    for (int i = 0; i < 4; ++i) v[i] *= kOutScale;
                }
                const half4_t h = {(_Float16)v[0], (_Float16)v[1], (_Float16)v[2], (_Float16)v[3]};
                *(half4_t *)(p.C + (int64_t)(r0 + m) * p.N + nbg * 16 + lg * 4) = h;
            }
        }
    };

    const int slot_floats = kBlocks * 256;
    float *const my_slots = p.partials + (int64_t)wg * 2 * slot_floats;  // slot 0; slot 1 follows
    bool has_first = false, has_last = false;
    float4_t last_out[kOwn];
#pragma unroll
    for (int j = 0; j < kOwn; ++j) last_out[j] = zero4;

    // ---- compute cursor ----
    int cp_c = c_first, cp_ku = k0, cp_begin = k0;
    int cp_end = (c_first == c_last) ? k1 : KU;

    // A segment is complete: sum the waves' tiles in LDS, then write C
    // (whole column), keep the sum (shared last tile) or write slot 0
    // (shared first tile).
    auto finish_segment = [&](int j) {
        if constexpr (PER_CHANNEL && !kMagic) {
#pragma unroll
            for (int b = 0; b < NB; ++b)
#pragma unroll
                for (int mb = 0; mb < MB; ++mb) acc[b][mb] -= bacc[mb];
#pragma unroll
            for (int mb = 0; mb < MB; ++mb) bacc[mb] = zero4;
        }
        float4_t out[kOwn];
        if constexpr (!kRingRed) {
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
                } else {
                    out[j] = zero4;
                }
            }
            lds_barrier();
        } else {
            // Every wave's ring slot j is free: the wave has read its rows
            // (its later stages land in other slots), and the stage's refill
            // is issued after the last barrier here.  Rounds of kR blocks
            // (one slot, 1 KiB each): every wave writes its blocks
            // r*kR .. r*kR + kR-1, then sums its own among them over the
            // waves (block blk belongs to wave blk % KW, as own(j)).
            constexpr int kR = kAStage / 1024;
            const auto slot_of_wave = [&](int w) {
                return reinterpret_cast<float4_t *>(a_lds + (w * D + j) * kAStage);
            };
            float4_t *const mine = slot_of_wave(kw);
#pragma unroll
            for (int r = 0; r < kBlocks / kR; ++r) {
#pragma unroll
                for (int b = 0; b < NB; ++b)
#pragma unroll
                    for (int mb = 0; mb < MB; ++mb)
                        if ((b * MB + mb) / kR == r) mine[((b * MB + mb) % kR) * 64 + lane] = acc[b][mb];
                lds_barrier();
#pragma unroll
                for (int i = 0; i < kR / KW; ++i) {
                    const int at = (kw + i * KW) * 64 + lane;
                    float4_t s = slot_of_wave(0)[at];
#pragma unroll
                    for (int k2 = 1; k2 < KW; ++k2) s += slot_of_wave(k2)[at];
                    out[r * (kR / KW) + i] = s;
                }
                lds_barrier();
            }
        }
#pragma unroll
        for (int b = 0; b < NB; ++b)
#pragma unroll
            for (int mb = 0; mb < MB; ++mb) acc[b][mb] = zero4;
        if (cp_begin == 0 && cp_end == KU) {
            store_c(cp_c, out);
        } else if (cp_c == c_last) {
            has_last = true;
#pragma unroll
            for (int j = 0; j < kOwn; ++j) last_out[j] = out[j];
        } else {
            has_first = true;
#pragma unroll
            for (int j = 0; j < kOwn; ++j)
                if (own(j) < kBlocks) store_partial(my_slots, own(j), lane, out[j]);
        }
    };

    // Stage st in ring slot j, with `later` stages issued after it: compute,
    // and close the tile segment at its end.
    auto step = [&](int j, int st, int later) {
        if (st < n_st) {
            if (cp_ku + kw < cp_end) compute(j, later);
            if (cp_ku + KW >= cp_end) {
                // four row blocks: the last segment is closed after the loop,
                // so that no sum is held across it
                if (!kRingRed || cp_c != c_last) {
                    finish_segment(j);
                    cp_c += 1;
                    cp_ku = 0;
                    cp_begin = 0;
                    cp_end = (cp_c < c_last) ? KU : k1;
                }
            } else {
                cp_ku += KW;
            }
        }
    };
    // Groups of D stages.  Every group but the last refills each slot after
    // computing it; loads are issued unconditionally (past the range through
    // empty descriptors) so that every stage has the same load pattern and
    // the vmcnt waits stay static.  The last group issues nothing: its slot j
    // waits with only the D-1-j stages issued after it behind it.
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
    if constexpr (kRingRed) {
        // Stages past the range were issued (through empty descriptors) but
        // never waited for: drain them before the ring is reused.
        wait_vmcnt<0>();
        finish_segment(0);
    }

    // ---- combination of shared tiles ----
    auto own_slot = [&](int j) { return own(j) < kBlocks ? own(j) : -1; };
    combine_tiles<kOwn>(p, flags, wg, grid, slot_floats, lane, has_first, c_first, has_last, c_last, last_out,
                        own_slot, store_c);
}

template <int MB, int NB, int D, int AR, int KW, bool PER_CHANNEL>
__global__ void __launch_bounds__(64 * KW, 1) w4a16_stream_kernel(GemmProblem p)
{
    stream_body<MB, NB, D, AR, KW, PER_CHANNEL, false>(p);
}

template <int MB, int NB, int D, int AR, int KW, bool PER_CHANNEL>
__global__ void __launch_bounds__(64 * KW, 1) w4a16_sparse_kernel(GemmProblem p)
{
    stream_body<MB, NB, D, AR, KW, PER_CHANNEL, true>(p);
}

}  // namespace

// Ring depth: stages in flight per wave (weights in registers: NB words of
// 16 bytes per lane per stage, so narrow tiles afford deep rings).  Eight
// waves keep as many bytes in flight per work-group with half the depth
// (and half the LDS ring each).
template <int MB, int NB, int AR, int KW>
constexpr int stream_depth()
{
    if constexpr (MB == 1) {
        constexpr int d = NB == 8 ? 3 : NB == 4 ? 4 : NB == 2 ? 5 : 8;
        // (32-column tiles with eight waves measured 2-5% faster with two
        // stages than with three)
        return KW == 8 ? (NB == 2 ? 2 : (d + 1) / 2) : d;
    }
    // LDS ring of 32 rows: 8 KiB per wave-stage (eight waves: 16-column
    // tiles only, two stages, 128 KiB); of 64 rows: 16 KiB, two stages.
    // (64-column tiles measured 3-6% faster with two stages than with three
    // at 32..128 rows, 32-column tiles 1-2% with three than with four.)
    if constexpr (KW == 8 || MB == 4) return 2;
    return NB >= 4 ? 2 : 3;
}

// 2:4 sparse stages carry 3/4 of the dense bytes per column block (NB = 4:
// 3 KiB per wave, NB = 2: 1.5 KiB), in 3 or 2 loads; up to 16 rows the
// ring is deeper than the dense one so that as many bytes are in flight.
// Bounded by the vmcnt range at four activation loads per stage.
template <int MB, int NB, int AR, int KW>
constexpr int sparse_depth()
{
    if constexpr (MB == 1) {
        constexpr int d = NB == 4 ? 5 : NB == 2 ? 8 : 7;
        // eight waves: half as deep, and two stages with 32- and 64-column
        // tiles (3-4% faster than three on 8192 x 28672 at M = 1..16)
        return KW == 8 ? (NB >= 2 ? 2 : (d + 1) / 2) : d;
    }
    return stream_depth<MB, NB, AR, KW>();
}

template <int MB, int NB, int AR, int KW>
constexpr int ring_depth(bool sparse)
{
    return sparse ? sparse_depth<MB, NB, AR, KW>() : stream_depth<MB, NB, AR, KW>();
}

template <int MB, int NB, int AR, int KW>
hipError_t launch_stream(const GemmConfig &cfg, const GemmProblem &p, hipStream_t stream)
{
    constexpr int D = stream_depth<MB, NB, AR, KW>();
    constexpr int DS = sparse_depth<MB, NB, AR, KW>();
    GemmProblem arg = p;
    void *args[] = {&arg};
    const bool pc = p.group_units == 0;
    const void *fn = pc ? (const void *)&w4a16_stream_kernel<MB, NB, D, AR, KW, true>
                        : (const void *)&w4a16_stream_kernel<MB, NB, D, AR, KW, false>;
    if constexpr (NB <= 4 || (NB == 8 && MB == 2)) {  // 2:4: 128-column tiles with two row blocks only
        if (cfg.sparse)
            fn = pc ? (const void *)&w4a16_sparse_kernel<MB, NB, DS, AR, KW, true>
                    : (const void *)&w4a16_sparse_kernel<MB, NB, DS, AR, KW, false>;
    } else if (cfg.sparse) {
        return hipErrorInvalidValue;
    }
    return hipLaunchKernel(fn, dim3(cfg.grid), dim3(64 * KW), args, 0, stream);
}

void kernel_name(const GemmConfig &cfg, bool per_channel, char *buf, size_t n)
{
    if (cfg.kind == kKindTile) {
        tile_kernel_name(cfg, per_channel, buf, n);
        return;
    }
    if (cfg.kind == kKindWide) {
        wide_kernel_name(cfg, per_channel, buf, n);
        return;
    }
    if (cfg.mb == 4 && cfg.waves == 8) {
        pair_kernel_name(per_channel, buf, n);
        return;
    }
    int d = 0;
    switch (cfg.waves * 1000 + cfg.mb * 100 + cfg.nb * 10 + cfg.ar) {
    case 4111: d = ring_depth<1, 1, 1, 4>(cfg.sparse); break;
    case 4112: d = ring_depth<1, 1, 2, 4>(cfg.sparse); break;
    case 4114: d = ring_depth<1, 1, 4, 4>(cfg.sparse); break;
    case 4121: d = ring_depth<1, 2, 1, 4>(cfg.sparse); break;
    case 4122: d = ring_depth<1, 2, 2, 4>(cfg.sparse); break;
    case 4124: d = ring_depth<1, 2, 4, 4>(cfg.sparse); break;
    case 4141: d = ring_depth<1, 4, 1, 4>(cfg.sparse); break;
    case 4142: d = ring_depth<1, 4, 2, 4>(cfg.sparse); break;
    case 4144: d = ring_depth<1, 4, 4, 4>(cfg.sparse); break;
    case 4218: d = ring_depth<2, 1, 8, 4>(cfg.sparse); break;
    case 4228: d = ring_depth<2, 2, 8, 4>(cfg.sparse); break;
    case 4248: d = ring_depth<2, 4, 8, 4>(cfg.sparse); break;
    case 8111: d = ring_depth<1, 1, 1, 8>(cfg.sparse); break;
    case 8112: d = ring_depth<1, 1, 2, 8>(cfg.sparse); break;
    case 8114: d = ring_depth<1, 1, 4, 8>(cfg.sparse); break;
    case 8121: d = ring_depth<1, 2, 1, 8>(cfg.sparse); break;
    case 8122: d = ring_depth<1, 2, 2, 8>(cfg.sparse); break;
    case 8124: d = ring_depth<1, 2, 4, 8>(cfg.sparse); break;
    case 8141: d = ring_depth<1, 4, 1, 8>(cfg.sparse); break;
    case 8142: d = ring_depth<1, 4, 2, 8>(cfg.sparse); break;
    case 8144: d = ring_depth<1, 4, 4, 8>(cfg.sparse); break;
    case 8218: d = ring_depth<2, 1, 8, 8>(cfg.sparse); break;
    case 4181: d = ring_depth<1, 8, 1, 4>(cfg.sparse); break;
    case 4182: d = ring_depth<1, 8, 2, 4>(cfg.sparse); break;
    case 4184: d = ring_depth<1, 8, 4, 4>(cfg.sparse); break;
    case 4288: d = ring_depth<2, 8, 8, 4>(cfg.sparse); break;
    case 8181: d = ring_depth<1, 8, 1, 8>(cfg.sparse); break;
    case 8182: d = ring_depth<1, 8, 2, 8>(cfg.sparse); break;
    case 8184: d = ring_depth<1, 8, 4, 8>(cfg.sparse); break;
    case 4496: d = ring_depth<4, 8, 16, 4>(cfg.sparse); break;
    default: break;
    }
    if (d == 0) {
        if (n) buf[0] = 0;
        return;
    }
    snprintf(buf, n, "%s<%d, %d, %d, %d, %d, %s>", cfg.sparse ? "w4a16_sparse_kernel" : "w4a16_stream_kernel",
             cfg.mb, cfg.nb, d, cfg.ar, cfg.waves, per_channel ? "true" : "false");
}

hipError_t launch_gemm(const GemmConfig &cfg, const GemmProblem &p, hipStream_t stream)
{
    if (cfg.kind == kKindTile) return launch_tile_gemm(cfg, p, stream);
    if (cfg.kind == kKindWide) return launch_wide_gemm(cfg, p, stream);
    if (cfg.mb == 4 && cfg.waves == 8) return launch_pair_gemm(cfg, p, stream);
    switch (cfg.waves * 1000 + cfg.mb * 100 + cfg.nb * 10 + cfg.ar) {
    case 4111: return launch_stream<1, 1, 1, 4>(cfg, p, stream);
    case 4112: return launch_stream<1, 1, 2, 4>(cfg, p, stream);
    case 4114: return launch_stream<1, 1, 4, 4>(cfg, p, stream);
    case 4121: return launch_stream<1, 2, 1, 4>(cfg, p, stream);
    case 4122: return launch_stream<1, 2, 2, 4>(cfg, p, stream);
    case 4124: return launch_stream<1, 2, 4, 4>(cfg, p, stream);
    case 4141: return launch_stream<1, 4, 1, 4>(cfg, p, stream);
    case 4142: return launch_stream<1, 4, 2, 4>(cfg, p, stream);
    case 4144: return launch_stream<1, 4, 4, 4>(cfg, p, stream);
    case 4218: return launch_stream<2, 1, 8, 4>(cfg, p, stream);
    case 4228: return launch_stream<2, 2, 8, 4>(cfg, p, stream);
    case 4248: return launch_stream<2, 4, 8, 4>(cfg, p, stream);
    case 8111: return launch_stream<1, 1, 1, 8>(cfg, p, stream);
    case 8112: return launch_stream<1, 1, 2, 8>(cfg, p, stream);
    case 8114: return launch_stream<1, 1, 4, 8>(cfg, p, stream);
    case 8121: return launch_stream<1, 2, 1, 8>(cfg, p, stream);
    case 8122: return launch_stream<1, 2, 2, 8>(cfg, p, stream);
    case 8124: return launch_stream<1, 2, 4, 8>(cfg, p, stream);
    case 8141: return launch_stream<1, 4, 1, 8>(cfg, p, stream);
    case 8142: return launch_stream<1, 4, 2, 8>(cfg, p, stream);
    case 8144: return launch_stream<1, 4, 4, 8>(cfg, p, stream);
    case 8218: return launch_stream<2, 1, 8, 8>(cfg, p, stream);
    case 4181: return launch_stream<1, 8, 1, 4>(cfg, p, stream);
    case 4182: return launch_stream<1, 8, 2, 4>(cfg, p, stream);
    case 4184: return launch_stream<1, 8, 4, 4>(cfg, p, stream);
    case 4288: return launch_stream<2, 8, 8, 4>(cfg, p, stream);
    case 8181: return launch_stream<1, 8, 1, 8>(cfg, p, stream);
    case 8182: return launch_stream<1, 8, 2, 8>(cfg, p, stream);
    case 8184: return launch_stream<1, 8, 4, 8>(cfg, p, stream);
    case 4496: return launch_stream<4, 8, 16, 4>(cfg, p, stream);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace marlin
