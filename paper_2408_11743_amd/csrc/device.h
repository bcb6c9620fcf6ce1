// Device helpers shared by the GEMM kernels: vector types, wait and barrier
// primitives, the striped partition, and the combination of column tiles
// shared by several work-groups (Section 3.4, "Striped Partitioning").
#pragma once

#include <hip/hip_runtime.h>

#include "internal.h"

namespace marlin {
namespace dev {

typedef _Float16 half2_t __attribute__((ext_vector_type(2)));
typedef _Float16 half4_t __attribute__((ext_vector_type(4)));
typedef _Float16 half8_t __attribute__((ext_vector_type(8)));
typedef float float4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

constexpr int kAuxNonTemporal = 2;  // cache-policy bit: non-temporal (streamed once)
// Word 3 of a gfx9 buffer descriptor for raw (untyped) dword access.
constexpr int kBufferFlags = 0x00020000;

// s_waitcnt immediate for gfx9: vmcnt[3:0] | expcnt[6:4] | lgkmcnt[11:8] | vmcnt[5:4]<<14.
template <int V>
__device__ __forceinline__ void wait_vmcnt()
{
    static_assert(V >= 0 && V < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((V & 15) | (7 << 4) | (15 << 8) | ((V >> 4) << 14));
    asm volatile("" ::: "memory");
}

// wait_vmcnt<V> for a V known only after unrolling: the switch folds to
// one wait when n is a constant (a loop index of a fully unrolled loop).
__device__ __forceinline__ void wait_vmcnt_n(int n)
{
#define MARLIN_VMCNT_CASE(V) \
    case V:                  \
        wait_vmcnt<V>();     \
        break;
#define MARLIN_VMCNT_CASE8(V) MARLIN_VMCNT_CASE(V) MARLIN_VMCNT_CASE(V + 1) MARLIN_VMCNT_CASE(V + 2) \
    MARLIN_VMCNT_CASE(V + 3) MARLIN_VMCNT_CASE(V + 4) MARLIN_VMCNT_CASE(V + 5) MARLIN_VMCNT_CASE(V + 6) \
    MARLIN_VMCNT_CASE(V + 7)
    switch (n) {
        MARLIN_VMCNT_CASE8(0)
        MARLIN_VMCNT_CASE8(8)
        MARLIN_VMCNT_CASE8(16)
        MARLIN_VMCNT_CASE8(24)
        MARLIN_VMCNT_CASE8(32)
        MARLIN_VMCNT_CASE8(40)
        MARLIN_VMCNT_CASE8(48)
        MARLIN_VMCNT_CASE8(56)
    default:
        wait_vmcnt<0>();
        break;
    }
#undef MARLIN_VMCNT_CASE8
#undef MARLIN_VMCNT_CASE
}

// Wait until at most n LDS (and scalar-memory) operations are outstanding;
// n is clamped to the counter's range (a smaller n only waits longer).  The
// switch folds to one wait when n is a constant after unrolling.
__device__ __forceinline__ void wait_lgkmcnt_n(int n)
{
#define MARLIN_LGKM_CASE(V)                                                          \
    case V:                                                                          \
        __builtin_amdgcn_s_waitcnt(15 | (7 << 4) | ((V) << 8) | (3 << 14));         \
        break;
    switch (n < 0 ? 0 : n > 15 ? 15 : n) {
        MARLIN_LGKM_CASE(0) MARLIN_LGKM_CASE(1) MARLIN_LGKM_CASE(2) MARLIN_LGKM_CASE(3)
        MARLIN_LGKM_CASE(4) MARLIN_LGKM_CASE(5) MARLIN_LGKM_CASE(6) MARLIN_LGKM_CASE(7)
        MARLIN_LGKM_CASE(8) MARLIN_LGKM_CASE(9) MARLIN_LGKM_CASE(10) MARLIN_LGKM_CASE(11)
        MARLIN_LGKM_CASE(12) MARLIN_LGKM_CASE(13) MARLIN_LGKM_CASE(14)
    default:
        __builtin_amdgcn_s_waitcnt(15 | (7 << 4) | (15 << 8) | (3 << 14));
        break;
    }
#undef MARLIN_LGKM_CASE
    asm volatile("" ::: "memory");
}

__device__ __forceinline__ void wait_lgkmcnt0()
{
    __builtin_amdgcn_s_waitcnt(63 | (7 << 4) | (0 << 8) | (3 << 14));
    asm volatile("" ::: "memory");
}

// Keeps every memory operation and every instruction on its side: neither
// the IR passes (the memory clobber) nor the machine scheduler (the
// scheduling barrier) move loads across it.  The kernels wait for their
// direct-to-LDS loads by counting the vector-memory operations issued after
// them (they complete in order), which holds only if the loads are emitted in
// the order the code issues them; the compiler is otherwise free to
// interleave independent loads.
__device__ __forceinline__ void issue_order_point()
{
    asm volatile("" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
}

// Work-group barrier that does not wait for outstanding global loads.
__device__ __forceinline__ void lds_barrier()
{
    wait_lgkmcnt0();
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

__device__ __forceinline__ half2_t as_h2(uint32_t x) { return __builtin_bit_cast(half2_t, x); }
__device__ __forceinline__ uint32_t as_u32(half2_t x) { return __builtin_bit_cast(uint32_t, x); }

__device__ __forceinline__ float4_t mfma(half8_t w, half8_t a, float4_t c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(w, a, c, 0, 0, 0);
}

// Masks of the int4 -> fp16 conversion, made opaque once per kernel (an empty
// asm "redefines" them in vector registers) so that (x & m) | o selects the
// single v_and_or_b32 with register operands.
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
// order j = 0..7 (code j sits in nibble (j >> 1) + 4 (j & 1)), with the
// paper's magic number (Section 3.4, "Dequantization and Tensor Cores"): the
// code in the low mantissa bits of 1024.0 is 1024 + q, minus 1032 gives q - 8
// exactly; a code four bits up gives 1024 + 16q, and one fma (x/16 - 72)
// gives q - 8.
__device__ __forceinline__ half8_t dequant_magic(uint32_t x, const DequantConsts &k)
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

// Scale row of 128-row block ku: ku / group_units as one multiply-high with
// the host's rounded-up reciprocal 2^26 / group_units (exact for ku < 2^13).
__device__ __forceinline__ int scale_row_of(int ku, const GemmProblem &p)
{
    return (int)__umulhi((uint32_t)ku << 6, p.gmagic);
}

// Work-group index in the partition, arranged so that consecutive indices
// run on one XCD: the dispatcher hands work-group b to XCD b mod 8, so XCD x
// gets the indices [x*q + min(x, r), ...) for grid = 8q + r.  Consecutive
// ranges then share an L2 (the row groups of one column tile read the same
// weights, from one L2).
constexpr int kXcds = 8;
__device__ __forceinline__ int xcd_local_wg(int b, int grid)
{
    const int q = grid / kXcds, r = grid % kXcds;
    const int x = b % kXcds;
    return x * q + (x < r ? x : r) + b / kXcds;
}

// First unit of work-group w: gran * floor(w * (units / gran) / grid), from
// the host's quotient and remainder and its reciprocal of grid, so that no
// division is needed.  gran = KU hands out whole tiles; gran = 1 splits tiles
// (Stream-K).  grid is the launch's (the reciprocal was made for it).
__device__ __forceinline__ int range_start(const GemmProblem &p, int w, int grid)
{
    (void)grid;
    return (w * p.per_wg + (int)__umulhi((uint32_t)(w * p.extra), p.grid_magic)) * p.gran;
}

// Tile of unit u: u / KU, by the host's reciprocal where that is exact.
__device__ __forceinline__ int tile_of(const GemmProblem &p, int u)
{
    return p.ku_magic ? (int)__umulhi((uint32_t)u, p.ku_magic) : (int)((uint32_t)u / (uint32_t)p.KU);
}

// Work-group that owns unit u: the largest w with range_start(w) <= u
// (used only when tiles are split, gran = 1).
__device__ __forceinline__ int unit_owner(const GemmProblem &p, int u, int grid)
{
    return (int)((((int64_t)u + 1) * grid - 1) / p.units);
}

// ---- partial tiles in the workspace ----
// A work-group that covers a tile only in part writes its fp32 tile to one of
// its two workspace slots (0: its first tile, 1: its last), in
// structure-of-arrays order so every store instruction covers 256 contiguous
// bytes: float index ((blk*4 + i)*64 + lane).  Those bytes are written and
// read with relaxed agent-scope atomics, which the compiler emits as ordinary
// vector stores / loads carrying the device-coherence bit, so they bypass the
// per-XCD L2 non-coherence without a whole-cache writeback or invalidate.
// Ordering: a wave waits for its stores to complete (vmcnt 0) before the
// work-group barrier that precedes the arrival counter's atomic increment,
// and a reducer issues its loads only after it has read the counter.
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

// Combination at the end of a work-group's range.  The first tile (if shared
// and not also the last) was written to slot 0 when its segment ended; the
// last tile (if shared) is in registers (last_out) and is written to slot 1
// now.  The work-group then arrives at each shared tile's counter with an
// increment; whoever completes a count sums the contributors' slots in
// work-group order (bitwise reproducible; its own last tile from registers)
// and resets the counter.  No work-group waits for another.
//
// Arrival is not preceded by a look at the counter: with balanced ranges all
// contributors of a tile finish together, so the look almost never finds the
// count complete and would only add a device-coherent round trip.  A shared
// tile's counter is indexed by its first contributor (unique: a work-group
// that owns the first block of two tiles owns the whole first one) and has a
// 128-byte line of its own, so concurrent arrivals at different tiles do not
// queue on one cache line.
//   KOWN         tile blocks this wave holds;  own(j): slot block index of
//                block j, or -1 if the wave holds none there
//   store_c(c, out[KOWN])  writes tile c's C from full sums
template <int KOWN, typename OwnFn, typename StoreFn>
__device__ __forceinline__ void combine_tiles(const GemmProblem &p, int *flags, int wg, int grid,
                                              int slot_floats, int lane, bool has_first, int c_first,
                                              bool has_last, int c_last, const float4_t (&last_out)[KOWN],
                                              OwnFn own, StoreFn store_c)
{
    if (!has_first && !has_last) return;  // uniform across the work-group
    const int KU = p.KU;
    float *const my_slots = p.partials + (int64_t)wg * 2 * slot_floats;
    // Contributors of tile c: work-groups owner(c*KU) .. owner(c*KU + KU - 1);
    // the slot a contributor used for c: 1 if c is its last tile, else 0.
    auto slot_of = [&](int w, int c) -> const float * {
        const int w_last = tile_of(p, range_start(p, w + 1, grid) - 1);
        return p.partials + ((int64_t)w * 2 + (c == w_last ? 1 : 0)) * slot_floats;
    };
    auto others_of = [&](int c) { return unit_owner(p, c * KU + KU - 1, grid) - unit_owner(p, c * KU, grid); };
    auto counter_of = [&](int c) { return p.counters + kCounterStride * unit_owner(p, c * KU, grid); };
    if (has_last) {
#pragma unroll
        for (int j = 0; j < KOWN; ++j)
            if (own(j) >= 0) store_partial(my_slots + slot_floats, own(j), lane, last_out[j]);
    }
    wait_vmcnt<0>();  // this wave's slot stores are complete
    lds_barrier();
    if (threadIdx.x == 0) {
        int f0 = 0, f1 = 0;
        if (has_first) {
            uint32_t *const ctr = counter_of(c_first);
            if (__hip_atomic_fetch_add(ctr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
                (uint32_t)others_of(c_first)) {
                f0 = 1;
                __hip_atomic_store(ctr, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
        }
        if (has_last) {
            uint32_t *const ctr = counter_of(c_last);
            if (__hip_atomic_fetch_add(ctr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
                (uint32_t)others_of(c_last)) {
                f1 = 1;
                __hip_atomic_store(ctr, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
        }
        flags[0] = f0;
        flags[1] = f1;
    }
    lds_barrier();
    const bool reduce_first = has_first && flags[0] != 0;
    const bool reduce_last = has_last && flags[1] != 0;
    // Sum the contributors' slots in work-group order; this work-group's own
    // last-tile sum comes from registers (the same values it would store).
    // The slots of up to kBatch contributors are loaded before they are added
    // (past the last contributor the last one is reloaded and ignored), so
    // their round trips overlap.
    constexpr int kBatch = KOWN >= 4 ? 1 : 4 / KOWN;
    auto reduce = [&](int c, bool own_in_regs) {
        const int wf = unit_owner(p, c * KU, grid);
        const int wl = unit_owner(p, c * KU + KU - 1, grid);
        float4_t out[KOWN];
        for (int w0 = wf; w0 <= wl; w0 += kBatch) {
            float4_t v[kBatch][KOWN];
#pragma unroll
            for (int b = 0; b < kBatch; ++b) {
                const int w = w0 + b <= wl ? w0 + b : wl;
                const float *slot = slot_of(w, c);
#pragma unroll
                for (int j = 0; j < KOWN; ++j) {
                    const int blk = own(j) >= 0 ? own(j) : 0;
                    v[b][j] = (own_in_regs && w == wg) ? last_out[j] : load_partial(slot, blk, lane);
                }
            }
#pragma unroll
            for (int b = 0; b < kBatch; ++b) {
                if (w0 + b > wl) break;
#pragma unroll
                for (int j = 0; j < KOWN; ++j) out[j] = (w0 + b == wf) ? v[b][j] : out[j] + v[b][j];
            }
        }
        store_c(c, out);
    };
    if (reduce_last) reduce(c_last, true);
    if (reduce_first) reduce(c_first, false);
}

}  // namespace dev
}  // namespace marlin
