// Launch planning of the GEMM: the kernel, tile shape and striped partition
// a call runs with, and the workspace it needs (Section 3.4, "Striped
// Partitioning").  Pure host C++ (no HIP types), so the planner can be built
// and checked on any machine.  Not part of the public ABI (include/marlin.h
// is).
#pragma once

#include <stddef.h>
#include <stdint.h>

namespace marlin {

constexpr int kStreamOcc = 1;  // stream kernel work-groups per compute unit

constexpr int kKindStream = 0;  // w4a16_stream_kernel (any M; row groups of 32)
constexpr int kKindTile = 1;    // w4a16_tile_kernel (activation tile shared by the waves)
constexpr int kKindWide = 2;    // w4a16_wide_kernel (four waves along N, weights in registers)

// One launch configuration of the GEMM kernel.
//   mb   : 16-row blocks of A per row group (1, 2, or 4: 128-column dense tiles
//          with four waves, or eight in the pair kernel)
//   rg   : row groups of 16 * mb rows, each a separate set of tiles
//   nb   : 16-column blocks per column tile (1, 2, 4 or 8)
//   ar   : 0 (tile and wide kernels), or the activation rows that arrive in
//          LDS per row group, 4 * ar of them
//   whole: work-groups own whole column tiles (else 128-row blocks: Stream-K)
//   grid : work-groups
//   waves: stream kernel waves per work-group (they split K): 4, or 8 (two per
//          SIMD) with one 16-row block, one 16-column block, or four row
//          blocks (the pair kernel, pair.hip)
struct GemmConfig {
    int kind;
    int mb;
    int nb;
    int ar;
    int rg;
    int whole;
    int grid;
    int tile_wm;  // tile kernel: waves along M (1: 4x1 waves; 2: 2x2 waves); mb, nb: row and
                  // column blocks per wave
    int sparse;   // 2:4 sparse weights (stream kernel only)
    int tile_ks;  // tile kernel: 128-row blocks of K per work-group stage
    int tile_nw;  // tile kernel: waves per work-group (4 or 8)
    int waves;    // stream kernel: waves per work-group (4 or 8)
};

// Columns and rows of one tile of a configuration.
inline int tile_cols(const GemmConfig &c)
{
    return c.kind == kKindTile ? (c.tile_nw / c.tile_wm) * 16 * c.nb : c.kind == kKindWide ? 64 * c.nb : 16 * c.nb;
}
inline int tile_rows(const GemmConfig &c) { return c.kind == kKindTile ? c.tile_wm * 16 * c.mb : 16 * c.mb; }

// ceil(2^32 / d) for 2 <= d: with it, floor(n / d) = floor(n * m / 2^32) for
// every n with n * d <= 2^32 (m = (2^32 + e) / d, 0 <= e < d, so the error
// n * e / (d 2^32) stays below 1/d).  0 when d < 2.
inline uint32_t reciprocal32(uint64_t d)
{
    return d < 2 ? 0u : (uint32_t)((((uint64_t)1 << 32) + d - 1) / d);
}

// Upper bound on compute units used (MI355X has 256).  marlin_workspace_bytes
// sizes for this bound, never for the device's count.
constexpr int kMaxCus = 256;
constexpr int kMaxPerCu = 2;  // work-groups per compute unit, at most
// Arrival counters at the start of every workspace.  A shared tile's counter
// is indexed by the tile's first contributor (a work-group index, below
// kMaxCus * kMaxPerCu) and sits kCounterStride words (one 128-byte line)
// from the next.  The region keeps its size of 1 MiB (it held one counter
// per tile of the finest tiling of the largest N before) so that the
// workspace layout, and a caller's once-zeroed workspace, stay valid.
constexpr int kCounterStride = 32;
constexpr size_t kCounterRegionBytes = ((size_t)1 << 20) / 16 * 4 * 4;
static_assert((size_t)kMaxCus * kMaxPerCu * kCounterStride * 4 <= kCounterRegionBytes, "counter region");

// Rows of A per launch.  A launch covers ceil(rows / 32) row groups of the
// stream kernel, or one row group per tile height of the tile kernel, each a
// copy of the weight matrix's tiles in the striped partition (the weights
// replicated virtually, one copy per segment of A: Section 3.4, Striped
// Partitioning); the copies read the same weights, mostly through L2.  With
// K * N < 2^32, the units of a launch (N / 16 column blocks times K / 128
// weight blocks, below 2^21, times at most 128 row groups) stay below 2^28,
// so every unit index fits in 32 bits; larger M runs as several launches.
constexpr int kPassRows = 4096;

// Tile-kernel instantiations (waves, waves along M, 16-row blocks per wave,
// 16-column blocks per wave, 128-row blocks per stage), encoded as
// nw*10000 + wm*1000 + mbw*100 + nbw*10 + ks.  tile.hip instantiates exactly
// these (its launch switch has one case per entry).
constexpr int kTileConfigs[] = {41441, 42441, 82441, 82241, 41142, 41124, 41222, 41214};
inline bool tile_config_supported(int nw, int wm, int mbw, int nbw, int ks)
{
    const int code = nw * 10000 + wm * 1000 + mbw * 100 + nbw * 10 + ks;
    for (int c : kTileConfigs)
        if (c == code) return true;
    return false;
}

// Tuning and test override of the configuration (the cost model is the
// default): MARLIN_FORCE_CONFIG="nb=<1|2|4|8>,grid=<n>,whole=<0|1>,
// kind=<stream|tile|wide>,waves=<4|8>,nw=<4|8>,ks=<1|2|4>,mb=<1|2|4>" forces
// the column-tile width, the work-group count, the partition, the kernel, the
// stream kernel's waves per work-group, the tile kernel's waves and blocks
// per stage and the stream kernel's 16-row blocks per row group, where the
// shape allows it (mb = 4: dense weights; mb = 1 and 2 follow from M).
// Fields left out are free (0, or -1 for whole/kind).
struct Override {
    int nb = 0;
    int grid = 0;
    int whole = -1;
    int kind = -1;
    int ks = 0;
    int nw = 0;
    int waves = 0;
    int mb = 0;
    bool operator==(const Override &o) const
    {
        return nb == o.nb && grid == o.grid && whole == o.whole && kind == o.kind && ks == o.ks && nw == o.nw &&
               waves == o.waves && mb == o.mb;
    }
};
Override parse_override(const char *spec);  // NULL: no override
// The override in effect for this call: the environment variable, read at
// every call (a process may change it between calls) and parsed again only
// when its text changes.
Override current_override();

// Words of one fp32 partial slot of a configuration (two slots per work-group).
int slot_floats(const GemmConfig &cfg);
// Workspace bytes a launch of cfg may touch: the counter region plus two
// partial slots per work-group (whole-tile partitions touch neither, but are
// sized the same way, so that the size is a function of the shape alone).
size_t workspace_bytes_for(const GemmConfig &cfg);
// Bytes a launch of cfg actually uses: 0 for whole tiles (no tile is shared,
// so neither counters nor slots are touched), else workspace_bytes_for(cfg).
size_t workspace_bytes_used(const GemmConfig &cfg);

// Cost-model choice for one pass of M rows (1..kPassRows) on `cus` compute
// units.  partial_budget: bytes available for a Stream-K split's counters and
// partial slots (SIZE_MAX: unlimited); configurations that would need more
// are planned with whole tiles only.
GemmConfig choose_config(int M, int N, int K, int group_units, int cus, bool sparse, const Override &ov,
                         size_t partial_budget);

// The configuration of one launch of a call: choose_config for the device's
// compute units, unless that needs more than workspace_bytes, in which case
// the best configuration that fits.  Memoised per (shape, device compute
// units, sparse, override, workspace class), so a repeated call costs a table
// lookup.
GemmConfig plan_pass(int M, int N, int K, int group_units, int cus, bool sparse, size_t workspace_bytes,
                     const Override &ov);

// Workspace that any M-row call (dense or 2:4 sparse, every launch of it)
// needs on a device of up to kMaxCus compute units under the override ov.
// Memoised.
size_t required_workspace(int64_t M, int N, int K, int group_units, const Override &ov);

}  // namespace marlin
