// Internal declarations shared by the host API and the kernel launchers.
// Not part of the public ABI (include/marlin.h is).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace marlin {

// One launch configuration of the GEMM kernel.
//   mb   : 16-row blocks of A per row group (1 or 2)
//   rg   : row groups of 32 rows (M > 32), each a separate set of tiles
//   nb   : 16-column blocks per column tile (1, 2 or 4)
//   ar   : 0, or (mb <= 2) the activation rows arrive in LDS, 4 * ar of them
//   whole: work-groups own whole column tiles (else 128-row blocks: Stream-K)
//   grid : work-groups
//   waves: stream kernel waves per work-group (they split K): 4, or 8 (two per
//          SIMD) with one 16-row block or one 16-column block
constexpr int kStreamOcc = 1;    // work-groups per compute unit

constexpr int kKindStream = 0;  // w4a16_stream_kernel (any M; row groups of 32)
constexpr int kKindTile = 1;    // w4a16_tile_kernel (activation tile shared by the waves)

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
    return c.kind == kKindTile ? (c.tile_nw / c.tile_wm) * 16 * c.nb : 16 * c.nb;
}
inline int tile_rows(const GemmConfig &c) { return c.kind == kKindTile ? c.tile_wm * 16 * c.mb : 16 * c.mb; }

struct GemmProblem {
    const uint16_t *A;
    const uint32_t *W;
    const uint16_t *S;
    uint16_t *C;
    float *partials;      // fp32 partial tiles, 2 slots per work-group
    uint32_t *counters;   // arrival counters: one per shared tile, kCounterStride words apart
    int M;                // rows in this pass (1 .. 32 * rg)
    int rg;               // row groups (tiles = column tiles * rg)
    int N;
    int K;
    int G;                // scale rows
    int KU;               // 128-row blocks of K
    int units;            // column tiles * KU: 128-row blocks of all column tiles
    int gran;             // units per partition item: KU (whole tiles) or 1
    int per_wg;           // (units / gran) / grid
    int extra;            // (units / gran) % grid
    int group_units;      // 128-row blocks per scale group; 0 = per-channel
    uint32_t gmagic;      // ceil(2^26 / group_units): row of block ku = (ku * 2^6 * gmagic) >> 32
    uint32_t grid_magic;  // ceil(2^32 / grid) (0 for grid 1): w * extra / grid = mulhi(w * extra, grid_magic)
    uint32_t ku_magic;    // ceil(2^32 / KU) where u / KU = mulhi(u, ku_magic) for every unit u, else 0
};

// ceil(2^32 / d) for 2 <= d: with it, floor(n / d) = floor(n * m / 2^32) for
// every n with n * d <= 2^32 (m = (2^32 + e) / d, 0 <= e < d, so the error
// n * e / (d 2^32) stays below 1/d).  0 when d < 2.
inline uint32_t reciprocal32(uint64_t d)
{
    return d < 2 ? 0u : (uint32_t)((((uint64_t)1 << 32) + d - 1) / d);
}

// Upper bound on compute units used (MI355X has 256).  Workspace sizes are
// computed with this bound, never with the device's.
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

// Device facts cached per device.
int device_cu_count(int device);

GemmConfig choose_config(int M, int N, int K, int group_units, int grid_cap, bool sparse = false);
size_t workspace_bytes_for(const GemmConfig &cfg, int N);

hipError_t launch_gemm(const GemmConfig &cfg, const GemmProblem &p, hipStream_t stream);
// Name of the kernel instantiation launch_gemm runs for cfg ("" if none).
void kernel_name(const GemmConfig &cfg, bool per_channel, char *buf, size_t n);
hipError_t launch_tile_gemm(const GemmConfig &cfg, const GemmProblem &p, hipStream_t stream);
void tile_kernel_name(const GemmConfig &cfg, bool per_channel, char *buf, size_t n);
bool tile_config_supported(int nw, int wm, int mbw, int nbw, int ks);

hipError_t launch_pack(const uint8_t *q, const uint16_t *s, int K, int N, int G,
                       uint32_t *w_packed, uint16_t *s_packed, hipStream_t stream);
hipError_t launch_unpack(const uint32_t *w_packed, const uint16_t *s_packed, int K, int N,
                         int G, uint8_t *q, uint16_t *s, hipStream_t stream);
hipError_t launch_pack_sparse(const uint8_t *q, const uint16_t *s, int K, int N, int G, uint32_t *w_packed,
                              uint16_t *s_packed, hipStream_t stream);
hipError_t launch_unpack_sparse(const uint32_t *w_packed, const uint16_t *s_packed, int K, int N, int G,
                                uint8_t *q, uint16_t *s, hipStream_t stream);

}  // namespace marlin
