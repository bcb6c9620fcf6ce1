// Host side of the C ABI declared in include/marlin.h: argument checks (all
// before any HIP call), launch configuration, workspace sizing and launches.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>

#include "marlin.h"
#include "internal.h"
#include "quant.h"

namespace marlin {

namespace {
constexpr int kMaxDevices = 64;
std::atomic<int> g_cu_count[kMaxDevices];
std::mutex g_cu_mutex;

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// 0 = invalid; otherwise the number of scale rows G.
int64_t scale_rows(int64_t K, int64_t group)
{
    if (group == -1 || group == K) return 1;
    if (group <= 0 || group % 128 != 0 || K % group != 0) return 0;
    return K / group;
}

bool shape_ok(int64_t K, int64_t N)
{
    return K >= 128 && N >= 64 && K % 128 == 0 && N % 64 == 0 && K <= (1 << 20) && N <= (1 << 20) &&
           (uint64_t)K * (uint64_t)N < ((uint64_t)1 << 32);
}

marlin_status_t check_weights(int64_t K, int64_t N, int64_t group)
{
    if (!shape_ok(K, N)) return MARLIN_ERR_INVALID_SHAPE;
    if (scale_rows(K, group) == 0) return MARLIN_ERR_UNSUPPORTED_GROUP;
    return MARLIN_OK;
}
}  // namespace

int device_cu_count(int device)
{
    if (device < 0 || device >= kMaxDevices) return 0;
    int v = g_cu_count[device].load(std::memory_order_acquire);
    if (v > 0) return v;
    std::lock_guard<std::mutex> lock(g_cu_mutex);
    v = g_cu_count[device].load(std::memory_order_relaxed);
    if (v > 0) return v;
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device) != hipSuccess ||
        cus <= 0)
        return 0;
    g_cu_count[device].store(cus, std::memory_order_release);
    return cus;
}

// Tuning and test override, read at every call (a process may change it
// between calls):
// MARLIN_FORCE_CONFIG="nb=<1|2|4>,grid=<n>,whole=<0|1>,kind=<stream|tile>,
// waves=<4|8>,nw=<4|8>,ks=<1|2|4>" forces the column-tile width, the
// work-group count, the partition, the kernel, the stream kernel's waves per
// work-group and the tile kernel's waves and blocks per stage where the shape
// allows it (the cost model below is the default).
struct ForcedConfig {
    int nb = 0;
    int grid = 0;
    int whole = -1;
    int kind = -1;
    int ks = 0;
    int nw = 0;
    int waves = 0;
};

static ForcedConfig read_forced()
{
    ForcedConfig f;
    const char *e = getenv("MARLIN_FORCE_CONFIG");
    if (!e) return f;
    const char *q = strstr(e, "nb=");
    if (q) f.nb = atoi(q + 3);
    q = strstr(e, "grid=");
    if (q) f.grid = atoi(q + 5);
    q = strstr(e, "whole=");
    if (q) f.whole = atoi(q + 6) ? 1 : 0;
    if (strstr(e, "kind=stream")) f.kind = kKindStream;
    if (strstr(e, "kind=tile")) f.kind = kKindTile;
    q = strstr(e, "ks=");
    if (q) f.ks = atoi(q + 3);
    q = strstr(e, "nw=");
    if (q) f.nw = atoi(q + 3);
    q = strstr(e, "waves=");
    if (q) f.waves = atoi(q + 6);
    if (f.waves != 4 && f.waves != 8) f.waves = 0;
    if (f.nb != 1 && f.nb != 2 && f.nb != 4) f.nb = 0;
    if (f.grid < 0) f.grid = 0;
    return f;
}

// Read at every call, so that a process can change it between calls.
static ForcedConfig forced() { return read_forced(); }

// Configuration by rows of A per pass (at most 128): mb = 1 (M <= 16) or 2
// 16-row blocks per row group; beyond 32 rows the pass is split into row
// groups of 32 that are tiles of their own (a tile is a column tile of one
// row group); 4 * ar activation rows per group arrive in LDS; 4 or (one
// row block, or one column block) 8 waves split K, kStreamOcc work-groups
// per CU.
//
// Column tile width (nb 16-column blocks), waves and partition come from a
// cost model fitted to MI355X measurements (218 whole-tile timings over the
// Llama-7B and 70B layer shapes, 4% rms): a fixed cost per launch, plus the
// larger of the busiest work-group's weight bytes over its streaming rate
// (which depends on the tile width, the rows of A and the waves: narrow tiles
// and more rows cost more instructions per weight byte) and the layer's
// weight bytes over the chip's sustained rate.  Whole tiles per work-group
// cost ceil(tiles / grid) tiles (idle CUs allowed); Stream-K costs the
// average share plus the combination of shared tiles at the end
// (device-coherent round trips, longer with larger partial tiles).
// cus bounds the compute units used (the device's when launching, kMaxCus when
// sizing the workspace, so that the size does not depend on the device).
namespace {
// Tile kernel: time of one 128-row block of a tile, and the cost of
// combining shared tiles (fixed part, and per contributor: the reducer reads
// one fp32 slot per contributor), fitted to MI355X measurements.
struct TileCost {
    double unit_us, tail_us, tail_per_contributor_us;
};
TileCost tile_cost(int nw, int wm, int mbw, int nbw)
{
    if (nw == 8) return mbw == 4 ? TileCost{2.2, 12.0, 1.5}   // 256 x 128 tiles, 128 KiB slots
                                 : TileCost{1.35, 10.0, 1.0};  // 256 x 64, 64 KiB slots
    if (mbw == 4) return {wm == 2 ? 1.55 : 1.50, 10.4, 1.36};  // 64 KiB slots
    // up to 32 rows (several 128-row blocks per stage): time per unit of
    // 4 KiB * nbw of weights, measured with whole tiles on 8192 x 28672
    const double per4k = mbw == 1 ? (nbw == 4 ? 0.195 : 0.23) : (nbw == 2 ? 0.275 : 0.355);
    return {per4k * nbw, 7.0, 0.5};
}
// Fixed cost of a launch (dispatch, prologue, epilogue), the sustained weight
// stream of the whole chip, and the stream kernel's combination of a shared
// tile: 3 us with fp32 partial tiles up to 4 KiB per work-group, 4.5 us with
// 8 KiB, plus 0.45 us per contributor beyond four (ranges of a few blocks,
// as on tensor-parallel shards of a layer, give a dozen contributors per
// tile; fitted to 192 Stream-K timings on layer shapes and such shards).
constexpr double kFixedUs = 4.0;
constexpr double kChipBytesPerUs = 7.0e6;
double stream_tail_us(int slot_kib) { return slot_kib > 4 ? 4.5 : 3.0; }
constexpr double kStreamFreeContributors = 4.0;
constexpr double kStreamTailPerExtraContributorUs = 0.45;

// Bytes of weights per microsecond one work-group streams, by rows of A,
// nb = 4, 2, 1 and waves per work-group (measured; the activation rows arrive
// in LDS in every class).
double wg_rate(int mb, int ar, int nb, int waves)
{
    static const double r4[4][3] = {
        {31.8e3, 22.3e3, 13.3e3},  // M <= 4
        {32.5e3, 20.8e3, 13.0e3},  // M <= 8
        {25.2e3, 16.6e3, 10.7e3},  // M <= 16
        {17.6e3, 11.6e3, 7.1e3},   // M <= 32 (also each row group of 32 for larger M)
    };
    static const double r8[3][3] = {
        {38.8e3, 34.2e3, 20.2e3},  // M <= 4
        {32.7e3, 22.1e3, 15.6e3},  // M <= 8
        {26.0e3, 16.4e3, 11.0e3},  // M <= 16
    };
    const int row = (mb == 1) ? (ar == 1 ? 0 : ar == 2 ? 1 : 2) : 3;
    const int col = (nb == 4) ? 0 : (nb == 2) ? 1 : 2;
    if (waves == 8) return row < 3 ? r8[row][col] : (nb == 1 ? 7.4e3 : 0.0);
    return r4[row][col];
}
}  // namespace

namespace {
// Best partition of `tiles` tiles of KU units each over at most `grid`
// work-groups, given the time of one unit: whole tiles per work-group, or a
// Stream-K split that pays for combining shared tiles at the end (tail_us,
// plus tail_per_contributor_us per contributor of a shared tile, plus
// tail_per_extra_contributor_us per contributor beyond free_contributors).  Every
// launch costs kFixedUs, and no partition streams faster than floor_us.
struct Partition {
    double t;
    int whole;
    int64_t grid;
};

Partition best_partition(int64_t tiles, int KU, int64_t grid, double unit_us, double tail_us,
                         double tail_per_contributor_us, double floor_us, double free_contributors = 0.0,
                         double tail_per_extra_contributor_us = 0.0)
{
    Partition best{1e30, 0, 1};
    if (forced().whole != 0) {
        const int64_t g = tiles < grid ? tiles : grid;
        const double stream = (double)((tiles + g - 1) / g) * KU * unit_us;
        const double t = kFixedUs + (stream > floor_us ? stream : floor_us);
        if (t < best.t) best = {t, 1, g};
    }
    if (forced().whole != 1) {
        const int64_t units = tiles * KU;
        const int64_t g = grid < units ? grid : units;
        const double per = (double)units / (double)g;  // units per work-group
        const bool split = (units % g) != 0 || (units / g) % KU != 0;
        const double contributors = split ? 1.0 + (double)KU / per : 1.0;
        const double extra = contributors > free_contributors ? contributors - free_contributors : 0.0;
        const double tail = split ? tail_us + tail_per_contributor_us * contributors +
                                        tail_per_extra_contributor_us * extra
                                  : 0.0;
        const double stream = per * unit_us;
        const double t = kFixedUs + (stream > floor_us ? stream : floor_us) + tail;
        if (t < best.t) best = {t, 0, g};
    }
    return best;
}
}  // namespace

GemmConfig choose_config(int M, int N, int K, int group_units, int cus, bool sparse)
{
    (void)group_units;
    GemmConfig cfg;
    const int KU = K / 128;
    const int tiles16 = N / 16;
    const int ncu = cus < kMaxCus ? cus : kMaxCus;
    int64_t grid = (int64_t)ncu * kStreamOcc;
    if (forced().grid) grid = forced().grid;
    if (grid > (int64_t)kMaxCus * kMaxPerCu) grid = (int64_t)kMaxCus * kMaxPerCu;

    // stream kernel
    cfg.kind = kKindStream;
    cfg.tile_wm = 0;
    cfg.tile_ks = 0;
    cfg.tile_nw = 0;
    cfg.waves = 4;
    cfg.sparse = sparse ? 1 : 0;
    cfg.mb = (M <= 16) ? 1 : 2;
    cfg.ar = (M <= 4) ? 1 : (M <= 8) ? 2 : (M <= 16) ? 4 : 8;
    cfg.rg = (M + 31) / 32;  // row groups of 32 beyond M = 32, each a copy of the column tiles
    if (cfg.rg < 1) cfg.rg = 1;
    double best = 1e30;
    cfg.nb = 0;
    cfg.whole = 0;
    int64_t best_grid = grid;
    if (forced().kind != kKindTile) {
        // eight waves exist for one 16-row block, or two with one 16-column
        // block; an override to eight applies where they do
        const int forced_waves =
            (forced().waves == 8 && cfg.mb != 1 && forced().nb > 1) ? 4 : forced().waves;
        for (int waves = 8; waves >= 4; waves -= 4) {
            if (forced_waves && waves != forced_waves) continue;
            for (int nb = 4; nb >= 1; nb >>= 1) {
                const double rate = wg_rate(cfg.mb, cfg.ar, nb, waves);
                if (tiles16 % nb != 0 || rate <= 0.0) continue;
                if (forced().nb && nb != forced().nb) continue;
                const int64_t tiles = (int64_t)(tiles16 / nb) * cfg.rg;
                // sparse units carry 3/4 of the dense bytes (codes and row indices)
                const double unit_bytes = (double)nb * (sparse ? 768.0 : 1024.0);
                const double layer_bytes = (double)KU * (double)(tiles16 / nb) * unit_bytes;
                // fp32 partial tile: 16 x 16 x 4 bytes per block
                const Partition pt = best_partition(tiles, KU, grid, unit_bytes / rate,
                                                    stream_tail_us(nb * cfg.mb), 0.0,
                                                    layer_bytes / kChipBytesPerUs, kStreamFreeContributors,
                                                    kStreamTailPerExtraContributorUs);
                if (pt.t < best) {
                    best = pt.t;
                    cfg.nb = nb;
                    cfg.waves = waves;
                    cfg.whole = pt.whole;
                    best_grid = pt.grid;
                }
            }
        }
    }
    // tile kernel: the activation tile is shared by the waves of a
    // work-group.  Beyond 32 rows each wave owns 64 x 64 outputs (four waves:
    // 2x2 beyond 64 rows, else 4x1; eight waves, two per SIMD: 4x2), one
    // 128-row block per stage; up to 32 rows, 4x1 waves of 16 or 32 rows over
    // 2 or 4 blocks per stage (measured to win only where whole 128-column
    // tiles fill the chip at 17..32 rows, e.g. N = 28672).
    if (!sparse && forced().kind != kKindStream) {
        for (int nw = 8; nw >= 4; nw -= 4) {
            if (forced().nw && nw != forced().nw) continue;
            // rows per tile: 64*wm with 64-row waves; eight waves at 33..64
            // rows use 4x2 waves of 32 rows
            const int wm = (M > 64 || (nw == 8 && M > 32)) ? 2 : 1;
            const int mbw = (nw == 8 && M > 32 && M <= 64) ? 2 : M > 32 ? 4 : M > 16 ? 2 : 1;
            for (int nbw = 4; nbw >= 1; nbw >>= 1) {
                for (int ks = 4; ks >= 1; ks >>= 1) {
                    if (!tile_config_supported(nw, wm, mbw, nbw, ks)) continue;
                    if (forced().nb && nbw != forced().nb) continue;
                    if (forced().ks && ks != forced().ks) continue;
                    const int cols = (nw / wm) * 16 * nbw, rows = wm * 16 * mbw;
                    if (N % cols != 0) continue;
                    const int64_t tiles = (int64_t)(N / cols) * ((M + rows - 1) / rows);
                    const TileCost tc = tile_cost(nw, wm, mbw, nbw);
                    const Partition pt =
                        best_partition(tiles, KU, grid, tc.unit_us, tc.tail_us, tc.tail_per_contributor_us, 0.0);
                    if (pt.t < best) {
                        best = pt.t;
                        cfg.kind = kKindTile;
                        cfg.tile_nw = nw;
                        cfg.waves = 0;
                        cfg.tile_wm = wm;
                        cfg.tile_ks = ks;
                        cfg.nb = nbw;
                        cfg.mb = mbw;
                        cfg.ar = 0;
                        cfg.rg = (M + rows - 1) / rows;
                        cfg.whole = pt.whole;
                        best_grid = pt.grid;
                    }
                }
            }
        }
    }
    if (cfg.nb == 0) {  // only when an override excludes every choice (or asks for the tile kernel, sparse)
        cfg.kind = kKindStream;
        cfg.waves = 4;
        cfg.nb = (tiles16 % 2 == 0) ? 2 : 1;
        cfg.whole = 0;
        const int64_t units = (int64_t)(tiles16 / cfg.nb) * cfg.rg * KU;
        best_grid = grid < units ? grid : units;
    }
    if (best_grid < 1) best_grid = 1;
    cfg.grid = (int)best_grid;
    return cfg;
}

int slot_floats(const GemmConfig &cfg);

// The workspace starts with a fixed 1 MiB region of arrival counters (one
// per shared tile, on its own 128-byte line).  It never moves, whatever the
// shape, so any sequence of calls on one workspace finds every counter it
// uses at zero; the fp32 partial slots follow it.
size_t workspace_bytes_for(const GemmConfig &cfg, int N)
{
    (void)N;
    return kCounterRegionBytes + (size_t)cfg.grid * 2 * (size_t)slot_floats(cfg) * sizeof(float);
}

namespace {
// Largest workspace over the passes of at most kPassRows rows that an M-row
// call makes, dense or 2:4 sparse (one size serves both entry points).
size_t required_workspace(int64_t M, int N, int K, int gu)
{
    const int m_first = M < kPassRows ? (int)M : kPassRows;
    const int m_last = (int)(M % kPassRows);
    size_t need = 0;
    for (int sp = 0; sp < 2; ++sp) {
        size_t b = workspace_bytes_for(choose_config(m_first, N, K, gu, kMaxCus, sp != 0), N);
        if (b > need) need = b;
        if (M > kPassRows && m_last != 0) {
            b = workspace_bytes_for(choose_config(m_last, N, K, gu, kMaxCus, sp != 0), N);
            if (b > need) need = b;
        }
    }
    return need;
}
}  // namespace

}  // namespace marlin

using namespace marlin;

namespace {
marlin_status_t gemm_impl(const uint16_t *A, const void *w_packed, const void *s_packed, uint16_t *C,
                          void *workspace, size_t workspace_bytes, int64_t M, int64_t N, int64_t K,
                          int64_t group, hipStream_t stream, bool sparse)
{
    if (M < 0 || M > (1 << 24)) return MARLIN_ERR_INVALID_SHAPE;
    marlin_status_t st = check_weights(K, N, group);
    if (st != MARLIN_OK) return st;
    if (M == 0) return MARLIN_OK;
    if (!A || !w_packed || !s_packed || !C || !workspace) return MARLIN_ERR_NULL_POINTER;
    if (!aligned16(A) || !aligned16(w_packed) || !aligned16(s_packed) || !aligned16(C) ||
        !aligned16(workspace))
        return MARLIN_ERR_MISALIGNED;

    const int64_t G = scale_rows(K, group);
    const int gu = (group == -1 || group == K) ? 0 : (int)(group / 128);
    if (workspace_bytes < required_workspace(M, (int)N, (int)K, gu))
        return MARLIN_ERR_WORKSPACE_TOO_SMALL;

    int device = 0;
    if (hipGetDevice(&device) != hipSuccess) return MARLIN_ERR_HIP;
    const int cus = device_cu_count(device);
    if (cus <= 0) return MARLIN_ERR_HIP;

    for (int64_t m0 = 0; m0 < M; m0 += kPassRows) {
        const int mp = (M - m0) < kPassRows ? (int)(M - m0) : kPassRows;
        const GemmConfig cfg = choose_config(mp, (int)N, (int)K, gu, cus, sparse);
        const size_t counter_bytes = kCounterRegionBytes;
        GemmProblem p;
        p.A = A + m0 * K;
        p.W = (const uint32_t *)w_packed;
        p.S = (const uint16_t *)s_packed;
        p.C = C + m0 * N;
        p.counters = (uint32_t *)workspace;
        p.partials = (float *)((char *)workspace + counter_bytes);
        p.M = mp;
        p.N = (int)N;
        p.K = (int)K;
        p.G = (int)G;
        p.KU = (int)(K / 128);
        p.rg = cfg.rg;
        p.units = (int)(N / tile_cols(cfg)) * cfg.rg * p.KU;
        p.gran = cfg.whole ? p.KU : 1;
        p.per_wg = (p.units / p.gran) / cfg.grid;
        p.extra = (p.units / p.gran) % cfg.grid;
        p.group_units = gu;
        // Exact for every block index below 2^13 (K <= 2^20): with
        // e = gmagic * gu - 2^26 < gu <= 2^13, ku * e < 2^26.
        p.gmagic = gu > 0 ? (uint32_t)((((uint64_t)1 << 26) + (uint64_t)gu - 1) / (uint64_t)gu) : 0u;
        // w * extra < grid^2 <= 2^18, so w * extra * grid < 2^27: always exact
        p.grid_magic = reciprocal32((uint64_t)cfg.grid);
        // units below p.units: exact when p.units * KU <= 2^32
        p.ku_magic = (uint64_t)p.units * (uint64_t)p.KU <= ((uint64_t)1 << 32) ? reciprocal32((uint64_t)p.KU) : 0u;
        const hipError_t e = launch_gemm(cfg, p, stream);
        if (e != hipSuccess) return MARLIN_ERR_HIP;
    }
    return MARLIN_OK;
}

marlin_status_t describe_impl(int64_t M, int64_t N, int64_t K, int64_t group, char *buf, size_t buf_bytes,
                              bool sparse)
{
    if (!buf) return MARLIN_ERR_NULL_POINTER;
    if (M < 0 || M > (1 << 24)) return MARLIN_ERR_INVALID_SHAPE;
    const marlin_status_t st = check_weights(K, N, group);
    if (st != MARLIN_OK) return st;
    int cus = kMaxCus;
    int device = 0;
    int count = 0;
    if (hipGetDeviceCount(&count) == hipSuccess && count > 0 && hipGetDevice(&device) == hipSuccess) {
        const int c = device_cu_count(device);
        if (c > 0) cus = c;
    } else {
        (void)hipGetLastError();
    }
    const int gu = (group == -1 || group == K) ? 0 : (int)(group / 128);
    const int mp = M < kPassRows ? (M > 0 ? (int)M : 1) : kPassRows;
    const GemmConfig cfg = choose_config(mp, (int)N, (int)K, gu, cus, sparse);
    char name[96];
    kernel_name(cfg, gu == 0, name, sizeof(name));
    if (buf_bytes > 0)
        snprintf(buf, buf_bytes, "%s cols=%d rg=%d partition=%s grid=%d", name,
                 tile_cols(cfg), cfg.rg,
                 cfg.whole ? "whole" : "streamk", cfg.grid);
    return MARLIN_OK;
}
}  // namespace

extern "C" {

int marlin_layout_version(void) { return MARLIN_LAYOUT_VERSION; }

const char *marlin_status_string(marlin_status_t status)
{
    switch (status) {
    case MARLIN_OK: return "MARLIN_OK";
    case MARLIN_ERR_NULL_POINTER: return "MARLIN_ERR_NULL_POINTER";
    case MARLIN_ERR_INVALID_SHAPE: return "MARLIN_ERR_INVALID_SHAPE";
    case MARLIN_ERR_UNSUPPORTED_GROUP: return "MARLIN_ERR_UNSUPPORTED_GROUP";
    case MARLIN_ERR_MISALIGNED: return "MARLIN_ERR_MISALIGNED";
    case MARLIN_ERR_WORKSPACE_TOO_SMALL: return "MARLIN_ERR_WORKSPACE_TOO_SMALL";
    case MARLIN_ERR_HIP: return "MARLIN_ERR_HIP";
    case MARLIN_ERR_INVALID_SPARSITY: return "MARLIN_ERR_INVALID_SPARSITY";
    case MARLIN_ERR_INVALID_ARGUMENT: return "MARLIN_ERR_INVALID_ARGUMENT";
    }
    return "MARLIN_ERR_UNKNOWN";
}

size_t marlin_packed_weight_bytes(int64_t K, int64_t N)
{
    if (!shape_ok(K, N)) return 0;
    return (size_t)K * (size_t)N / 2;
}

size_t marlin_packed_scale_bytes(int64_t K, int64_t N, int64_t group)
{
    if (check_weights(K, N, group) != MARLIN_OK) return 0;
    return (size_t)scale_rows(K, group) * (size_t)N * 2;
}

size_t marlin_workspace_bytes(int64_t M, int64_t N, int64_t K, int64_t group)
{
    if (M < 0 || M > (1 << 24) || check_weights(K, N, group) != MARLIN_OK) return 0;
    const int64_t gu = (group == -1 || group == K) ? 0 : group / 128;
    return required_workspace(M > 0 ? M : 1, (int)N, (int)K, (int)gu);
}

marlin_status_t marlin_pack_weights(const uint8_t *q, const uint16_t *s, int64_t K, int64_t N,
                                    int64_t group, void *w_packed, void *s_packed,
                                    hipStream_t stream)
{
    if (!q || !s || !w_packed || !s_packed) return MARLIN_ERR_NULL_POINTER;
    marlin_status_t st = check_weights(K, N, group);
    if (st != MARLIN_OK) return st;
    if (!aligned16(w_packed) || !aligned16(s_packed)) return MARLIN_ERR_MISALIGNED;
    const hipError_t e = launch_pack(q, s, (int)K, (int)N, (int)scale_rows(K, group),
                                     (uint32_t *)w_packed, (uint16_t *)s_packed, stream);
    return e == hipSuccess ? MARLIN_OK : MARLIN_ERR_HIP;
}

marlin_status_t marlin_quantize(const uint16_t *W, int64_t K, int64_t N, int64_t group, const float *ratios,
                                int n_ratios, uint8_t *q, uint16_t *s, hipStream_t stream)
{
    if (!W || !ratios || !q || !s) return MARLIN_ERR_NULL_POINTER;
    const marlin_status_t st = check_weights(K, N, group);
    if (st != MARLIN_OK) return st;
    if (!aligned16(W) || !aligned16(q) || !aligned16(s)) return MARLIN_ERR_MISALIGNED;
    if (n_ratios < 1 || n_ratios > kMaxQuantRatios) return MARLIN_ERR_INVALID_ARGUMENT;
    for (int i = 0; i < n_ratios; ++i)
        if (!(ratios[i] > 0.0f && ratios[i] <= 1.0f)) return MARLIN_ERR_INVALID_ARGUMENT;  // NaN too
    const int64_t g = (group == -1) ? K : group;
    const hipError_t e = launch_quantize(W, (int)K, (int)N, (int)g, ratios, n_ratios, q, s, stream);
    return e == hipSuccess ? MARLIN_OK : MARLIN_ERR_HIP;
}

size_t marlin_packed_sparse_weight_bytes(int64_t K, int64_t N)
{
    if (!shape_ok(K, N)) return 0;
    return (size_t)K * (size_t)N / 8 * 3;
}

marlin_status_t marlin_pack_sparse_weights(const uint8_t *q, const uint16_t *s, int64_t K, int64_t N,
                                           int64_t group, void *w_packed, void *s_packed, hipStream_t stream)
{
    if (!q || !s || !w_packed || !s_packed) return MARLIN_ERR_NULL_POINTER;
    marlin_status_t st = check_weights(K, N, group);
    if (st != MARLIN_OK) return st;
    if (!aligned16(w_packed) || !aligned16(s_packed)) return MARLIN_ERR_MISALIGNED;
    const hipError_t e = launch_pack_sparse(q, s, (int)K, (int)N, (int)scale_rows(K, group),
                                            (uint32_t *)w_packed, (uint16_t *)s_packed, stream);
    return e == hipSuccess ? MARLIN_OK : MARLIN_ERR_HIP;
}

marlin_status_t marlin_unpack_sparse_weights(const void *w_packed, const void *s_packed, int64_t K, int64_t N,
                                             int64_t group, uint8_t *q, uint16_t *s, hipStream_t stream)
{
    if (!q || !s || !w_packed || !s_packed) return MARLIN_ERR_NULL_POINTER;
    marlin_status_t st = check_weights(K, N, group);
    if (st != MARLIN_OK) return st;
    if (!aligned16(w_packed) || !aligned16(s_packed)) return MARLIN_ERR_MISALIGNED;
    const hipError_t e = launch_unpack_sparse((const uint32_t *)w_packed, (const uint16_t *)s_packed, (int)K,
                                              (int)N, (int)scale_rows(K, group), q, s, stream);
    return e == hipSuccess ? MARLIN_OK : MARLIN_ERR_HIP;
}

marlin_status_t marlin_unpack_weights(const void *w_packed, const void *s_packed, int64_t K,
                                      int64_t N, int64_t group, uint8_t *q, uint16_t *s,
                                      hipStream_t stream)
{
    if (!q || !s || !w_packed || !s_packed) return MARLIN_ERR_NULL_POINTER;
    marlin_status_t st = check_weights(K, N, group);
    if (st != MARLIN_OK) return st;
    if (!aligned16(w_packed) || !aligned16(s_packed)) return MARLIN_ERR_MISALIGNED;
    const hipError_t e = launch_unpack((const uint32_t *)w_packed, (const uint16_t *)s_packed,
                                       (int)K, (int)N, (int)scale_rows(K, group), q, s, stream);
    return e == hipSuccess ? MARLIN_OK : MARLIN_ERR_HIP;
}

marlin_status_t marlin_gemm(const uint16_t *A, const void *w_packed, const void *s_packed,
                            uint16_t *C, void *workspace, size_t workspace_bytes, int64_t M,
                            int64_t N, int64_t K, int64_t group, hipStream_t stream)
{
    return gemm_impl(A, w_packed, s_packed, C, workspace, workspace_bytes, M, N, K, group, stream, false);
}

marlin_status_t marlin_gemm_sparse(const uint16_t *A, const void *w_packed, const void *s_packed,
                                   uint16_t *C, void *workspace, size_t workspace_bytes, int64_t M,
                                   int64_t N, int64_t K, int64_t group, hipStream_t stream)
{
    return gemm_impl(A, w_packed, s_packed, C, workspace, workspace_bytes, M, N, K, group, stream, true);
}

marlin_status_t marlin_describe(int64_t M, int64_t N, int64_t K, int64_t group, char *buf,
                                size_t buf_bytes)
{
    return describe_impl(M, N, K, group, buf, buf_bytes, false);
}

marlin_status_t marlin_describe_sparse(int64_t M, int64_t N, int64_t K, int64_t group, char *buf,
                                       size_t buf_bytes)
{
    return describe_impl(M, N, K, group, buf, buf_bytes, true);
}

}  // extern "C"
