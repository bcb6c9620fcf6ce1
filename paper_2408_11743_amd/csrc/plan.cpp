// Launch planning (see plan.h): a cost model of the two GEMM kernels fitted
// to MI355X measurements, the striped partition (Section 3.4, "Striped
// Partitioning": whole column tiles per work-group, or Stream-K ranges of
// 128-row blocks combined across work-groups), workspace sizing, and a memo
// of the choices so that a repeated call plans in a table lookup.
#include "plan.h"

#include <cstdint>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <string>
#include <unordered_map>

namespace marlin {

Override parse_override(const char *e)
{
    Override f;
    if (!e) return f;
    const char *q = strstr(e, "nb=");
    if (q) f.nb = atoi(q + 3);
    q = strstr(e, "grid=");
    if (q) f.grid = atoi(q + 5);
    q = strstr(e, "whole=");
    if (q) f.whole = atoi(q + 6) ? 1 : 0;
    if (strstr(e, "kind=stream")) f.kind = kKindStream;
    if (strstr(e, "kind=tile")) f.kind = kKindTile;
    if (strstr(e, "kind=wide")) f.kind = kKindWide;
    q = strstr(e, "ks=");
    if (q) f.ks = atoi(q + 3);
    q = strstr(e, "nw=");
    if (q) f.nw = atoi(q + 3);
    q = strstr(e, "waves=");
    if (q) f.waves = atoi(q + 6);
    if (f.waves != 4 && f.waves != 8) f.waves = 0;
    q = strstr(e, "mb=");
    if (q) f.mb = atoi(q + 3);
    if (f.mb != 1 && f.mb != 2 && f.mb != 4) f.mb = 0;
    if (f.nb != 1 && f.nb != 2 && f.nb != 4 && f.nb != 8) f.nb = 0;
    if (f.grid < 0) f.grid = 0;
    return f;
}

Override current_override()
{
    const char *e = getenv("MARLIN_FORCE_CONFIG");
    if (!e) return Override{};
    thread_local std::string last;
    thread_local Override parsed;
    thread_local bool have = false;
    if (!have || last != e) {
        last = e;
        parsed = parse_override(e);
        have = true;
    }
    return parsed;
}

int slot_floats(const GemmConfig &cfg)
{
    if (cfg.kind == kKindTile) return cfg.tile_nw * cfg.nb * cfg.mb * 256;
    if (cfg.kind == kKindWide) return 4 * cfg.nb * cfg.mb * 256;
    return cfg.nb * cfg.mb * 256;
}

// The counter region never moves, whatever the shape, so any sequence of
// calls on one workspace finds every counter it uses at zero; the fp32
// partial slots follow it.
size_t workspace_bytes_for(const GemmConfig &cfg)
{
    return kCounterRegionBytes + (size_t)cfg.grid * 2 * (size_t)slot_floats(cfg) * sizeof(float);
}

size_t workspace_bytes_used(const GemmConfig &cfg) { return cfg.whole ? 0 : workspace_bytes_for(cfg); }

// Configuration by rows of A per pass (at most kPassRows): mb = 1 (M <= 16),
// 2 or (dense, beyond 32 rows) 4 16-row blocks per row group; beyond one
// group's rows the pass is split into row groups that are tiles of their own
// (a tile is a column tile of one row group); 4 * ar activation rows per
// group arrive in LDS; 4 or (one row block, or one column block) 8 waves
// split K, kStreamOcc work-groups per CU.
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
// Four row blocks per wave (64 x 128 per wave, 32 KiB fp32 partial tiles):
// weight bytes per microsecond one work-group streams (its waves convert
// and multiply twice as much per weight byte as with two row blocks, with no
// second wave per SIMD to overlap the two: measured 49 us for whole tiles
// on 8192 x 28672 at 33..64 rows), and the combination (fixed, and per
// contributor: the reducer reads one 32 KiB slot each).
constexpr double kRate64Rows = 11.65e3;
// ... with eight waves, each pair sharing the activations of one 128-deep
// block of K (pair.hip): a SIMD's two waves overlap one's conversion with
// the other's MFMAs (measured 10-20% faster than four waves).  At this rate
// it is weighed for whole tiles only, up to 512 rows (elsewhere it runs in
// place of the four-wave kernel, below): its Stream-K ranges were measured no
// faster than those of 32-row groups at 33..64 rows (K = 28672, N = 8192)
// and slower than the model predicts beyond 64 (K = 4096, N = 11008 at
// M = 128: 29.8 against 24.4 us whole), and at 1024 rows the wide kernel
// leads.
constexpr double kRatePair = 12.7e3;
constexpr double kTail64RowsUs = 4.0;
constexpr double kTail64RowsPerContributorUs = 1.0;

// Bytes of weights per microsecond one work-group streams, by rows of A,
// nb = 8, 4, 2, 1 and waves per work-group (measured; the activation rows
// arrive in LDS in every class).  nb = 8 (two packed 64-column tiles per
// wave) holds twice the weight bytes in flight per wave and reads each
// activation block for twice the columns: fitted to whole-tile and Stream-K
// timings on the 70B-class layers (8192 x 28672, 28672 x 8192) at M = 1..32.
double wg_rate(int mb, int ar, int nb, int waves)
{
    static const double r4[4][4] = {
        {28.0e3, 31.8e3, 22.3e3, 13.3e3},  // M <= 4
        {28.0e3, 32.5e3, 20.8e3, 13.0e3},  // M <= 8
        {26.0e3, 25.2e3, 16.6e3, 10.7e3},  // M <= 16
        {21.5e3, 17.6e3, 11.6e3, 7.1e3},   // M <= 32 (also each row group of 32 for larger M)
    };
    static const double r8[3][4] = {
        {30.0e3, 38.8e3, 34.2e3, 20.2e3},  // M <= 4
        {32.0e3, 32.7e3, 22.1e3, 15.6e3},  // M <= 8
        {27.0e3, 26.0e3, 17.6e3, 11.0e3},  // M <= 16
    };
    const int row = (mb == 1) ? (ar == 1 ? 0 : ar == 2 ? 1 : 2) : 3;
    const int col = (nb == 8) ? 0 : (nb == 4) ? 1 : (nb == 2) ? 2 : 3;
    if (waves == 8) return row < 3 ? r8[row][col] : (nb == 1 ? 7.4e3 : 0.0);
    return r4[row][col];
}

// Best partition of `tiles` tiles of KU units each over at most `grid`
// work-groups, given the time of one unit: whole tiles per work-group, or a
// Stream-K split that pays for combining shared tiles at the end (tail_us,
// plus tail_per_contributor_us per contributor of a shared tile, plus
// tail_per_extra_contributor_us per contributor beyond free_contributors).  Every
// launch costs kFixedUs, and no partition streams faster than floor_us.  A
// split is considered only when its counters and partial slots (slot_bytes
// per work-group) fit in `budget` bytes.
struct Partition {
    double t;
    int whole;
    int64_t grid;
};

Partition best_partition(const Override &ov, int64_t tiles, int KU, int64_t grid, double unit_us, double tail_us,
                         double tail_per_contributor_us, double floor_us, size_t slot_bytes, size_t budget,
                         double free_contributors = 0.0, double tail_per_extra_contributor_us = 0.0)
{
    Partition best{1e30, 0, 1};
    if (ov.whole != 0) {
        const int64_t g = tiles < grid ? tiles : grid;
        const double stream = (double)((tiles + g - 1) / g) * KU * unit_us;
        const double t = kFixedUs + (stream > floor_us ? stream : floor_us);
        if (t < best.t) best = {t, 1, g};
    }
    const int64_t units = tiles * KU;
    const int64_t gs = grid < units ? grid : units;
    const bool fits = budget == SIZE_MAX || kCounterRegionBytes + (size_t)gs * slot_bytes <= budget;
    if (ov.whole != 1 && fits) {
        const double per = (double)units / (double)gs;  // units per work-group
        const bool split = (units % gs) != 0 || (units / gs) % KU != 0;
        const double contributors = split ? 1.0 + (double)KU / per : 1.0;
        const double extra = contributors > free_contributors ? contributors - free_contributors : 0.0;
        const double tail = split ? tail_us + tail_per_contributor_us * contributors +
                                        tail_per_extra_contributor_us * extra
                                  : 0.0;
        const double stream = per * unit_us;
        const double t = kFixedUs + (stream > floor_us ? stream : floor_us) + tail;
        if (t < best.t) best = {t, 0, gs};
    }
    return best;
}
}  // namespace

GemmConfig choose_config(int M, int N, int K, int group_units, int cus, bool sparse, const Override &ov,
                         size_t partial_budget)
{
    (void)group_units;
    GemmConfig cfg;
    const int KU = K / 128;
    const int tiles16 = N / 16;
    const int ncu = cus < kMaxCus ? cus : kMaxCus;
    int64_t grid = (int64_t)ncu * kStreamOcc;
    if (ov.grid) grid = ov.grid;
    if (grid > (int64_t)kMaxCus * kMaxPerCu) grid = (int64_t)kMaxCus * kMaxPerCu;

    // stream kernel
    cfg.kind = kKindStream;
    cfg.tile_wm = 0;
    cfg.tile_ks = 0;
    cfg.tile_nw = 0;
    cfg.waves = 4;
    cfg.sparse = sparse ? 1 : 0;
    // Rows per row group: 16 (M <= 16), 32, or (dense, beyond 32 rows, or
    // forced) 64 in four row blocks per wave, which read each weight once for
    // twice the rows and take their activations in 16 KiB stages.
    const int mb_small = (M <= 16) ? 1 : 2;
    const bool mb4_ok = !sparse && (M > 32 || ov.mb == 4);
    cfg.mb = mb_small;
    cfg.ar = (M <= 4) ? 1 : (M <= 8) ? 2 : (M <= 16) ? 4 : 8;
    cfg.rg = (M + 16 * cfg.mb - 1) / (16 * cfg.mb);  // row groups, each a copy of the column tiles
    double best = 1e30;
    cfg.nb = 0;
    cfg.whole = 0;
    int64_t best_grid = grid;
    for (int mb : {mb_small, 4}) {
        if (ov.kind == kKindTile || ov.kind == kKindWide) break;
        if (mb == 4 && !mb4_ok) continue;
        if (ov.mb && mb != ov.mb && (ov.mb == 4 ? mb4_ok : ov.mb == mb_small)) continue;
        const int ar = mb == 4 ? 16 : cfg.ar;
        const int64_t rg = (M + 16 * mb - 1) / (16 * mb);
        // eight waves exist for one 16-row block, or two with one 16-column
        // block; an override to eight applies where they do
        const int forced_waves = (ov.waves == 8 && mb == 2 && ov.nb > 1) ? 4 : ov.waves;
        for (int waves = 8; waves >= 4; waves -= 4) {
            if (forced_waves && waves != forced_waves) continue;
            for (int nb = (sparse && mb != 2) ? 4 : 8; nb >= 1; nb >>= 1) {
                if (mb == 4 && nb != 8) continue;  // four row blocks: 128-column tiles
                const double rate = mb == 4 ? (waves == 8 ? kRatePair : kRate64Rows) : wg_rate(mb, ar, nb, waves);
                if (tiles16 % nb != 0 || rate <= 0.0) continue;
                if (ov.nb && nb != ov.nb) continue;
                const int64_t tiles = (int64_t)(tiles16 / nb) * rg;
                // sparse units carry 3/4 of the dense bytes (codes and row indices)
                const double unit_bytes = (double)nb * (sparse ? 768.0 : 1024.0);
                const double layer_bytes = (double)KU * (double)(tiles16 / nb) * unit_bytes;
                // fp32 partial tile: 16 x 16 x 4 bytes per block, two slots
                const size_t slot_bytes = (size_t)2 * nb * mb * 256 * sizeof(float);
                // the eight-wave kernel: whole tiles, up to 512 rows, unless forced
                Override ovp = ov;
                if (mb == 4 && waves == 8) {
                    if (M > 512 && ov.waves != 8) continue;
                    if (ov.whole != 0) ovp.whole = 1;
                }
                const Partition pt =
                    mb == 4 ? best_partition(ovp, tiles, KU, grid, unit_bytes / rate, kTail64RowsUs,
                                             kTail64RowsPerContributorUs, layer_bytes / kChipBytesPerUs, slot_bytes,
                                             partial_budget)
                            : best_partition(ov, tiles, KU, grid, unit_bytes / rate, stream_tail_us(nb * mb), 0.0,
                                             layer_bytes / kChipBytesPerUs, slot_bytes, partial_budget,
                                             kStreamFreeContributors, kStreamTailPerExtraContributorUs);
                if (pt.t < best) {
                    best = pt.t;
                    cfg.mb = mb;
                    cfg.ar = ar;
                    cfg.rg = (int)rg;
                    cfg.nb = nb;
                    cfg.waves = waves;
                    cfg.whole = pt.whole;
                    best_grid = pt.grid;
                }
            }
        }
    }
    // Four row blocks with four waves are modelled as measured, but run with
    // eight (the pair kernel, measured 7-22% faster at every partition and
    // row-group count tried) unless four are forced.
    if (cfg.kind == kKindStream && cfg.mb == 4 && cfg.waves == 4 && ov.waves != 4) cfg.waves = 8;
    // tile kernel: the activation tile is shared by the waves of a
    // work-group.  Beyond 32 rows each wave owns 64 x 64 outputs (four waves:
    // 2x2 beyond 64 rows, else 4x1; eight waves, two per SIMD: 4x2), one
    // 128-row block per stage; up to 32 rows, 4x1 waves of 16 or 32 rows over
    // 2 or 4 blocks per stage (measured to win only where whole 128-column
    // tiles fill the chip at 17..32 rows, e.g. N = 28672).
    if (!sparse && ov.kind != kKindStream && ov.kind != kKindWide) {
        for (int nw = 8; nw >= 4; nw -= 4) {
            if (ov.nw && nw != ov.nw) continue;
            // rows per tile: 64*wm with 64-row waves; eight waves at 33..64
            // rows use 4x2 waves of 32 rows
            const int wm = (M > 64 || (nw == 8 && M > 32)) ? 2 : 1;
            const int mbw = (nw == 8 && M > 32 && M <= 64) ? 2 : M > 32 ? 4 : M > 16 ? 2 : 1;
            for (int nbw = 4; nbw >= 1; nbw >>= 1) {
                for (int ks = 4; ks >= 1; ks >>= 1) {
                    if (!tile_config_supported(nw, wm, mbw, nbw, ks)) continue;
                    if (ov.nb && nbw != ov.nb) continue;
                    if (ov.ks && ks != ov.ks) continue;
                    const int cols = (nw / wm) * 16 * nbw, rows = wm * 16 * mbw;
                    if (N % cols != 0) continue;
                    const int64_t tiles = (int64_t)(N / cols) * ((M + rows - 1) / rows);
                    const TileCost tc = tile_cost(nw, wm, mbw, nbw);
                    const size_t slot_bytes = (size_t)2 * nw * nbw * mbw * 256 * sizeof(float);
                    const Partition pt = best_partition(ov, tiles, KU, grid, tc.unit_us, tc.tail_us,
                                                        tc.tail_per_contributor_us, 0.0, slot_bytes, partial_budget);
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
    // wide kernel: four waves along N, each 64 x 128 or 128 x 64 outputs,
    // weights in registers, activations and group scales shared in LDS.  One
    // wave per SIMD: its dequantization and its MFMAs do not overlap, so it
    // wins only where each dequantized weight feeds 128 rows, beyond 128 rows
    // (measured per 128-row block of a tile: 1.92 us for 128 x 256 tiles,
    // 2.15 us for 64 x 512; the combination reads 128 KiB fp32 slots).
    if (!sparse && ov.kind != kKindStream && ov.kind != kKindTile && (M > 128 || ov.kind == kKindWide)) {
        const int shapes[2][2] = {{8, 4}, {4, 8}};  // 16-row blocks, 16-column blocks per wave
        for (const auto &sh : shapes) {
            const int mbw = sh[0], nbw = sh[1];
            if (ov.nb && nbw != ov.nb) continue;
            const int cols = 64 * nbw, rows = 16 * mbw;
            if (N % cols != 0) continue;
            const int64_t tiles = (int64_t)(N / cols) * ((M + rows - 1) / rows);
            const size_t slot_bytes = (size_t)2 * 4 * nbw * mbw * 256 * sizeof(float);
            const double unit_us = mbw == 8 ? 1.92 : 2.15;
            const Partition pt =
                best_partition(ov, tiles, KU, grid, unit_us, 8.0, 2.0, 0.0, slot_bytes, partial_budget);
            if (pt.t < best) {
                best = pt.t;
                cfg.kind = kKindWide;
                cfg.tile_nw = 4;
                cfg.tile_wm = 1;
                cfg.tile_ks = 1;
                cfg.waves = 0;
                cfg.nb = nbw;
                cfg.mb = mbw;
                cfg.ar = 0;
                cfg.rg = (M + rows - 1) / rows;
                cfg.whole = pt.whole;
                best_grid = pt.grid;
            }
        }
    }
    if (cfg.nb == 0) {  // only when an override excludes every choice (or asks for the tile kernel, sparse)
        cfg.kind = kKindStream;
        cfg.waves = 4;
        cfg.nb = (tiles16 % 2 == 0) ? 2 : 1;
        const int64_t tiles = (int64_t)(tiles16 / cfg.nb) * cfg.rg;
        const int64_t units = tiles * KU;
        const int64_t gs = grid < units ? grid : units;
        const size_t slot_bytes = (size_t)2 * cfg.nb * cfg.mb * 256 * sizeof(float);
        const bool fits = partial_budget == SIZE_MAX || kCounterRegionBytes + (size_t)gs * slot_bytes <= partial_budget;
        cfg.whole = fits ? 0 : 1;
        best_grid = fits ? gs : (grid < tiles ? grid : tiles);
    }
    if (best_grid < 1) best_grid = 1;
    cfg.grid = (int)best_grid;
    return cfg;
}

namespace {
struct PlanKey {
    int M, N, K, gu, cus, sparse;
    Override ov;
    size_t budget;
    bool operator==(const PlanKey &o) const
    {
        return M == o.M && N == o.N && K == o.K && gu == o.gu && cus == o.cus && sparse == o.sparse && ov == o.ov &&
               budget == o.budget;
    }
};
struct PlanKeyHash {
    size_t operator()(const PlanKey &k) const
    {
        uint64_t h = 1469598103934665603ull;
        auto mix = [&](uint64_t v) { h = (h ^ v) * 1099511628211ull; };
        mix((uint64_t)k.M);
        mix((uint64_t)k.N);
        mix((uint64_t)k.K);
        mix((uint64_t)(k.gu * 4 + k.sparse * 2));
        mix((uint64_t)k.cus);
        mix((uint64_t)(k.ov.nb + 8 * (k.ov.whole + 2) + 64 * (k.ov.kind + 2) + 512 * k.ov.ks + 8192 * k.ov.nw +
                       131072 * k.ov.waves + 2097152 * k.ov.mb));
        mix((uint64_t)k.ov.grid);
        mix((uint64_t)k.budget);
        return (size_t)h;
    }
};
std::mutex g_plan_mutex;
std::unordered_map<PlanKey, GemmConfig, PlanKeyHash> g_plans;
constexpr size_t kMaxPlans = 1 << 14;

GemmConfig cached_choose(int M, int N, int K, int gu, int cus, bool sparse, const Override &ov, size_t budget)
{
    const PlanKey key{M, N, K, gu, cus, sparse ? 1 : 0, ov, budget};
    {
        std::lock_guard<std::mutex> lock(g_plan_mutex);
        auto it = g_plans.find(key);
        if (it != g_plans.end()) return it->second;
    }
    const GemmConfig cfg = choose_config(M, N, K, gu, cus, sparse, ov, budget);
    std::lock_guard<std::mutex> lock(g_plan_mutex);
    if (g_plans.size() >= kMaxPlans) g_plans.clear();
    g_plans.emplace(key, cfg);
    return cfg;
}
}  // namespace

GemmConfig plan_pass(int M, int N, int K, int gu, int cus, bool sparse, size_t workspace_bytes, const Override &ov)
{
    const GemmConfig cfg = cached_choose(M, N, K, gu, cus, sparse, ov, SIZE_MAX);
    if (workspace_bytes_used(cfg) <= workspace_bytes) return cfg;
    // the device's preferred split needs more than the caller's workspace
    // (a device with fewer compute units than the size was computed for, or
    // a fixed scratch area): the best configuration that fits
    return cached_choose(M, N, K, gu, cus, sparse, ov, workspace_bytes);
}

size_t required_workspace(int64_t M, int N, int K, int gu, const Override &ov)
{
    const int m_first = M < kPassRows ? (int)M : kPassRows;
    const int m_last = (int)(M % kPassRows);
    size_t need = 0;
    for (int sp = 0; sp < 2; ++sp) {
        size_t b = workspace_bytes_for(cached_choose(m_first, N, K, gu, kMaxCus, sp != 0, ov, SIZE_MAX));
        if (b > need) need = b;
        if (M > kPassRows && m_last != 0) {
            b = workspace_bytes_for(cached_choose(m_last, N, K, gu, kMaxCus, sp != 0, ov, SIZE_MAX));
            if (b > need) need = b;
        }
    }
    return need;
}

}  // namespace marlin
