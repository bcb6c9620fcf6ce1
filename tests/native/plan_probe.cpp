// Test harness for the launch planner (paper_2408_11743_amd/csrc/plan.cpp),
// built with the host compiler alone: the planner is pure C++, so its
// choices for any compute-unit count and workspace size can be checked on a
// machine without a GPU.
#include <chrono>
#include <cstdint>

#include "plan.h"

using namespace marlin;

extern "C" {

// The configuration of one launch of M rows (<= kPassRows) on `cus` compute
// units with `ws` workspace bytes.  out: kind, nb, mb, whole, grid, rg,
// tile_nw, tile_wm, tile_ks, waves.  Returns the workspace bytes the launch
// touches.
uint64_t probe_plan(int M, int N, int K, int gu, int cus, int sparse, uint64_t ws, int *out)
{
    const GemmConfig c = plan_pass(M, N, K, gu, cus, sparse != 0, (size_t)ws, Override{});
    const int v[10] = {c.kind, c.nb, c.mb, c.whole, c.grid, c.rg, c.tile_nw, c.tile_wm, c.tile_ks, c.waves};
    for (int i = 0; i < 10; ++i) out[i] = v[i];
    return (uint64_t)workspace_bytes_used(c);
}

uint64_t probe_required(int64_t M, int N, int K, int gu) { return (uint64_t)required_workspace(M, N, K, gu, Override{}); }

// Nanoseconds per planning of one call (the override read, the workspace
// size and the launch plan), averaged over `iters` repeats of a sweep of
// shapes already planned once.
double probe_plan_ns(int iters)
{
    const int shapes[4][3] = {{4096, 4096, 1}, {28672, 8192, 224}, {8192, 28672, 64}, {4096, 11008, 32}};
    const int Ms[8] = {1, 2, 4, 8, 16, 32, 64, 128};
    volatile uint64_t sink = 0;
    auto once = [&]() {
        for (auto &s : shapes)
            for (int M : Ms) {
                const Override ov = current_override();
                const size_t ws = required_workspace(M, s[0], s[1], 1, ov);
                const GemmConfig c = plan_pass(M, s[0], s[1], 1, 256, false, ws, ov);
                sink += (uint64_t)c.grid + ws;
            }
    };
    once();
    const auto t0 = std::chrono::steady_clock::now();
    for (int i = 0; i < iters; ++i) once();
    const auto t1 = std::chrono::steady_clock::now();
    (void)sink;
    return std::chrono::duration<double, std::nano>(t1 - t0).count() / (iters * 32.0);
}

}  // extern "C"
