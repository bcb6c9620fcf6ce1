// Host side of the C ABI declared in include/marlin.h: argument checks (all
// before any HIP call), workspace checks and launches.  The launch
// configuration and workspace sizes come from the planner (plan.cpp).
#include <hip/hip_runtime.h>

#include <atomic>
#include <cstdint>
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

}  // namespace marlin

using namespace marlin;

marlin_status_t marlin::check_gemm_args(const uint16_t *A, const void *w_packed, const void *s_packed,
                                        const uint16_t *C, int64_t M, int64_t N, int64_t K, int64_t group)
{
    if (M < 0 || M > (1 << 24)) return MARLIN_ERR_INVALID_SHAPE;
    const marlin_status_t st = check_weights(K, N, group);
    if (st != MARLIN_OK) return st;
    if (M == 0) return MARLIN_OK;
    if (!A || !w_packed || !s_packed || !C) return MARLIN_ERR_NULL_POINTER;
    if (!aligned16(A) || !aligned16(w_packed) || !aligned16(s_packed) || !aligned16(C)) return MARLIN_ERR_MISALIGNED;
    return MARLIN_OK;
}

marlin_status_t marlin::gemm_entry(const uint16_t *A, const void *w_packed, const void *s_packed, uint16_t *C,
                                   void *workspace, size_t workspace_bytes, int64_t M, int64_t N, int64_t K,
                                   int64_t group, hipStream_t stream, bool sparse, bool fit)
{
    const marlin_status_t st = check_gemm_args(A, w_packed, s_packed, C, M, N, K, group);
    if (st != MARLIN_OK || M == 0) return st;
    if (!workspace) return MARLIN_ERR_NULL_POINTER;
    if (!aligned16(workspace)) return MARLIN_ERR_MISALIGNED;

    const int64_t G = scale_rows(K, group);
    const int gu = (group == -1 || group == K) ? 0 : (int)(group / 128);
    const Override ov = current_override();
    if (!fit && workspace_bytes < required_workspace(M, (int)N, (int)K, gu, ov))
        return MARLIN_ERR_WORKSPACE_TOO_SMALL;

    int device = 0;
    if (hipGetDevice(&device) != hipSuccess) return MARLIN_ERR_HIP;
    const int cus = device_cu_count(device);
    if (cus <= 0) return MARLIN_ERR_HIP;

    for (int64_t m0 = 0; m0 < M; m0 += kPassRows) {
        const int mp = (M - m0) < kPassRows ? (int)(M - m0) : kPassRows;
        // The device's choice, or (fewer compute units than the workspace
        // was sized for, or a fixed scratch area) the best one that fits.
        const GemmConfig cfg = plan_pass(mp, (int)N, (int)K, gu, cus, sparse, workspace_bytes, ov);
        if (workspace_bytes_used(cfg) > workspace_bytes) return MARLIN_ERR_WORKSPACE_TOO_SMALL;
        GemmProblem p;
        p.A = A + m0 * K;
        p.W = (const uint32_t *)w_packed;
        p.S = (const uint16_t *)s_packed;
        p.C = C + m0 * N;
        p.counters = (uint32_t *)workspace;
        p.partials = (float *)((char *)workspace + kCounterRegionBytes);
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

namespace {
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
    const GemmConfig cfg = plan_pass(mp, (int)N, (int)K, gu, cus, sparse, SIZE_MAX, current_override());
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
    return required_workspace(M > 0 ? M : 1, (int)N, (int)K, (int)gu, current_override());
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
    return gemm_entry(A, w_packed, s_packed, C, workspace, workspace_bytes, M, N, K, group, stream, false, false);
}

marlin_status_t marlin_gemm_sparse(const uint16_t *A, const void *w_packed, const void *s_packed,
                                   uint16_t *C, void *workspace, size_t workspace_bytes, int64_t M,
                                   int64_t N, int64_t K, int64_t group, hipStream_t stream)
{
    return gemm_entry(A, w_packed, s_packed, C, workspace, workspace_bytes, M, N, K, group, stream, true, false);
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
