// Internal declarations shared by the host API and the kernel launchers.
// Not part of the public ABI (include/marlin.h is).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "marlin.h"
#include "plan.h"

namespace marlin {

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

// Device facts cached per device.
int device_cu_count(int device);

// The host-side checks of a GEMM call's arguments, workspace aside (shape,
// group, pointers, alignment); MARLIN_OK for M == 0 with any pointers.
marlin_status_t check_gemm_args(const uint16_t *A, const void *w_packed, const void *s_packed, const uint16_t *C,
                                int64_t M, int64_t N, int64_t K, int64_t group);

// A validated GEMM call (marlin_gemm, marlin_gemm_sparse and the
// allocation-free entry point).  Argument checks run first; then each launch
// of up to kPassRows rows is planned on the current device.  fit = false:
// the workspace must hold required_workspace (else
// MARLIN_ERR_WORKSPACE_TOO_SMALL); fit = true: every launch is planned to fit
// workspace_bytes (whole tiles need none of it).
marlin_status_t gemm_entry(const uint16_t *A, const void *w_packed, const void *s_packed, uint16_t *C,
                           void *workspace, size_t workspace_bytes, int64_t M, int64_t N, int64_t K, int64_t group,
                           hipStream_t stream, bool sparse, bool fit);

hipError_t launch_gemm(const GemmConfig &cfg, const GemmProblem &p, hipStream_t stream);
// Name of the kernel instantiation launch_gemm runs for cfg ("" if none).
void kernel_name(const GemmConfig &cfg, bool per_channel, char *buf, size_t n);
hipError_t launch_tile_gemm(const GemmConfig &cfg, const GemmProblem &p, hipStream_t stream);
void tile_kernel_name(const GemmConfig &cfg, bool per_channel, char *buf, size_t n);
hipError_t launch_wide_gemm(const GemmConfig &cfg, const GemmProblem &p, hipStream_t stream);
void wide_kernel_name(const GemmConfig &cfg, bool per_channel, char *buf, size_t n);
// The stream kernel's 64-row tiles with eight waves (pair.hip).
hipError_t launch_pair_gemm(const GemmConfig &cfg, const GemmProblem &p, hipStream_t stream);
void pair_kernel_name(bool per_channel, char *buf, size_t n);

hipError_t launch_pack(const uint8_t *q, const uint16_t *s, int K, int N, int G,
                       uint32_t *w_packed, uint16_t *s_packed, hipStream_t stream);
hipError_t launch_unpack(const uint32_t *w_packed, const uint16_t *s_packed, int K, int N,
                         int G, uint8_t *q, uint16_t *s, hipStream_t stream);
hipError_t launch_pack_sparse(const uint8_t *q, const uint16_t *s, int K, int N, int G, uint32_t *w_packed,
                              uint16_t *s_packed, hipStream_t stream);
hipError_t launch_unpack_sparse(const uint32_t *w_packed, const uint16_t *s_packed, int K, int N, int G,
                                uint8_t *q, uint16_t *s, hipStream_t stream);

}  // namespace marlin
