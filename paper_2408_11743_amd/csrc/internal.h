// Internal declarations shared by the host API and the kernel launchers.
// Not part of the public ABI (include/marlin.h is).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace marlin {

// One launch configuration of the GEMM kernel.
//   mb  : 16-row blocks of A handled per pass (M_pad = 16 * mb, M <= M_pad)
//   nw  : waves along N; each wave owns one 64-column tile
//   kw  : waves along K; each takes a different 128-row block of a stage
//   grid: work-groups (Stream-K workers)
constexpr int kKindStream = 0;  // register-streaming kernel (M <= 32)
constexpr int kKindLds = 1;     // LDS-pipeline kernel (M > 32)
constexpr int kStreamDepthMB1 = 6;
constexpr int kStreamDepthMB2 = 4;

struct GemmConfig {
    int kind;
    int mb;
    int nw;
    int kw;
    int grid;
};

struct GemmProblem {
    const uint16_t *A;
    const uint32_t *W;
    const uint16_t *S;
    uint16_t *C;
    float *partials;      // fp32 partial tiles, 2 slots per work-group
    uint32_t *counters;   // one arrival counter per column tile
    int M;                // rows in this pass (1 .. 16*mb)
    int N;
    int K;
    int G;                // scale rows
    int group_units;      // 128-row blocks per scale group; 0 = per-channel
};

// Upper bound on compute units used (MI355X has 256).  Workspace sizes are
// computed with this bound, never with the device's.
constexpr int kMaxCus = 256;

// Device facts cached per device.
int device_cu_count(int device);

GemmConfig choose_config(int M, int N, int K, int group_units, int grid_cap);
size_t workspace_bytes_for(const GemmConfig &cfg, int N);

hipError_t launch_gemm(const GemmConfig &cfg, const GemmProblem &p, hipStream_t stream);

hipError_t launch_pack(const uint8_t *q, const uint16_t *s, int K, int N, int G,
                       uint32_t *w_packed, uint16_t *s_packed, hipStream_t stream);
hipError_t launch_unpack(const uint32_t *w_packed, const uint16_t *s_packed, int K, int N,
                         int G, uint8_t *q, uint16_t *s, hipStream_t stream);

}  // namespace marlin
