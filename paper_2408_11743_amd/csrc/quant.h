// Internal declarations of the weight quantiser (quant.hip).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace marlin {

// Clipping ratios a caller may pass to one quantiser call (kernel argument).
constexpr int kMaxQuantRatios = 64;

// W [K][N] fp16 -> q [K][N] codes, s [K/g][N] fp16; g divides K; ratios
// (host, n_ratios of them, 1..kMaxQuantRatios) are copied into the launch.
hipError_t launch_quantize(const uint16_t *W, int K, int N, int g, const float *ratios, int n_ratios,
                           uint8_t *q, uint16_t *s, hipStream_t stream);

}  // namespace marlin
