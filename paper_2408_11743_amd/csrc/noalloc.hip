// marlin_gemm_no_alloc: marlin_gemm for callers that cannot allocate (code
// under HIP graph capture, serving loops that forbid allocation).  Its
// workspace (the arrival counters and fp32 partial tiles of a Stream-K style
// split) is a file-scope device array instead of a caller's buffer.
//
// In host code the array's name is a host-side stand-in, not a device
// address: every use below goes through the address hipGetSymbolAddress
// returns for the current device (each device holds its own copy of the
// array, at its own address), looked up once per device.
#include <hip/hip_runtime.h>

#include <mutex>

#include "internal.h"
#include "marlin.h"

namespace marlin {
namespace {

// Counters first (the region every workspace starts with), then the partial
// slots: 32 MiB covers every Stream-K split of the stream kernel and of the
// four-wave tile kernels on a 256-compute-unit device; a split that would
// need more is planned with whole tiles or another shape that fits.
constexpr size_t kScratchBytes = kCounterRegionBytes + ((size_t)32 << 20);

// The counters must be zero when a call starts: the first call on a device
// clears them, and every launch returns the counters it used to zero.
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void *g_scratch_ptr[kMaxDevices];

// Zero fill of the counter region (a kernel, not hipMemsetAsync, so that a
// first call made under graph capture records a kernel node).
__global__ void clear_counters(uint4 *p, int n)
{
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x)
        p[i] = make_uint4(0u, 0u, 0u, 0u);
}

// The device address of this device's copy of the array, looked up on the
// device's first call, whose stream then clears the counter region ahead of
// the call's launches (NULL on failure).
void *scratch_on(int device, hipStream_t stream)
{
    if (device < 0 || device >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (!g_scratch_ptr[device]) {
        void *ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) {
            (void)hipGetLastError();
            return nullptr;
        }
        constexpr int n = (int)(kCounterRegionBytes / sizeof(uint4));
        hipLaunchKernelGGL(clear_counters, dim3(n / 256), dim3(256), 0, stream, (uint4 *)ptr, n);
        if (hipGetLastError() != hipSuccess) return nullptr;
        g_scratch_ptr[device] = ptr;
    }
    return g_scratch_ptr[device];
}

}  // namespace
}  // namespace marlin

extern "C" marlin_status_t marlin_gemm_no_alloc(const uint16_t *A, const void *w_packed, const void *s_packed,
                                                uint16_t *C, int64_t M, int64_t N, int64_t K, int64_t group,
                                                hipStream_t stream)
{
    using namespace marlin;
    // Every argument check runs before any HIP call.
    const marlin_status_t st = check_gemm_args(A, w_packed, s_packed, C, M, N, K, group);
    if (st != MARLIN_OK || M == 0) return st;
    int device = 0;
    if (hipGetDevice(&device) != hipSuccess) return MARLIN_ERR_HIP;
    void *ws = scratch_on(device, stream);
    if (!ws) return MARLIN_ERR_HIP;
    return gemm_entry(A, w_packed, s_packed, C, ws, kScratchBytes, M, N, K, group, stream, false, true);
}
