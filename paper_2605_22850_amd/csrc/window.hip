// Compute-window stand-in: holds its stream for a fixed wall time.  Used
// when a pipeline run emulates the rest of the model's per-layer compute
// (eq. (3)'s C_l), so that the overlap of transfer and compute can be set to
// a given window.  One wavefront sleeps on the constant 100 MHz real-time
// counter; it occupies almost nothing of the chip, and every wavefront leaves
// once the deadline has passed.
#include "common.hpp"

namespace oc {

__global__ __launch_bounds__(64) void compute_window_kernel(uint64_t ticks) {
    const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
    while (__builtin_amdgcn_s_memrealtime() - t0 < ticks) __builtin_amdgcn_s_sleep(32);
}

hipError_t launch_compute_window(double seconds, hipStream_t s) {
    if (!(seconds > 0.0)) return hipSuccess;
    const uint64_t ticks = (uint64_t)(seconds * 1e8 + 0.5);   // 100 MHz
    hipLaunchKernelGGL(compute_window_kernel, dim3(1), dim3(64), 0, s, ticks);
    return hipGetLastError();
}

}  // namespace oc
