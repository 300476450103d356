// Shader clock sampler (a measurement aid, not part of the method): one
// wave records pairs (shader clock count, 100 MHz real-time count) at a
// fixed real-time interval, so that the clock a workload runs at can be read
// by launching it on another stream beside that workload.  Lane 0 alone
// works; the loop ends after n samples whatever the clocks do.
#include <hip/hip_runtime.h>
#include "../../include/oc.h"
#include "oc_internal.h"

namespace oc {

__global__ __launch_bounds__(64) void k_clock_sample(long long *__restrict__ out, int n, int gap) {
    if (threadIdx.x != 0) return;
    for (int i = 0; i < n; ++i) {
        const long long r0 = wall_clock64();
        out[2 * i] = clock64();
        out[2 * i + 1] = r0;
        // the real-time counter always advances: the wait ends after `gap` ticks
        while (wall_clock64() - r0 < gap) {
        }
    }
}

}  // namespace oc

extern "C" oc_status oc_clock_sample(int64_t *samples, int32_t n, int32_t gap_ticks, hipStream_t stream) {
    if (samples == nullptr || n <= 0 || gap_ticks < 0 || gap_ticks > 100000000) return OC_ERR_INVALID_ARG;
    hipLaunchKernelGGL(oc::k_clock_sample, dim3(1), dim3(64), 0, stream, (long long *)samples, (int)n, (int)gap_ticks);
    return hipGetLastError() == hipSuccess ? OC_OK : OC_ERR_HIP;
}
