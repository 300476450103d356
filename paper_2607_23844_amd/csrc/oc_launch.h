// Kernel launches of the library.  When a stage timer (oc_timer_*) is
// attached to the calling thread inside a StageScope, each launch carries
// start/stop events that the runtime timestamps at the kernel's own start
// and end (hipExtLaunchKernelGGL), so stage times are kernel durations
// without dispatch gaps.
#pragma once
#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>
#include "oc_internal.h"

namespace oc {

// An event pair for the next launch on st when a stage is being timed.
bool timed_launch_events(hipStream_t st, hipEvent_t *start, hipEvent_t *stop);

// Allows `kernel` `bytes` of dynamic LDS on the current device (a no-op up to
// 64 KB; once per kernel and device above, thread-safe).
hipError_t raise_lds_limit(const void *kernel, size_t bytes);

template <typename... KArgs, typename... Args>
inline void launch_k(void (*k)(KArgs...), dim3 grid, dim3 block, size_t lds, hipStream_t st, Args... args) {
    hipEvent_t a = nullptr, b = nullptr;
    if (timed_launch_events(st, &a, &b))
        hipExtLaunchKernelGGL(k, grid, block, (std::uint32_t)lds, st, a, b, 0u, args...);
    else
        hipLaunchKernelGGL(k, grid, block, (std::uint32_t)lds, st, args...);
}

}  // namespace oc
