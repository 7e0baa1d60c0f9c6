// Kernel launch helper of libfqvit's gfx950 kernels (device translation units
// only).
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include "fqvit_internal.h"

namespace fqvit {

// Every kernel launch of the library goes through here so that the events, if
// any, record the kernel's own start and end.
template <typename... KArgs, typename... Args>
inline void launch_kernel(void (*kernel)(KArgs...), dim3 grid, dim3 block, size_t lds,
                          hipStream_t stream, Args... args) {
    const LaunchEvents& ev = launch_events();
    if (ev.start || ev.stop)
        hipExtLaunchKernelGGL(kernel, grid, block, (uint32_t)lds, stream, ev.start, ev.stop, 0,
                              args...);
    else
        hipLaunchKernelGGL(kernel, grid, block, lds, stream, args...);
}

}  // namespace fqvit
