// Kernel launch helper of the HIP sources (not needed by the host-only
// C ABI code, which includes pf_internal.h alone).
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include "pf_internal.h"

namespace pf {

// Launch on stream s; when the kernel timing hook handed this thread a pair
// of events, the dispatch itself records them at the kernel's start and end.
template <typename F, typename... Args>
inline void launch_kernel(F kernel, dim3 grid, dim3 block, hipStream_t s, Args... args) {
  LaunchEvents &e = next_launch_events();
  if (e.start) {
    hipExtLaunchKernelGGL(kernel, grid, block, 0, s, e.start, e.stop, 0, args...);
    e.start = e.stop = nullptr;
  } else {
    hipLaunchKernelGGL(kernel, grid, block, 0, s, args...);
  }
}

}  // namespace pf
