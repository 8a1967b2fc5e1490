// Kernel launch with optional timing.  While a LaunchTimer is set on the calling
// thread, launches go through hipExtLaunchKernelGGL, whose dispatch records the
// timer's start event as the first kernel of a launcher begins and its stop event
// as the last one ends (the kernels' own execution, without launch gaps);
// otherwise they are plain hipLaunchKernelGGL launches (and can be captured).
#pragma once
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include "kernels.h"

namespace wici {

enum LaunchEdge { kFirst = 1, kLast = 2, kOnly = 3 };

template <typename F, typename... Args>
inline void launch_k(F kernel, dim3 grid, dim3 block, size_t lds, hipStream_t st, int edge,
                     Args... args) {
  if (const LaunchTimer* t = launch_timer())
    hipExtLaunchKernelGGL(kernel, grid, block, (std::uint32_t)lds, st,
                          (edge & kFirst) ? t->start : nullptr, (edge & kLast) ? t->stop : nullptr,
                          0u, args...);
  else
    hipLaunchKernelGGL(kernel, grid, block, lds, st, args...);
}

}  // namespace wici
