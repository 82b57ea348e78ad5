// Kernel launch with optional dispatch-attached event timing.  Internal to
// libnamoh.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include "internal.h"

namespace namoh {

// Launches kernel<<<grid, block, 0, st>>>(args...).  With event timing on
// (namoh_profile_enable), the launch goes through hipExtLaunchKernel with the
// next event pair of `section` attached to the dispatch, so the recorded
// interval is the kernel's own execution.
template <typename... Params, typename... Args>
inline void launch_k(const char* section, void (*kernel)(Params...), dim3 grid, dim3 block,
                     hipStream_t st, Args... args) {
  hipEvent_t e0, e1;
  if (prof_pair(section, &e0, &e1))
    hipExtLaunchKernelGGL(kernel, grid, block, 0, st, e0, e1, 0, static_cast<Params>(args)...);
  else
    kernel<<<grid, block, 0, st>>>(static_cast<Params>(args)...);
}

}  // namespace namoh
