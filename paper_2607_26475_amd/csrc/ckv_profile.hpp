// ckv_profile.hpp -- optional per-kernel timing with dispatch-stamped events.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include "ckv.h"

namespace ckv {

// When recording is on, hands out an event pair for a launch of kernel class
// `id` and returns true; otherwise returns false and the launch is plain.
bool profile_events(int id, hipEvent_t* start, hipEvent_t* stop);

template <typename F, typename... Args>
inline void launch_kernel(int id, F kernel, dim3 grid, dim3 block, hipStream_t s,
                          Args... args) {
  hipEvent_t a, b;
  if (profile_events(id, &a, &b))
    hipExtLaunchKernelGGL(kernel, grid, block, 0, s, a, b, 0, args...);
  else
    hipLaunchKernelGGL(kernel, grid, block, 0, s, args...);
}

}  // namespace ckv
