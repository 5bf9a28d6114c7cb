// ckv_profile.hpp -- optional per-kernel timing with dispatch-stamped events.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include "ckv.h"

namespace ckv {

// When recording is on, hands out an event pair for a launch of kernel class
// `id` and returns true; otherwise returns false and the launch is plain.
bool profile_events(int id, hipEvent_t* start, hipEvent_t* stop);

// Debug mode (ckv_set_debug): every launch synchronises its stream; a failure
// is kept for launch_status().
bool debug_on();
void debug_after_launch(hipStream_t s);
// The status of the launches since the last call: a failure that a debug
// synchronisation saw, else hipGetLastError().
hipError_t launch_status();

template <typename F, typename... Args>
inline void launch_kernel(int id, F kernel, dim3 grid, dim3 block, hipStream_t s,
                          Args... args) {
  hipEvent_t a, b;
  if (profile_events(id, &a, &b))
    hipExtLaunchKernelGGL(kernel, grid, block, 0, s, a, b, 0, args...);
  else
    hipLaunchKernelGGL(kernel, grid, block, 0, s, args...);
  if (debug_on()) debug_after_launch(s);
}

}  // namespace ckv
