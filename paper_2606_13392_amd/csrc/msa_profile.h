// Opt-in per-kernel timing (msa_profile_* in msa.h): while enabled, every
// launch made through msa_prof::launch is bracketed by a pair of HIP events
// recorded on the launch's stream.  Disabled, a launch costs one load and a
// branch more than a bare hipLaunchKernelGGL.
#pragma once

#include <hip/hip_runtime.h>

namespace msa_prof {

bool enabled();
void record(const char* kernel, hipEvent_t* start, hipEvent_t* stop);   // hands out an event pair

template <typename Kernel, typename... Args>
inline void launch(const char* name, Kernel kernel, dim3 grid, dim3 block, size_t shmem, hipStream_t stream,
                   Args... args) {
  hipEvent_t start = nullptr, stop = nullptr;
  const bool on = enabled();
  if (on) {
    record(name, &start, &stop);
    if (start) (void)hipEventRecord(start, stream);   // a failed record makes the read fail
  }
  hipLaunchKernelGGL(kernel, grid, block, shmem, stream, args...);
  if (on && stop) (void)hipEventRecord(stop, stream);
}

}  // namespace msa_prof
