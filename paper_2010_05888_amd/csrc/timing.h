// Opt-in per-kernel timing. When enabled, every kernel of every call is
// launched with hipExtLaunchKernelGGL and a pair of HIP events that the
// runtime stamps at the start and the end of that kernel's own dispatch (the
// same interval a kernel trace reports, without the extra commands a
// separate event record would put on the stream); the elapsed times are
// summed per kernel name on request. Disabled (the default) it costs one
// relaxed atomic load per launch.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

namespace garfield {

bool timing_enabled();
void timing_set(bool on);  // also drops every pending record

// Events for one timed launch named `name` (a string literal); both null if
// timing is off or no event could be created.
struct LaunchEvents {
  hipEvent_t start = nullptr;
  hipEvent_t stop = nullptr;
};
LaunchEvents timing_record(const char* name);

// Wait for all recorded events and write "name launches total_ms\n" lines.
// Returns the number of bytes written (excluding the terminating NUL).
size_t timing_summary(char* buf, size_t len);

// Launch `kernel` on stream `s`, timed under `name` when timing is enabled.
template <typename F, typename... Args>
void launch(const char* name, F kernel, dim3 grid, dim3 block, uint32_t shmem, hipStream_t s,
            Args... args) {
  if (timing_enabled()) {
    const LaunchEvents ev = timing_record(name);
    hipExtLaunchKernelGGL(kernel, grid, block, shmem, s, ev.start, ev.stop, 0, args...);
  } else {
    hipLaunchKernelGGL(kernel, grid, block, shmem, s, args...);
  }
}

}  // namespace garfield
