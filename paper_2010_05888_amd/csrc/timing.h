// Opt-in per-kernel timing: when enabled, a HIP event pair is recorded on the
// launch stream around every kernel of every call, and the elapsed times are
// summed per kernel name on request. Disabled (the default) it costs one
// relaxed atomic load per launch.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>

namespace garfield {

bool timing_enabled();
void timing_set(bool on);  // also drops every pending record
// Record the start event of a launch named `name` (a string literal).
void timing_begin(const char* name, hipStream_t s);
// Record the stop event of the launch most recently begun on this thread.
void timing_end(hipStream_t s);
// Wait for all recorded events and write "name launches total_ms\n" lines.
// Returns the number of bytes written (excluding the terminating NUL).
size_t timing_summary(char* buf, size_t len);

// RAII helper: `TimedLaunch t("k_median", s);` around one kernel launch.
struct TimedLaunch {
  hipStream_t s;
  bool on;
  TimedLaunch(const char* name, hipStream_t stream) : s(stream), on(timing_enabled()) {
    if (on) timing_begin(name, s);
  }
  ~TimedLaunch() {
    if (on) timing_end(s);
  }
};

}  // namespace garfield
