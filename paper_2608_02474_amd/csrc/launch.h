// Host-side launch helpers shared by the kernel files and the C ABI:
// launch-error capture and optional per-kernel event timing.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace echo {

// Per-thread kernel timing.  While enabled, a TimedLaunch records a start and
// stop event around the launch it wraps; profile_read() drains the record.
bool profile_enabled();
void profile_set(bool on);
struct TimedLaunch {
  TimedLaunch(const char* name, hipStream_t s);
  ~TimedLaunch();
  int slot;
  hipStream_t stream;
};

}  // namespace echo

// Launch `kernel<<<grid, block, lds, stream>>>(args...)` under a timing scope and
// return the launch error.
#define ECHO_LAUNCH(name, kernel, grid, block, lds, stream, ...)              \
  ([&]() -> hipError_t {                                                       \
    ::echo::TimedLaunch _tl((name), (stream));                                 \
    hipLaunchKernelGGL((kernel), (grid), (block), (lds), (stream), __VA_ARGS__); \
    return hipGetLastError();                                                  \
  }())
