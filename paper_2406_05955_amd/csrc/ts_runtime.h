// Host runtime helpers shared by the entry points: error capture and the
// optional per-kernel event timing.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include "turbosparse.h"

namespace ts {

// Stores the message of a failed HIP call for ts_last_error().
void set_last_error(const char *where, hipError_t e);

// Stores a message of the library's own for ts_last_error().
void set_last_message(const char *msg);

// Returns TS_ERR_HIP (after recording the message) if a launch failed.
ts_status check_launch(const char *where);

// While profiling is enabled, hands out an event pair registered under
// `kernel` (false otherwise).
bool prof_events(const char *kernel, hipEvent_t *start, hipEvent_t *stop);

// Launches `kernel` on `stream`.  While profiling is enabled the launch
// carries an event pair that the runtime stamps when the kernel itself
// starts and ends (hipExtLaunchKernel), so the recorded time excludes the
// queueing around it.
template <typename... Args, typename F = void (*)(Args...)>
void launch(const char *name, F kernel, dim3 grid, dim3 block, hipStream_t stream, Args... args) {
    hipEvent_t e0 = nullptr, e1 = nullptr;
    if (prof_events(name, &e0, &e1))
        hipExtLaunchKernelGGL(kernel, grid, block, 0, stream, e0, e1, 0, args...);
    else
        hipLaunchKernelGGL(kernel, grid, block, 0, stream, args...);
}

// While profiling is enabled, brackets a sequence of launches with an event
// pair recorded on `stream`.
class ProfScope {
  public:
    ProfScope(const char *kernel, hipStream_t stream);
    ~ProfScope();
    ProfScope(const ProfScope &) = delete;
    ProfScope &operator=(const ProfScope &) = delete;

  private:
    int slot_ = -1;
    hipStream_t stream_;
};

}  // namespace ts
