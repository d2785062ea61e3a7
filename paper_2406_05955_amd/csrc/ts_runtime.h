// Host runtime helpers shared by the entry points: error capture and the
// optional per-kernel event timing.
#pragma once

#include <hip/hip_runtime.h>

#include "turbosparse.h"

namespace ts {

// Stores the message of a failed HIP call for ts_last_error().
void set_last_error(const char *where, hipError_t e);

// Returns TS_ERR_HIP (after recording the message) if a launch failed.
ts_status check_launch(const char *where);

// While profiling is enabled, brackets one kernel launch with an event pair
// recorded on `stream`.
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
