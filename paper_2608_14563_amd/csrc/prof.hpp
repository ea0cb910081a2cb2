// Launch-site hooks of the opt-in kernel timer (fpo_prof.h).
#pragma once
#include <hip/hip_runtime.h>

namespace fpo {
void prof_begin(const char* name, hipStream_t st);
void prof_end(hipStream_t st);
}  // namespace fpo

// Launch `...` (a kernel<<<>>> expression) on stream `st`, timed when enabled.
#define FPO_LAUNCH(name, st, ...)     \
  do {                                \
    ::fpo::prof_begin(name, st);      \
    __VA_ARGS__;                      \
    ::fpo::prof_end(st);              \
  } while (0)
