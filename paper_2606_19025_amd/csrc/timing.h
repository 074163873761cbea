// Optional per-launch timing of the library's kernels (moe_timing_* in the
// public header).  When enabled, every kernel launch is bracketed by a pair of
// events taken from a pool created by moe_timing_enable().
#pragma once
#include <hip/hip_runtime.h>

namespace moe {
bool timing_on();
void timing_begin(const char* name, hipStream_t s);
void timing_end(hipStream_t s);
}  // namespace moe

#define MOE_TIMED(name, stream, ...)                   \
  do {                                                 \
    const bool moe_t_ = moe::timing_on();              \
    if (moe_t_) moe::timing_begin(name, stream);       \
    __VA_ARGS__;                                       \
    if (moe_t_) moe::timing_end(stream);               \
  } while (0)
