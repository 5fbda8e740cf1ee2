// Internal interface of the PPO-EWMA update kernel.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dppo {

hipError_t launch_ewma(void* xp, const void* xn, bool bf16, int64_t n, float ca, float cb,
                       bool read_old, bool aligned, hipStream_t st);

}  // namespace dppo
