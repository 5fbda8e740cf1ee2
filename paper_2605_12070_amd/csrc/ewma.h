// Internal interface of the PPO-EWMA update kernel.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "dppo.h"

namespace dppo {

hipError_t launch_ewma(void* xp, const void* xn, bool bf16, int64_t n, float ca, float cb,
                       bool read_old, bool aligned, hipStream_t st);

// Controller kernel (reset rule, coefficients) into *state, then the element kernel with
// the coefficients read from *state.
hipError_t launch_ewma_step(void* xp, const void* xn, bool bf16, int64_t n, float beta,
                            double tau, int32_t patience, bool normalized, const int32_t* stats,
                            dppo_ewma_state* state, bool aligned, hipStream_t st);

}  // namespace dppo
