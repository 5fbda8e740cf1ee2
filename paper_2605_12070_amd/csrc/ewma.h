// Internal interface of the PPO-EWMA update kernel.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "dppo.h"

namespace dppo {

// rho_t = n_active / n_valid, the kept fraction behind the automatic reset (Sec. 5.2;
// App. E); 1 when no token is valid.
__host__ __device__ inline double mask_value(const int32_t* stats) {
  const int32_t nv = stats[DPPO_STAT_N_VALID];
  return nv == 0 ? 1.0 : (double)stats[DPPO_STAT_N_ACTIVE] / (double)nv;
}

// The reset rule (Sec. 5.2; App. E): the streak counts consecutive steps with rho_t < tau
// (compared in double); a reset fires once the streak reaches `patience`, and the streak
// then restarts at 0. The host export and the device controller both call this.
__host__ __device__ inline bool reset_rule(double rho, double tau, int32_t patience,
                                           int32_t* streak) {
  *streak = rho < tau ? *streak + 1 : 0;
  const bool fire = *streak >= patience;
  if (fire) *streak = 0;
  return fire;
}

// Coefficients of x_prox <- ca x_new + cb x_prox for one step, in double (Eq. 5; App. B):
// a reset copies x_new (and sets w = 1); the normalised form has w_t = 1 + beta w_{t-1},
// ca = 1 / w_t, cb = beta w_{t-1} / w_t; the fixed form has ca = 1 - beta, cb = beta.
// *w is w_{t-1} on entry and w_t on return (untouched by the fixed form).
__host__ __device__ inline void ewma_coefficients(bool reset, bool normalized, double beta,
                                                  double* w, double* ca, double* cb) {
  if (reset) {
    *ca = 1.0;
    *cb = 0.0;
    if (normalized) *w = 1.0;
  } else if (normalized) {
    const double wp = *w;
    *w = 1.0 + beta * wp;
    *ca = 1.0 / *w;
    *cb = beta * wp / *w;
  } else {
    *ca = 1.0 - beta;
    *cb = beta;
  }
}

hipError_t launch_ewma(void* xp, const void* xn, bool bf16, int64_t n, float ca, float cb,
                       bool read_old, bool aligned, hipStream_t st);

// Buffers of up to this many elements (per-token proxies) take one one-workgroup launch
// that runs the controller and the update (the tiny configuration's step 37.0 -> 25.3 us,
// small_vocab's 128.0 -> 126.1 us); larger ones take the controller kernel and then the
// element kernel.
constexpr int64_t kStepOneGroup = 16384;

// Controller kernel (reset rule, coefficients) into *state, then the element kernel with
// the coefficients read from *state; one launch that does both for a small buffer.
hipError_t launch_ewma_step(void* xp, const void* xn, bool bf16, int64_t n, float beta,
                            double tau, int32_t patience, bool normalized, const int32_t* stats,
                            dppo_ewma_state* state, bool aligned, hipStream_t st);

}  // namespace dppo
