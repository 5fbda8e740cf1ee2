// PPO-EWMA proxy update on a flat buffer (Sec. 5.2, Eq. 5; App. B of arXiv 2605.12070):
// x_prox <- a * x_new + b * x_prox, with the coefficients (a, b) computed on the host, or
// on the device together with the reset rule of Sec. 5.2 (ewma_controller). b = 0 means
// the old contents are not read (first step, reset). HBM-bound: one 16-byte vector per
// thread, float32 arithmetic, bf16 storage rounded to nearest even.
#include "dppo.h"
#include "dppo_device.h"
#include "ewma.h"

namespace dppo {

// x_prox <- ca x_new + cb x_prox for the 16-byte vector i (or, past the vectors, the tail
// element it stands for); the old value is not read when read_old is false.
template <bool BF16>
__device__ __forceinline__ void ewma_vec(void* xp_, const void* xn_, int64_t n, int64_t i,
                                         float ca, float cb, bool read_old) {
  constexpr int E = BF16 ? 8 : 4;  // elements per 16-byte vector
  const int64_t nvec = n / E;
  if (i < nvec) {
    u32x4* xp = (u32x4*)xp_;
    const u32x4 vn = __builtin_nontemporal_load((const u32x4*)xn_ + i);
    u32x4 vo = {0u, 0u, 0u, 0u};
    // Every byte is touched once: non-temporal loads and store (4.7 % faster on MI355X for
    // a 1 Gi-element fp32 buffer than cached x_prox accesses).
    if (read_old) vo = __builtin_nontemporal_load(xp + i);
    u32x4 out;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      if (BF16) {
        const float lo = read_old ? __builtin_fmaf(cb, bf16_lo(vo[k]), ca * bf16_lo(vn[k])) : ca * bf16_lo(vn[k]);
        const float hi = read_old ? __builtin_fmaf(cb, bf16_hi(vo[k]), ca * bf16_hi(vn[k])) : ca * bf16_hi(vn[k]);
        out[k] = pack_bf16(lo, hi);
      } else {
        const float x = __uint_as_float(vn[k]);
        const float r = read_old ? __builtin_fmaf(cb, __uint_as_float(vo[k]), ca * x) : ca * x;
        out[k] = __float_as_uint(r);
      }
    }
    __builtin_nontemporal_store(out, xp + i);
    return;
  }
  // the n % E tail elements, one per thread after the vector threads
  const int64_t e = nvec * E + (i - nvec);
  if (e >= n) return;
  if (BF16) {
    uint16_t* p = (uint16_t*)xp_;
    const float xnew = bf16_to_f32(((const uint16_t*)xn_)[e]);
    const float r = read_old ? __builtin_fmaf(cb, bf16_to_f32(p[e]), ca * xnew) : ca * xnew;
    p[e] = to_bf16(r);
  } else {
    float* p = (float*)xp_;
    const float xnew = ((const float*)xn_)[e];
    p[e] = read_old ? __builtin_fmaf(cb, p[e], ca * xnew) : ca * xnew;
  }
}

// Unaligned buffers: element e alone.
template <bool BF16>
__device__ __forceinline__ void ewma_elem(void* xp_, const void* xn_, int64_t e, float ca,
                                          float cb, bool read_old) {
  if (BF16) {
    uint16_t* p = (uint16_t*)xp_;
    const float xnew = bf16_to_f32(((const uint16_t*)xn_)[e]);
    const float r = read_old ? __builtin_fmaf(cb, bf16_to_f32(p[e]), ca * xnew) : ca * xnew;
    p[e] = to_bf16(r);
  } else {
    float* p = (float*)xp_;
    const float xnew = ((const float*)xn_)[e];
    p[e] = read_old ? __builtin_fmaf(cb, p[e], ca * xnew) : ca * xnew;
  }
}

// Host-computed coefficients.
template <bool BF16, bool READ_OLD>
__global__ __launch_bounds__(256) void ewma_kernel(void* xp_, const void* xn_,
                                                   int64_t n, float ca, float cb) {
  ewma_vec<BF16>(xp_, xn_, n, (int64_t)blockIdx.x * blockDim.x + threadIdx.x, ca, cb, READ_OLD);
}

template <bool BF16, bool READ_OLD>
__global__ __launch_bounds__(256) void ewma_kernel_scalar(void* xp_, const void* xn_, int64_t n,
                                                          float ca, float cb) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e < n) ewma_elem<BF16>(xp_, xn_, e, ca, cb, READ_OLD);
}

// Coefficients from the device-resident controller state (written by ewma_controller in
// the preceding launch on the same stream); a step that flagged an error writes nothing.
template <bool BF16>
__global__ __launch_bounds__(256) void ewma_kernel_dev(void* xp_, const void* xn_, int64_t n,
                                                       const dppo_ewma_state* s) {
  if (s->error) return;
  const float ca = s->ca, cb = s->cb;
  ewma_vec<BF16>(xp_, xn_, n, (int64_t)blockIdx.x * blockDim.x + threadIdx.x, ca, cb, cb != 0.0f);
}

template <bool BF16>
__global__ __launch_bounds__(256) void ewma_kernel_scalar_dev(void* xp_, const void* xn_,
                                                              int64_t n, const dppo_ewma_state* s) {
  if (s->error) return;
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const float ca = s->ca, cb = s->cb;
  if (e < n) ewma_elem<BF16>(xp_, xn_, e, ca, cb, cb != 0.0f);
}

// The reset rule (Sec. 5.2, App. E) and the coefficients of the recursion (App. B), in
// double as the host path computes them, from the state before the step to the state after
// it. False when w is negative or not finite (the step then changes nothing but `error`).
__device__ bool controller_step(const int32_t* stats, dppo_ewma_state& st, float beta,
                                double tau, int32_t patience, int32_t normalized) {
  if (normalized && !(__builtin_isfinite(st.w) && st.w >= 0.0)) return false;
  double rho = 1.0;
  bool fire = false;
  if (stats != nullptr) {
    rho = mask_value(stats);
    fire = reset_rule(rho, tau, patience, &st.streak);
    if (fire) st.resets += 1;
  }
  double ca, cb;
  ewma_coefficients(fire, normalized != 0, (double)beta, &st.w, &ca, &cb);
  st.last_reset = fire ? 1 : 0;
  st.error = 0;
  st.last_rho = (float)rho;
  st.ca = (float)ca;
  st.cb = (float)cb;
  return true;
}

// The controller alone, one thread; the element kernel follows on the stream.
__global__ __launch_bounds__(64) void ewma_controller(const int32_t* stats, dppo_ewma_state* s,
                                                      float beta, double tau, int32_t patience,
                                                      int32_t normalized) {
  if (threadIdx.x != 0) return;
  dppo_ewma_state st = *s;
  if (controller_step(stats, st, beta, tau, patience, normalized)) *s = st;
  else s->error = 1;
}

// Controller and update in one workgroup, for a buffer of at most kStepOneGroup elements
// (a per-token proxy): thread 0 runs the controller and stores the new state (no other
// workgroup reads it), then the workgroup applies the coefficients, four 16-byte vectors
// (or elements) per thread in flight.
template <bool BF16, bool VEC>
__global__ __launch_bounds__(1024) void ewma_step_group(void* xp_, const void* xn_, int64_t n,
                                                        const int32_t* stats,
                                                        dppo_ewma_state* s, float beta,
                                                        double tau, int32_t patience,
                                                        int32_t normalized) {
  __shared__ float coef[2];
  __shared__ int ok;
  if (threadIdx.x == 0) {
    dppo_ewma_state st = *s;
    const bool good = controller_step(stats, st, beta, tau, patience, normalized);
    if (good) *s = st;
    else s->error = 1;
    coef[0] = st.ca;
    coef[1] = st.cb;
    ok = good;
  }
  __syncthreads();
  if (!ok) return;
  const float ca = coef[0], cb = coef[1];
  constexpr int E = VEC ? (BF16 ? 8 : 4) : 1;
  const int64_t work = n / E + n % E;     // vector threads, then one per tail element
  for (int64_t i0 = threadIdx.x; i0 < work; i0 += 4 * 1024) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int64_t i = i0 + (int64_t)u * 1024;
      if (i < work) {
        if (VEC) ewma_vec<BF16>(xp_, xn_, n, i, ca, cb, cb != 0.0f);
        else ewma_elem<BF16>(xp_, xn_, i, ca, cb, cb != 0.0f);
      }
    }
  }
}

hipError_t launch_ewma(void* xp, const void* xn, bool bf16, int64_t n, float ca, float cb,
                       bool read_old, bool aligned, hipStream_t st) {
  // One thread per 16-byte vector (plus one per tail element), no grid-stride loop: on
  // MI355X this moves 6.1-6.3 TB/s on a 1 Gi-element fp32 buffer, against 4.9 TB/s for a
  // 2048-workgroup grid-stride loop and 5.7 TB/s for four vectors per thread.
  const int64_t E = aligned ? (bf16 ? 8 : 4) : 1;
  const int64_t threads = n / E + n % E;
  const int64_t blocks = (threads + 255) / 256;
  if (blocks < 1 || blocks > 0x7fffffff) return hipErrorInvalidValue;
  const dim3 g((unsigned)blocks), b(256);
  if (aligned) {
    if (bf16) {
      if (read_old) ewma_kernel<true, true><<<g, b, 0, st>>>(xp, xn, n, ca, cb);
      else ewma_kernel<true, false><<<g, b, 0, st>>>(xp, xn, n, ca, cb);
    } else {
      if (read_old) ewma_kernel<false, true><<<g, b, 0, st>>>(xp, xn, n, ca, cb);
      else ewma_kernel<false, false><<<g, b, 0, st>>>(xp, xn, n, ca, cb);
    }
  } else {
    if (bf16) {
      if (read_old) ewma_kernel_scalar<true, true><<<g, b, 0, st>>>(xp, xn, n, ca, cb);
      else ewma_kernel_scalar<true, false><<<g, b, 0, st>>>(xp, xn, n, ca, cb);
    } else {
      if (read_old) ewma_kernel_scalar<false, true><<<g, b, 0, st>>>(xp, xn, n, ca, cb);
      else ewma_kernel_scalar<false, false><<<g, b, 0, st>>>(xp, xn, n, ca, cb);
    }
  }
  return hipGetLastError();
}

hipError_t launch_ewma_step(void* xp, const void* xn, bool bf16, int64_t n, float beta,
                            double tau, int32_t patience, bool normalized, const int32_t* stats,
                            dppo_ewma_state* state, bool aligned, hipStream_t st) {
  if (n <= kStepOneGroup) {               // one launch for a small buffer
    const int32_t nz = normalized ? 1 : 0;
    if (aligned) {
      if (bf16) ewma_step_group<true, true><<<1, 1024, 0, st>>>(xp, xn, n, stats, state, beta, tau, patience, nz);
      else ewma_step_group<false, true><<<1, 1024, 0, st>>>(xp, xn, n, stats, state, beta, tau, patience, nz);
    } else {
      if (bf16) ewma_step_group<true, false><<<1, 1024, 0, st>>>(xp, xn, n, stats, state, beta, tau, patience, nz);
      else ewma_step_group<false, false><<<1, 1024, 0, st>>>(xp, xn, n, stats, state, beta, tau, patience, nz);
    }
    return hipGetLastError();
  }
  ewma_controller<<<1, 64, 0, st>>>(stats, state, beta, tau, patience, normalized ? 1 : 0);
  const int64_t E = aligned ? (bf16 ? 8 : 4) : 1;
  const int64_t threads = n / E + n % E;
  const int64_t blocks = (threads + 255) / 256;
  if (blocks < 1 || blocks > 0x7fffffff) return hipErrorInvalidValue;
  const dim3 g((unsigned)blocks), b(256);
  if (aligned) {
    if (bf16) ewma_kernel_dev<true><<<g, b, 0, st>>>(xp, xn, n, state);
    else ewma_kernel_dev<false><<<g, b, 0, st>>>(xp, xn, n, state);
  } else {
    if (bf16) ewma_kernel_scalar_dev<true><<<g, b, 0, st>>>(xp, xn, n, state);
    else ewma_kernel_scalar_dev<false><<<g, b, 0, st>>>(xp, xn, n, state);
  }
  return hipGetLastError();
}

}  // namespace dppo
