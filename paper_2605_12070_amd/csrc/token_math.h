// Token math of the decoupled MIS objective, shared by the row kernels and the fused
// LM-head kernels: inputs of one token, the ratios and decisions of Eq. 1-4, the per-token
// loss of Eq. 2 and the MIS weight of the Sec. 3.1 gradient.
#pragma once

#include "dppo.h"
#include "dppo_device.h"
#include "loss_stage.h"

namespace dppo {

// ---------------------------------------------------------------------------------------
// Token math shared by every row kernel (runs on one thread per row).
// ---------------------------------------------------------------------------------------
struct TokenOut {
  float lp;      // log pi_theta(y)
  float loss;    // l_t = -wd * min(r_s A, clip(r_s) A)
  float w;       // MIS weight: d L / d lp_theta = -w, dlogits = w (softmax - onehot)
  float dy;      // dlogits at v = y: w (p_y - 1) = w expm1(lp)
  uint8_t flags;
};

// Per-token inputs.
struct TokenIn {
  float lp_ref, lp_mu, adv, ts, scale;
};

__device__ __forceinline__ float row_scale(const RowArgs& a);

// Inputs of the row a workgroup works on (uniform address: scalar loads), with the call's
// scale (row_scale, the same for every row) already known.
__device__ __forceinline__ TokenIn token_inputs(const RowArgs& a, int64_t row, float scale) {
  TokenIn t;
  if (a.mode == kModeLogprob) {
    t.lp_ref = t.lp_mu = t.adv = 0.0f;
    t.ts = t.scale = 1.0f;
    return t;
  }
  t.lp_ref = a.lp_ref ? uload(a.lp_ref + row) : 0.0f;
  t.lp_mu = uload(a.lp_mu + row);
  t.adv = uload(a.adv + row);
  t.ts = a.tscale ? uload(a.tscale + row) : 1.0f;
  t.scale = scale;
  return t;
}
__device__ __forceinline__ TokenIn token_inputs(const RowArgs& a, int64_t row) {
  return token_inputs(a, row, a.mode == kModeLogprob ? 1.0f : row_scale(a));
}

__device__ __forceinline__ TokenOut token_math(const RowArgs& a, const TokenIn& t, float zy,
                                               float lse2) {
  TokenOut o;
  const float lse = lse2 * kLn2;
  const float lp = zy - lse;
  o.lp = lp;
  const float lp_mu = t.lp_mu;
  float lp_ref = t.lp_ref;
  if (a.ref_mode == DPPO_REF_LOGLINEAR) {
    // App. A: log pi_ref = alpha log mu_old + (1 - alpha) log pi_theta
    lp_ref = __builtin_fmaf(a.alpha, lp_mu, (1.0f - a.alpha) * lp);
  } else if (a.ref_mode == DPPO_REF_LINEAR) {
    // App. A: pi_ref = alpha mu_old + (1 - alpha) pi_theta, as a log-sum-exp of the two
    // weighted terms around their larger log-prob
    const float m = fmaxf(lp_mu, lp);
    lp_ref = m + logf(a.alpha * expf(lp_mu - m) + (1.0f - a.alpha) * expf(lp - m));
  }
  const float A = t.adv;
  const float ts = t.ts;
  const float scale = t.scale;
  // Eq. 1 / Sec. 3.2: r_s = pi_theta / pi_ref, r_d = pi_ref / mu_old.
  const float r_s = expf(lp - lp_ref);
  const float r_d = expf(lp_ref - lp_mu);
  // Eq. 4 band (inclusive) and Eq. 3 sign-dependent PPO mask (inclusive).
  const bool band = (a.band_lo <= r_d) && (r_d <= a.band_hi);
  const bool ppo = ((A >= 0.0f) && (r_s <= a.clip_hi)) || ((A < 0.0f) && (r_s >= a.clip_lo));
  float wd;
  bool gate;
  switch (a.rd_mode) {
    case DPPO_RD_NONE: wd = 1.0f; gate = ppo; break;
    case DPPO_RD_MASK: wd = band ? 1.0f : 0.0f; gate = ppo && band; break;
    case DPPO_RD_WEIGHT: wd = r_d; gate = ppo; break;
    default: wd = band ? r_d : 0.0f; gate = ppo && band; break;
  }
  // Eq. 2 summand with numpy min semantics (NaN in, NaN out).
  const float clipped = fminf(fmaxf(r_s, a.clip_lo), a.clip_hi);
  const float sur = nan_min(r_s * A, clipped * A);
  o.loss = -wd * sur;
  const float s = scale * ts;
  o.w = gate ? s * wd * r_s * A : 0.0f;
  o.dy = o.w * expm1f(lp);
  o.flags = (uint8_t)(DPPO_FLAG_VALID | (band ? DPPO_FLAG_BAND : 0u) | (ppo ? DPPO_FLAG_PPO : 0u));
  return o;
}

__device__ __forceinline__ float row_scale(const RowArgs& a) {
  if (a.scale_mode == DPPO_SCALE_TOKEN_MEAN) {
    // written by the count kernel before this one; constant while this kernel runs
    const int n = uload(a.stats + DPPO_STAT_N_VALID);
    return a.loss_scale / (float)(n > 1 ? n : 1);
  }
  return a.loss_scale;
}

// A workgroup's counters, kept by thread 0 over all of its rows and added to the global
// counters once, when the workgroup ends: device-scope atomics on the same five addresses
// serialise, and one per row made a batch of short rows wait on them.
struct StatCount {
  int band = 0, ppo = 0, active = 0, bad = 0;
};

__device__ __forceinline__ void count_stats(const RowArgs& a, uint8_t flags, StatCount& sc) {
  const bool band = flags & DPPO_FLAG_BAND;
  const bool ppo = flags & DPPO_FLAG_PPO;
  const bool uses_mask = a.rd_mode == DPPO_RD_MASK || a.rd_mode == DPPO_RD_MASK_WEIGHT;
  sc.band += band;
  sc.ppo += ppo;
  sc.active += ppo && (band || !uses_mask);
}

__device__ __forceinline__ void flush_stats(const RowArgs& a, const StatCount& sc) {
  if (sc.band) atomicAdd(&a.stats[DPPO_STAT_N_BAND], sc.band);
  if (sc.ppo) atomicAdd(&a.stats[DPPO_STAT_N_PPO], sc.ppo);
  if (sc.active) atomicAdd(&a.stats[DPPO_STAT_N_ACTIVE], sc.active);
  if (sc.bad) atomicAdd(&a.stats[DPPO_STAT_N_BAD], sc.bad);
}


// The same inputs for a token that differs between the threads of a wave (one token per
// thread): plain vector loads.
__device__ __forceinline__ TokenIn token_inputs_lane(const RowArgs& a, int64_t row) {
  TokenIn t;
  t.lp_ref = a.lp_ref ? a.lp_ref[row] : 0.0f;
  t.lp_mu = a.lp_mu[row];
  t.adv = a.adv[row];
  t.ts = a.tscale ? a.tscale[row] : 1.0f;
  t.scale = row_scale(a);
  return t;
}

}  // namespace dppo
