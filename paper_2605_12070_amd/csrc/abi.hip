// C-ABI layer: argument checks (all on the host, before any HIP call), kernel selection,
// launches on the caller's stream, error reporting and the profiling timer.
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <algorithm>
#include <cstring>
#include <mutex>
#include <string>
#include <utility>
#include <vector>

#include "dppo.h"
#include "ewma.h"
#include "lm_head.h"
#include "vocab_shard.h"
#include "loss_stage.h"


namespace {

thread_local std::string g_last_error;
int g_path_policy = dppo::kForceAuto;
// Path-policy bit: loss calls count with prep_stats and atomics even where count mode applies.
constexpr int kPolicyAtomicCounts = 2;

dppo_status fail(dppo_status s, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
dppo_status fail(dppo_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return s;
}

dppo_status hip_fail(hipError_t e, const char* what) {
  return fail(DPPO_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

int esize_of(int32_t dtype) { return dtype == DPPO_BF16 ? 2 : 4; }

// [begin, end) byte range of a [T, ld] matrix whose rows hold V used elements.
std::pair<uintptr_t, uintptr_t> span_of(const void* base, int64_t T, int64_t V, int64_t ld, int es) {
  const uintptr_t b = (uintptr_t)base;
  return {b, b + (uintptr_t)(((T - 1) * ld + V) * es)};
}

bool overlaps(std::pair<uintptr_t, uintptr_t> a, std::pair<uintptr_t, uintptr_t> b) {
  return a.first < b.second && b.first < a.second;
}

// ------------------------------------------------------------------ kernel timer
struct KernelTimer {
  std::mutex mu;
  bool on = false;
  std::vector<std::pair<hipEvent_t, hipEvent_t>> pool;
  size_t used = 0;
};
KernelTimer g_timer;

// Returns the event pair to record around the next launch, or nullptr when disabled.
std::pair<hipEvent_t, hipEvent_t>* timer_slot() {
  std::lock_guard<std::mutex> lk(g_timer.mu);
  if (!g_timer.on) return nullptr;
  if (g_timer.used == g_timer.pool.size()) {
    hipEvent_t a, b;
    if (hipEventCreate(&a) != hipSuccess) return nullptr;
    if (hipEventCreate(&b) != hipSuccess) {
      (void)hipEventDestroy(a);
      return nullptr;
    }
    g_timer.pool.emplace_back(a, b);
  }
  return &g_timer.pool[g_timer.used++];
}

// Workgroups of `fn` that fit on the current device at once (CUs x per-CU occupancy),
// cached per (device, kernel).

hipError_t resident_slots(const dppo::RowLaunch& L, int64_t* slots) {
  static std::mutex mu;
  static std::vector<std::pair<std::pair<int, const void*>, int64_t>> cache;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lk(mu);
  for (auto& kv : cache) {
    if (kv.first.first == dev && kv.first.second == (const void*)L.fn) {
      *slots = kv.second;
      return hipSuccess;
    }
  }
  int cus = 0, per_cu = 0;
  e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, (const void*)L.fn, L.threads, 0);
  if (e != hipSuccess) return e;
  *slots = (int64_t)cus * (per_cu > 0 ? per_cu : 1);
  cache.push_back({{dev, (const void*)L.fn}, *slots});
  return hipSuccess;
}

dppo_status launch_rows(const dppo::RowLaunch& L, const dppo::RowArgsV& args, int64_t T,
                        hipStream_t st) {
  int64_t grid = T;
  if (L.persistent) {
    int64_t slots = 0;
    const hipError_t oe = resident_slots(L, &slots);
    if (oe != hipSuccess) return hip_fail(oe, "occupancy query");
    // L.fill of every 32 slots: with every CU streaming, a row kernel moves fewer bytes per
    // second than with a few CUs of each 32-CU XCD idle (the fill is chosen per kernel).
    slots = slots * L.fill / 32;
    if (slots < 1) slots = 1;
    if (slots < grid) grid = slots;
  }
  dppo::RowArgsV a = args;
  a.stagger = L.stagger;
  auto* ev = timer_slot();
  if (ev) (void)hipEventRecord(ev->first, st);
  // Gradient kernels take the RowArgs part alone, the others the whole RowArgsV.
  const void* karg = L.bwd ? (const void*)static_cast<const dppo::RowArgs*>(&a) : (const void*)&a;
  void* kargs[] = {const_cast<void*>(karg)};
  hipError_t e = hipLaunchKernel((const void*)L.fn, dim3((unsigned)grid), dim3((unsigned)L.threads),
                                 kargs, 0, st);
  if (e == hipSuccess) e = hipGetLastError();
  if (ev) (void)hipEventRecord(ev->second, st);
  if (e != hipSuccess) return hip_fail(e, "row kernel launch");
  return DPPO_OK;
}

dppo_status check_matrix(const void* p, int32_t dtype, int64_t T, int64_t V, int64_t ld,
                         const char* name) {
  if (dtype != DPPO_F32 && dtype != DPPO_BF16)
    return fail(DPPO_ERR_INVALID_ARG, "unknown dtype %d", (int)dtype);
  if (T < 0 || T > 0x7FFFFFFF) return fail(DPPO_ERR_INVALID_ARG, "T = %lld out of [0, 2^31)", (long long)T);
  if (V < 1 || V > 0x7FFFFFFF) return fail(DPPO_ERR_INVALID_ARG, "V = %lld out of [1, 2^31)", (long long)V);
  if (ld < V) return fail(DPPO_ERR_INVALID_ARG, "%s stride %lld < V = %lld", name, (long long)ld, (long long)V);
  if (T > 0 && p == nullptr) return fail(DPPO_ERR_INVALID_ARG, "%s is NULL", name);
  return DPPO_OK;
}

struct LmhLayout {
  int64_t part, zy, w, lse2, dy, ev, g, total;  // byte offsets into the workspace, and its size
  int64_t chunk, ldg;                        // vocabulary rows per backward chunk, g's stride
  bool one_pass;                             // G from the forward tiles' exponentials
};

int64_t align256(int64_t x) { return (x + 255) & ~(int64_t)255; }

// Workspace of the fused LM head. With vocab_chunk <= 0 or >= V (one pass) g holds the
// forward tiles' fp16 exponentials for the whole vocabulary, [T, ldg] with ldg = V rounded
// up to the tile width, and becomes G in place; otherwise g holds one bf16 chunk of G,
// [T, chunk] with chunk rounded up to the tile width.
LmhLayout lmh_layout(int64_t T, int64_t V, int64_t vocab_chunk) {
  LmhLayout L;
  const int64_t ngroups = dppo::lmh_groups((int)V);
  const int64_t vpad = ((V + dppo::LMH_BN - 1) / dppo::LMH_BN) * dppo::LMH_BN;
  L.one_pass = vocab_chunk <= 0 || vocab_chunk >= V;
  int64_t chunk = L.one_pass ? vpad : ((vocab_chunk + dppo::LMH_BN - 1) / dppo::LMH_BN) * dppo::LMH_BN;
  if (chunk > vpad) chunk = vpad;
  L.chunk = L.one_pass ? V : chunk;
  L.ldg = chunk;
  int64_t o = 0;
  L.part = o; o = align256(o + ngroups * T * 2 * 4);
  L.zy = o;   o = align256(o + T * 4);
  L.w = o;    o = align256(o + T * 4);
  L.lse2 = o; o = align256(o + T * 4);
  L.dy = o;   o = align256(o + T * 4);
  L.ev = o;   o = align256(o + T);
  L.g = o;    o = align256(o + T * L.ldg * 2);
  L.total = o;
  return L;
}

// Parameters and per-token pointers shared by the loss entry points.
dppo_status check_token_args(const dppo_params* p, int64_t T, const int64_t* token_ids,
                             const float* logp_mu_old, const float* logp_ref,
                             const float* advantages, const float* logp_out,
                             const float* loss_tok_out) {
  if (p->ref_mode < DPPO_REF_GIVEN || p->ref_mode > DPPO_REF_LINEAR)
    return fail(DPPO_ERR_INVALID_ARG, "unknown ref_mode %d", (int)p->ref_mode);
  if (p->ref_mode != DPPO_REF_GIVEN && !(p->alpha > 0.0f && p->alpha < 1.0f))
    return fail(DPPO_ERR_INVALID_ARG, "alpha = %g must lie in (0, 1) for an interpolated reference",
                p->alpha);
  if (T > 0 && (!token_ids || !logp_mu_old || !advantages || !logp_out || !loss_tok_out))
    return fail(DPPO_ERR_INVALID_ARG,
                "token_ids, logp_mu_old, advantages, logp_out, loss_tok_out are required");
  if (T > 0 && p->ref_mode == DPPO_REF_GIVEN && !logp_ref)
    return fail(DPPO_ERR_INVALID_ARG, "logp_ref is required with ref_mode GIVEN");
  if (std::isnan(p->band_lo) || std::isnan(p->band_hi) || p->band_lo < 0.0f || p->band_lo > p->band_hi)
    return fail(DPPO_ERR_INVALID_ARG, "band [%g, %g] must satisfy 0 <= lo <= hi", p->band_lo, p->band_hi);
  if (!(p->clip_eps_lo >= 0.0f) || !(p->clip_eps_hi >= 0.0f) || !std::isfinite(p->clip_eps_lo) ||
      !std::isfinite(p->clip_eps_hi))
    return fail(DPPO_ERR_INVALID_ARG, "clip eps (%g, %g) must be finite and >= 0", p->clip_eps_lo, p->clip_eps_hi);
  if (!std::isfinite(p->loss_scale)) return fail(DPPO_ERR_INVALID_ARG, "loss_scale must be finite");
  if (p->rd_mode < DPPO_RD_NONE || p->rd_mode > DPPO_RD_MASK_WEIGHT)
    return fail(DPPO_ERR_INVALID_ARG, "unknown rd_mode %d", (int)p->rd_mode);
  if (p->scale_mode != DPPO_SCALE_CONST && p->scale_mode != DPPO_SCALE_TOKEN_MEAN)
    return fail(DPPO_ERR_INVALID_ARG, "unknown scale_mode %d", (int)p->scale_mode);
  return DPPO_OK;
}

}  // namespace

extern "C" {

const char* dppo_strerror(dppo_status s) {
  switch (s) {
    case DPPO_OK: return "success";
    case DPPO_ERR_INVALID_ARG: return "invalid argument";
    case DPPO_ERR_UNSUPPORTED: return "unsupported request";
    case DPPO_ERR_HIP: return "HIP runtime error";
  }
  return "unknown status";
}

const char* dppo_last_error(void) { return g_last_error.c_str(); }

int32_t dppo_abi_version(void) { return DPPO_ABI_VERSION; }

dppo_status dppo_set_path_policy(int32_t policy) {
  if (policy < 0 || policy > (dppo::kForceStream | kPolicyAtomicCounts))
    return fail(DPPO_ERR_INVALID_ARG, "unknown path policy %d", (int)policy);
  g_path_policy = policy;
  return DPPO_OK;
}

dppo_status dppo_timer_enable(int32_t on) {
  std::lock_guard<std::mutex> lk(g_timer.mu);
  if (!on) {
    for (auto& pr : g_timer.pool) {
      (void)hipEventDestroy(pr.first);
      (void)hipEventDestroy(pr.second);
    }
    g_timer.pool.clear();
  }
  g_timer.used = 0;
  g_timer.on = on != 0;
  return DPPO_OK;
}

dppo_status dppo_timer_read(double* total_ms, int64_t* launches) {
  if (!total_ms || !launches) return fail(DPPO_ERR_INVALID_ARG, "dppo_timer_read: NULL output");
  std::lock_guard<std::mutex> lk(g_timer.mu);
  double acc = 0.0;
  for (size_t i = 0; i < g_timer.used; ++i) {
    hipError_t e = hipEventSynchronize(g_timer.pool[i].second);
    if (e != hipSuccess) return hip_fail(e, "timer event sync");
    float ms = 0.0f;
    e = hipEventElapsedTime(&ms, g_timer.pool[i].first, g_timer.pool[i].second);
    if (e != hipSuccess) return hip_fail(e, "timer elapsed");
    acc += ms;
  }
  *total_ms = acc;
  *launches = (int64_t)g_timer.used;
  g_timer.used = 0;
  return DPPO_OK;
}

const char* dppo_row_kernel_name(int32_t dtype, int64_t V, int64_t ld, int32_t with_dlogits) {
  if ((dtype != DPPO_F32 && dtype != DPPO_BF16) || V < 1 || ld < V) return nullptr;
  const bool aligned = (ld * esize_of(dtype)) % 16 == 0;
  const dppo::RowLaunch L =
      dppo::select_row_kernel(dtype, V, aligned, with_dlogits != 0, g_path_policy, true);
  thread_local char buf[96];
  const char* ty = dtype == DPPO_BF16 ? "bf16" : "f32";
  const char* bw = with_dlogits ? "true" : "false";
  if (L.prefix)
    snprintf(buf, sizeof(buf), "dppo::rows_%s_prefix<%d, %d>", ty, L.threads, L.chunks);
  else if (L.phase && !with_dlogits)
    snprintf(buf, sizeof(buf), "dppo::rows_bf16_fwd_phase<%d, %d>", L.threads, L.chunks);
  else if (L.phase && L.two_buffers)
    snprintf(buf, sizeof(buf), "dppo::rows_bf16_phase_db<%d, %d>", L.threads, L.chunks);
  else if (L.phase)
    snprintf(buf, sizeof(buf), "dppo::rows_bf16_phase<%d, %d, true>", L.threads, L.chunks);
  else if (L.resident && dtype == DPPO_BF16 && !with_dlogits)
    snprintf(buf, sizeof(buf), "dppo::rows_bf16_fwd<%d, %d>", L.threads, L.chunks);
  else if (L.two_buffers)
    snprintf(buf, sizeof(buf), "dppo::rows_bf16_resident_db<%d, %d>", L.threads, L.chunks);
  else if (L.resident)
    snprintf(buf, sizeof(buf), "dppo::rows_%s_resident<%d, %d, %s>", ty, L.threads, L.chunks, bw);
  else
    snprintf(buf, sizeof(buf), "dppo::rows_stream<%s, %d, %s, %s>",
             dtype == DPPO_BF16 ? "unsigned short" : "float", L.threads, bw, aligned ? "true" : "false");
  return buf;
}

dppo_status dppo_effective_thresholds(double mask_lo, double mask_hi, double clip_lo,
                                      double clip_hi, double alpha, int32_t ref_mode,
                                      double* out) {
  if (!out) return fail(DPPO_ERR_INVALID_ARG, "dppo_effective_thresholds: NULL out");
  if (ref_mode != DPPO_REF_LOGLINEAR && ref_mode != DPPO_REF_LINEAR)
    return fail(DPPO_ERR_INVALID_ARG, "ref_mode %d is not an interpolated reference", (int)ref_mode);
  if (!(alpha > 0.0 && alpha < 1.0)) return fail(DPPO_ERR_INVALID_ARG, "alpha = %g not in (0, 1)", alpha);
  if (!(mask_lo >= 0.0 && mask_lo <= mask_hi) || !(clip_lo >= 0.0 && clip_lo <= clip_hi))
    return fail(DPPO_ERR_INVALID_ARG, "bounds must satisfy 0 <= lo <= hi");
  if (ref_mode == DPPO_REF_LOGLINEAR) {
    // r_d = r^(1 - alpha) and r_s = r^alpha are increasing in r: invert each bound.
    out[0] = std::pow(mask_lo, 1.0 / (1.0 - alpha));
    out[1] = std::pow(mask_hi, 1.0 / (1.0 - alpha));
    out[2] = std::pow(clip_lo, 1.0 / alpha);
    out[3] = std::pow(clip_hi, 1.0 / alpha);
  } else {
    // r_d = alpha + (1 - alpha) r is linear in r; r_s = r / (alpha + (1 - alpha) r) rises
    // from 0 towards 1 / (1 - alpha), so r_s = b has the root alpha b / (1 - (1 - alpha) b)
    // only below that limit; at or above it the bound is never reached.
    out[0] = (mask_lo - alpha) / (1.0 - alpha);
    out[1] = (mask_hi - alpha) / (1.0 - alpha);
    const double lim = 1.0 / (1.0 - alpha);
    out[2] = clip_lo < lim ? alpha * clip_lo / (1.0 - (1.0 - alpha) * clip_lo) : INFINITY;
    out[3] = clip_hi < lim ? alpha * clip_hi / (1.0 - (1.0 - alpha) * clip_hi) : INFINITY;
  }
  return DPPO_OK;
}

dppo_status dppo_beta_from_window(double window, double* beta) {
  if (!beta) return fail(DPPO_ERR_INVALID_ARG, "dppo_beta_from_window: NULL beta");
  if (!(window >= 0.0) || !std::isfinite(window))
    return fail(DPPO_ERR_INVALID_ARG, "staleness window %g must be finite and >= 0", window);
  *beta = window / (window + 2.0);
  return DPPO_OK;
}

dppo_status dppo_train_infer_mask_value(const int32_t* stats, double* rho) {
  if (!stats || !rho) return fail(DPPO_ERR_INVALID_ARG, "dppo_train_infer_mask_value: NULL pointer");
  *rho = dppo::mask_value(stats);
  return DPPO_OK;
}

dppo_status dppo_ppo_clip_ratio(const int32_t* stats, double* ratio) {
  if (!stats || !ratio) return fail(DPPO_ERR_INVALID_ARG, "dppo_ppo_clip_ratio: NULL pointer");
  const int32_t nv = stats[DPPO_STAT_N_VALID];
  *ratio = nv == 0 ? 0.0 : 1.0 - (double)stats[DPPO_STAT_N_PPO] / (double)nv;
  return DPPO_OK;
}

dppo_status dppo_reset_decision(const int32_t* stats, double tau, int32_t patience,
                                int32_t* streak, double* rho, int32_t* fire) {
  if (!streak || !fire) return fail(DPPO_ERR_INVALID_ARG, "dppo_reset_decision: NULL streak or fire");
  if (!std::isfinite(tau)) return fail(DPPO_ERR_INVALID_ARG, "tau = %g is not finite", tau);
  if (patience < 1) return fail(DPPO_ERR_INVALID_ARG, "patience = %d < 1", (int)patience);
  if (*streak < 0) return fail(DPPO_ERR_INVALID_ARG, "streak = %d < 0", (int)*streak);
  double r = 1.0;
  bool f = false;
  if (stats) {
    r = dppo::mask_value(stats);
    f = dppo::reset_rule(r, tau, patience, streak);
  }
  if (rho) *rho = r;
  *fire = f ? 1 : 0;
  return DPPO_OK;
}

dppo_status logprob_fwd(const void* logits, int32_t dtype, int64_t T, int64_t V, int64_t ld,
                        const int64_t* token_ids, float* logp_out, float* lse_out, void* stream) {
  dppo_status s = check_matrix(logits, dtype, T, V, ld, "logits");
  if (s != DPPO_OK) return s;
  if (T > 0 && (!token_ids || !logp_out))
    return fail(DPPO_ERR_INVALID_ARG, "logprob_fwd: token_ids and logp_out are required");
  if (T == 0) return DPPO_OK;
  const int es = esize_of(dtype);
  const bool aligned = aligned16(logits) && ((ld * es) % 16 == 0);
  const dppo::RowLaunch L = dppo::select_row_kernel(dtype, V, aligned, false, g_path_policy,
                                                    ((uintptr_t)logits & 1) == 0);
  dppo::RowArgsV a{};
  a.logits = logits;
  a.ld = ld;
  a.ids = token_ids;
  a.lp_out = logp_out;
  a.lse_out = lse_out;
  a.T = (int32_t)T;
  a.V = (int32_t)V;
  a.mode = dppo::kModeLogprob;
  return launch_rows(L, a, T, (hipStream_t)stream);
}

dppo_status logprob_fwd_versioned(const void* const* logits, int32_t K, int32_t dtype, int64_t T,
                                  int64_t V, int64_t ld, const int32_t* version_ids,
                                  const int64_t* token_ids, float* logp_out, float* lse_out,
                                  void* stream) {
  if (K < 1 || K > DPPO_MAX_VERSIONS)
    return fail(DPPO_ERR_INVALID_ARG, "K = %d versions out of [1, %d]", (int)K, DPPO_MAX_VERSIONS);
  if (T > 0 && !logits) return fail(DPPO_ERR_INVALID_ARG, "logits pointer array is NULL");
  for (int v = 0; v < K && T > 0; ++v) {
    dppo_status s = check_matrix(logits[v], dtype, T, V, ld, "logits[v]");
    if (s != DPPO_OK) return s;
  }
  if (T == 0) {
    dppo_status s = check_matrix(nullptr, dtype, T, V, ld, "logits");
    return s;
  }
  if (!version_ids || !token_ids || !logp_out)
    return fail(DPPO_ERR_INVALID_ARG, "version_ids, token_ids and logp_out are required");
  const int es = esize_of(dtype);
  bool aligned = (ld * es) % 16 == 0;
  bool even = true;
  for (int v = 0; v < K; ++v) {
    aligned = aligned && aligned16(logits[v]);
    even = even && ((uintptr_t)logits[v] & 1) == 0;
  }
  dppo::RowLaunch L = dppo::select_row_kernel(dtype, V, aligned, false, g_path_policy, even);
  // Rows gathered from several versions' logits want every slot of the device: at
  // 1024 x 19 (bf16, V = 151936, 4 versions) 32 of 32 slots took 0.753-0.757 ms against
  // 0.762-0.768 ms with the 30 that suit one matrix (same-box sweep).
  if (K > 1 && dtype == DPPO_BF16 && L.resident && L.threads == 1024 && L.chunks == 19) L.fill = 32;
  dppo::RowArgsV a{};
  a.logits = logits[0];
  a.version = version_ids;
  a.nver = K;
  for (int v = 0; v < K; ++v) a.vlogits[v] = logits[v];
  a.ld = ld;
  a.ids = token_ids;
  a.lp_out = logp_out;
  a.lse_out = lse_out;
  a.T = (int32_t)T;
  a.V = (int32_t)V;
  a.mode = dppo::kModeLogprob;
  return launch_rows(L, a, T, (hipStream_t)stream);
}

dppo_status decoupled_ppo_loss_fwd_bwd(
    const void* logits, int32_t dtype, int64_t T, int64_t V, int64_t ld,
    const int64_t* token_ids, const float* logp_mu_old, const float* logp_ref,
    const float* advantages, const uint8_t* loss_mask, const float* token_scale,
    const dppo_params* p, float* logp_out, float* loss_tok_out, float* loss_out,
    uint8_t* flags_out, void* dlogits, int64_t ld_dlogits, int32_t* stats_out, void* stream) {
  dppo_status s = check_matrix(logits, dtype, T, V, ld, "logits");
  if (s != DPPO_OK) return s;
  if (!p) return fail(DPPO_ERR_INVALID_ARG, "params pointer is NULL");
  if (!loss_out || !stats_out) return fail(DPPO_ERR_INVALID_ARG, "loss_out and stats_out are required");
  s = check_token_args(p, T, token_ids, logp_mu_old, logp_ref, advantages, logp_out, loss_tok_out);
  if (s != DPPO_OK) return s;
  const int es = esize_of(dtype);
  if (dlogits && T > 0) {
    if (ld_dlogits < V)
      return fail(DPPO_ERR_INVALID_ARG, "dlogits stride %lld < V = %lld", (long long)ld_dlogits, (long long)V);
    const bool same = dlogits == logits && ld_dlogits == ld;
    if (!same && overlaps(span_of(logits, T, V, ld, es), span_of(dlogits, T, V, ld_dlogits, es)))
      return fail(DPPO_ERR_INVALID_ARG, "dlogits overlaps logits without aliasing them exactly");
  }
  hipStream_t st = (hipStream_t)stream;
  dppo::RowLaunch L;
  if (T > 0) {
    const bool aligned = aligned16(logits) && ((ld * es) % 16 == 0) &&
                         (!dlogits || (aligned16(dlogits) && (ld_dlogits * es) % 16 == 0));
    // rows with a phase: dlogits row t must start at logits row t's offset within 16 bytes
    const bool phase_ok =
        ((uintptr_t)logits & 1) == 0 &&
        (!dlogits || ((((uintptr_t)dlogits - (uintptr_t)logits) & 15) == 0 &&
                      (ld_dlogits - ld) % 8 == 0));
    L = dppo::select_row_kernel(dtype, V, aligned, dlogits != nullptr, g_path_policy, phase_ok);
  }
  // Count mode: a persistent fp32 resident row kernel on a batch short enough for every
  // workgroup to read the mask counts the valid tokens itself and loss_sum takes the
  // counters from the flags, so prep_stats does not run (one launch fewer per call: the
  // tiny configuration's step 40.6 -> 36.6 us).
  const bool count_mode = T > 0 && T <= dppo::kCountModeMaxT && L.persistent && L.counts &&
                          flags_out != nullptr && !(g_path_policy & kPolicyAtomicCounts);
  hipError_t e = hipSuccess;
  if (!count_mode) {
    dppo::launch_prep_stats(loss_mask, T, stats_out, st);
    e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, "prep_stats launch");
  }
  if (T > 0) {
    dppo::RowArgsV a{};
    a.logits = logits;
    a.ld = ld;
    a.dlogits = dlogits;
    a.ldd = ld_dlogits;
    a.ids = token_ids;
    a.lp_mu = logp_mu_old;
    a.lp_ref = p->ref_mode == DPPO_REF_GIVEN ? logp_ref : nullptr;
    a.ref_mode = p->ref_mode;
    a.alpha = p->alpha;
    a.adv = advantages;
    a.mask = loss_mask;
    a.tscale = token_scale;
    a.lp_out = logp_out;
    a.loss_tok = loss_tok_out;
    a.flags = flags_out;
    a.stats = stats_out;
    a.T = (int32_t)T;
    a.V = (int32_t)V;
    a.mode = dppo::kModeLoss;
    a.band_lo = p->band_lo;
    a.band_hi = p->band_hi;
    a.clip_lo = 1.0f - p->clip_eps_lo;
    a.clip_hi = 1.0f + p->clip_eps_hi;
    a.loss_scale = p->loss_scale;
    a.rd_mode = p->rd_mode;
    a.scale_mode = p->scale_mode;
    a.count_mode = count_mode ? 1 : 0;
    s = launch_rows(L, a, T, st);
    if (s != DPPO_OK) return s;
  }
  dppo::launch_loss_sum(loss_tok_out, loss_mask, token_scale, stats_out, T, p->loss_scale,
                        p->scale_mode, loss_out, st, count_mode ? flags_out : nullptr,
                        p->rd_mode);
  e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, "loss_sum launch");
  return DPPO_OK;
}

int64_t fused_lm_head_workspace_bytes(int64_t T, int64_t d, int64_t V, int64_t vocab_chunk) {
  if (T < 0 || d < 8 || V < 1 || T >= ((int64_t)1 << 31) || V > ((int64_t)1 << 21)) return -1;
  return lmh_layout(T, V, vocab_chunk).total;
}

dppo_status fused_lm_head_loss_fwd_bwd(
    const void* hidden, const void* weight, int32_t dtype, int64_t T, int64_t d, int64_t V,
    const int64_t* token_ids, const float* logp_mu_old, const float* logp_ref,
    const float* advantages, const uint8_t* loss_mask, const float* token_scale,
    const dppo_params* p, float* logp_out, float* loss_tok_out, float* loss_out,
    uint8_t* flags_out, int32_t* stats_out, float* dhidden, float* dweight,
    int64_t vocab_chunk, void* workspace, int64_t workspace_bytes, void* stream) {
  if (dtype != DPPO_BF16 && dtype != DPPO_F32)
    return fail(DPPO_ERR_INVALID_ARG, "unknown dtype %d", (int)dtype);
  if (dtype != DPPO_BF16)
    return fail(DPPO_ERR_UNSUPPORTED, "the fused LM head takes bf16 hidden states and weights");
  if (T < 0 || T >= ((int64_t)1 << 31)) return fail(DPPO_ERR_INVALID_ARG, "T = %lld out of range", (long long)T);
  if (V < 1 || V > ((int64_t)1 << 21)) return fail(DPPO_ERR_INVALID_ARG, "V = %lld out of [1, 2^21]", (long long)V);
  if (d < 8 || d % 8 != 0 || d > (1 << 20))
    return fail(DPPO_ERR_INVALID_ARG, "d = %lld must be a multiple of 8 in [8, 2^20]", (long long)d);
  if (!p) return fail(DPPO_ERR_INVALID_ARG, "params pointer is NULL");
  if (!loss_out || !stats_out) return fail(DPPO_ERR_INVALID_ARG, "loss_out and stats_out are required");
  if (!weight || !aligned16(weight) || (T > 0 && (!hidden || !aligned16(hidden))))
    return fail(DPPO_ERR_INVALID_ARG, "hidden and weight must be non-NULL and 16-byte aligned");
  dppo_status s = check_token_args(p, T, token_ids, logp_mu_old, logp_ref, advantages, logp_out,
                                   loss_tok_out);
  if (s != DPPO_OK) return s;
  const LmhLayout L = lmh_layout(T, V, vocab_chunk);
  if (T > 0 && (!workspace || workspace_bytes < L.total))
    return fail(DPPO_ERR_INVALID_ARG, "workspace of %lld bytes needed, %lld given", (long long)L.total,
                (long long)workspace_bytes);
  if (T > 0 && ((uintptr_t)workspace & 255u))
    return fail(DPPO_ERR_INVALID_ARG, "workspace must be 256-byte aligned");
  hipStream_t st = (hipStream_t)stream;
  dppo::launch_prep_stats(loss_mask, T, stats_out, st);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, "prep_stats launch");
  if (T == 0) {
    if (dweight && (e = dppo::launch_lmh_zero(dweight, V * d, st)) != hipSuccess)
      return hip_fail(e, "zero fill");
  } else {
    const bool grads = dhidden || dweight;
    char* ws = (char*)workspace;
    dppo::LmhArgs m{};
    m.hidden = (const uint16_t*)hidden;
    m.weight = (const uint16_t*)weight;
    m.T = (int32_t)T;
    m.d = (int32_t)d;
    m.V = (int32_t)V;
    m.n0 = 0;
    m.n1 = (int32_t)V;
    m.part = (float*)(ws + L.part);
    m.zy = (float*)(ws + L.zy);
    m.w = (float*)(ws + L.w);
    m.lse2 = (float*)(ws + L.lse2);
    m.dy = (float*)(ws + L.dy);
    m.ev = (uint8_t*)(ws + L.ev);
    m.ids = token_ids;
    m.g = (uint16_t*)(ws + L.g);
    m.ldg = L.ldg;
    m.store_p = grads && L.one_pass;
    dppo::RowArgs a{};
    a.ids = token_ids;
    a.lp_mu = logp_mu_old;
    a.lp_ref = p->ref_mode == DPPO_REF_GIVEN ? logp_ref : nullptr;
    a.adv = advantages;
    a.mask = loss_mask;
    a.tscale = token_scale;
    a.lp_out = logp_out;
    a.loss_tok = loss_tok_out;
    a.flags = flags_out;
    a.stats = stats_out;
    a.T = (int32_t)T;
    a.V = (int32_t)V;
    a.mode = dppo::kModeLoss;
    a.band_lo = p->band_lo;
    a.band_hi = p->band_hi;
    a.clip_lo = 1.0f - p->clip_eps_lo;
    a.clip_hi = 1.0f + p->clip_eps_hi;
    a.loss_scale = p->loss_scale;
    a.rd_mode = p->rd_mode;
    a.scale_mode = p->scale_mode;
    a.ref_mode = p->ref_mode;
    a.alpha = p->alpha;
    // timed launches: the forward tiles and each gradient product
    auto timed = [&](auto&& launch) -> hipError_t {
      auto* ev = timer_slot();
      if (ev) (void)hipEventRecord(ev->first, st);
      const hipError_t le = launch();
      if (ev) (void)hipEventRecord(ev->second, st);
      return le;
    };
    // dhidden (+)= G_c W_c over the chunk's vocabulary rows [n0, n1) (K = n1 - n0), and
    // dweight rows [n0, n1) = G_c^T hidden (K = T); G_c is [T, ldg] bf16 in the workspace.
    auto products = [&](int64_t n0, int64_t n1) -> dppo_status {
      const int64_t kc = n1 - n0;
      if (dhidden) {
        dppo::GemmArgs g{};
        g.a = m.g;
        g.lda = L.ldg;
        g.a_ext = (int32_t)T;
        g.b = (const uint16_t*)weight + n0 * d;
        g.ldb = d;
        g.b_ext = (int32_t)d;
        g.M = (int32_t)T;
        g.N = (int32_t)d;
        g.K = (int32_t)kc;
        g.c = dhidden;
        g.ldc = d;
        g.accumulate = n0 > 0;
        if ((e = timed([&] { return dppo::launch_lmh_grad_gemm(g, false, true, st); })) != hipSuccess)
          return hip_fail(e, "dhidden product launch");
      }
      if (dweight) {
        dppo::GemmArgs g{};
        g.a = m.g;
        g.lda = L.ldg;
        g.a_ext = (int32_t)((kc + 7) & ~(int64_t)7);
        g.b = (const uint16_t*)hidden;
        g.ldb = d;
        g.b_ext = (int32_t)d;
        g.M = (int32_t)kc;
        g.N = (int32_t)d;
        g.K = (int32_t)T;
        g.c = dweight + n0 * d;
        g.ldc = d;
        g.accumulate = 0;
        if ((e = timed([&] { return dppo::launch_lmh_grad_gemm(g, true, true, st); })) != hipSuccess)
          return hip_fail(e, "dweight product launch");
      }
      return DPPO_OK;
    };
    if ((e = dppo::launch_lmh_zy(m, st)) != hipSuccess) return hip_fail(e, "z_y launch");
    if ((e = timed([&] { return dppo::launch_lmh_fwd_tiles(m, st); })) != hipSuccess)
      return hip_fail(e, "forward tile launch");
    if (m.store_p) {
      // one pass: the row pass finishes every token, the scale pass forms G in place
      if ((e = dppo::launch_lmh_grad_rows(a, m, st)) != hipSuccess) return hip_fail(e, "gradient row launch");
      s = products(0, V);
      if (s != DPPO_OK) return s;
    } else {
      if ((e = dppo::launch_lmh_finish(a, m, st)) != hipSuccess) return hip_fail(e, "finish launch");
      for (int64_t n0 = 0; grads && n0 < V; n0 += L.chunk) {
        const int64_t n1 = std::min<int64_t>(V, n0 + L.chunk);
        m.n0 = (int32_t)n0;
        m.n1 = (int32_t)n1;
        if ((e = timed([&] { return dppo::launch_lmh_bwd_tiles(m, st); })) != hipSuccess)
          return hip_fail(e, "backward tile launch");
        s = products(n0, n1);
        if (s != DPPO_OK) return s;
      }
    }
  }
  dppo::launch_loss_sum(loss_tok_out, loss_mask, token_scale, stats_out, T, p->loss_scale,
                        p->scale_mode, loss_out, st);
  e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, "loss_sum launch");
  return DPPO_OK;
}

}  // extern "C"

// ------------------------------------------------------------------ no-allocation variant
// Scratch of fused_lm_head_loss_fwd_bwd_noalloc: one copy on every device the library runs
// on, held until the process ends. In host code `scratch` is only a stand-in for the
// symbol; its device address comes from hipGetSymbolAddress, once per device.
constexpr int64_t kNoallocScratchBytes = (int64_t)64 << 20;
static __device__ __align__(256) char scratch[kNoallocScratchBytes];

namespace {

// Device address of `scratch` on the current device, looked up on the first call there.
dppo_status scratch_address(void** out) {
  static std::mutex mu;
  static std::vector<std::pair<int, void*>> addr;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  std::lock_guard<std::mutex> lk(mu);
  for (auto& kv : addr)
    if (kv.first == dev) {
      *out = kv.second;
      return DPPO_OK;
    }
  void* p = nullptr;
  e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
  if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
  if (!p || ((uintptr_t)p & 255u)) return fail(DPPO_ERR_HIP, "scratch address %p not 256-byte aligned", p);
  addr.push_back({dev, p});
  *out = p;
  return DPPO_OK;
}

// The vocab_chunk the no-allocation variant runs with: 0 (one pass) when its workspace fits
// the scratch, else the largest multiple of 256 whose chunked workspace fits; -1 if none.
int64_t noalloc_chunk(int64_t T, int64_t V) {
  if (lmh_layout(T, V, 0).total <= kNoallocScratchBytes) return 0;
  const int64_t vpad = ((V + dppo::LMH_BN - 1) / dppo::LMH_BN) * dppo::LMH_BN;
  for (int64_t c = vpad - dppo::LMH_BN; c >= dppo::LMH_BN; ) {
    const int64_t total = lmh_layout(T, V, c).total;
    if (total <= kNoallocScratchBytes) return c;
    // jump close to the largest chunk that fits, then step down by whole tiles
    const int64_t over = (total - kNoallocScratchBytes + 2 * T - 1) / (2 * T);
    c -= std::max<int64_t>(dppo::LMH_BN, (over + dppo::LMH_BN - 1) / dppo::LMH_BN * dppo::LMH_BN);
  }
  return -1;
}

}  // namespace

extern "C" {

int64_t fused_lm_head_noalloc_scratch_bytes(void) { return kNoallocScratchBytes; }

dppo_status fused_lm_head_loss_fwd_bwd_noalloc(
    const void* hidden, const void* weight, int32_t dtype, int64_t T, int64_t d, int64_t V,
    const int64_t* token_ids, const float* logp_mu_old, const float* logp_ref,
    const float* advantages, const uint8_t* loss_mask, const float* token_scale,
    const dppo_params* p, float* logp_out, float* loss_tok_out, float* loss_out,
    uint8_t* flags_out, int32_t* stats_out, float* dhidden, float* dweight,
    int64_t* vocab_chunk_used, void* stream) {
  if (T < 0 || T >= ((int64_t)1 << 31) || V < 1 || V > ((int64_t)1 << 21))
    return fail(DPPO_ERR_INVALID_ARG, "T = %lld or V = %lld out of range", (long long)T, (long long)V);
  const int64_t chunk = T > 0 ? noalloc_chunk(T, V) : 0;
  if (chunk < 0)
    return fail(DPPO_ERR_UNSUPPORTED,
                "T = %lld, V = %lld need more than the %lld-byte scratch of the no-allocation "
                "variant even in 256-row vocabulary chunks; use fused_lm_head_loss_fwd_bwd with a "
                "workspace", (long long)T, (long long)V, (long long)kNoallocScratchBytes);
  void* ws = nullptr;
  if (T > 0) {
    const dppo_status s = scratch_address(&ws);
    if (s != DPPO_OK) return s;
  }
  const dppo_status s = fused_lm_head_loss_fwd_bwd(
      hidden, weight, dtype, T, d, V, token_ids, logp_mu_old, logp_ref, advantages, loss_mask,
      token_scale, p, logp_out, loss_tok_out, loss_out, flags_out, stats_out, dhidden, dweight,
      chunk, ws, T > 0 ? kNoallocScratchBytes : 0, stream);
  if (s == DPPO_OK && vocab_chunk_used) *vocab_chunk_used = chunk;
  return s;
}

dppo_status ewma_proxy_update(void* x_prox, const void* x_new, int32_t dtype, int64_t n,
                              float beta, double* w, int32_t reset, int32_t normalized,
                              void* stream) {
  if (dtype != DPPO_F32 && dtype != DPPO_BF16)
    return fail(DPPO_ERR_INVALID_ARG, "unknown dtype %d", (int)dtype);
  if (n < 0) return fail(DPPO_ERR_INVALID_ARG, "n = %lld < 0", (long long)n);
  if (!(beta >= 0.0f && beta < 1.0f)) return fail(DPPO_ERR_INVALID_ARG, "beta = %g not in [0, 1)", beta);
  if (n > 0 && (!x_prox || !x_new)) return fail(DPPO_ERR_INVALID_ARG, "x_prox and x_new are required");
  if (normalized && !w) return fail(DPPO_ERR_INVALID_ARG, "w is required in normalized mode");
  if (normalized && !(std::isfinite(*w) && *w >= 0.0))
    return fail(DPPO_ERR_INVALID_ARG, "w_{t-1} = %g must be finite and >= 0", normalized ? *w : 0.0);
  const int es = esize_of(dtype);
  if (n > 0 && x_prox != x_new &&
      overlaps(span_of(x_prox, 1, n, n, es), span_of(x_new, 1, n, n, es)))
    return fail(DPPO_ERR_INVALID_ARG, "x_prox overlaps x_new without aliasing them exactly");

  // Coefficients of x_prox <- ca * x_new + cb * x_prox, in double on the host.
  double ca, cb, w_new = normalized ? *w : 0.0;
  dppo::ewma_coefficients(reset != 0, normalized != 0, (double)beta, &w_new, &ca, &cb);
  if (n > 0) {
    const bool aligned = aligned16(x_prox) && aligned16(x_new);
    const hipError_t e = dppo::launch_ewma(x_prox, x_new, dtype == DPPO_BF16, n, (float)ca,
                                           (float)cb, cb != 0.0, aligned, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "ewma launch");
  }
  if (normalized) *w = w_new;
  return DPPO_OK;
}

dppo_status ewma_proxy_step(void* x_prox, const void* x_new, int32_t dtype, int64_t n,
                            float beta, double tau, int32_t patience, int32_t normalized,
                            const int32_t* stats, dppo_ewma_state* state, void* stream) {
  if (dtype != DPPO_F32 && dtype != DPPO_BF16)
    return fail(DPPO_ERR_INVALID_ARG, "unknown dtype %d", (int)dtype);
  if (n < 0) return fail(DPPO_ERR_INVALID_ARG, "n = %lld < 0", (long long)n);
  if (!(beta >= 0.0f && beta < 1.0f)) return fail(DPPO_ERR_INVALID_ARG, "beta = %g not in [0, 1)", beta);
  if (!std::isfinite(tau)) return fail(DPPO_ERR_INVALID_ARG, "tau = %g is not finite", tau);
  if (patience < 1) return fail(DPPO_ERR_INVALID_ARG, "patience = %d < 1", (int)patience);
  if (!state) return fail(DPPO_ERR_INVALID_ARG, "state is required");
  if (reinterpret_cast<uintptr_t>(state) % 8 != 0)
    return fail(DPPO_ERR_INVALID_ARG, "state must be 8-byte aligned");
  if (n > 0 && (!x_prox || !x_new)) return fail(DPPO_ERR_INVALID_ARG, "x_prox and x_new are required");
  const int es = esize_of(dtype);
  if (n > 0 && x_prox != x_new &&
      overlaps(span_of(x_prox, 1, n, n, es), span_of(x_new, 1, n, n, es)))
    return fail(DPPO_ERR_INVALID_ARG, "x_prox overlaps x_new without aliasing them exactly");
  if (n > 0 && (overlaps(span_of(state, 1, 1, 1, (int)sizeof(dppo_ewma_state)), span_of(x_prox, 1, n, n, es)) ||
                overlaps(span_of(state, 1, 1, 1, (int)sizeof(dppo_ewma_state)), span_of(x_new, 1, n, n, es))))
    return fail(DPPO_ERR_INVALID_ARG, "state overlaps x_prox or x_new");
  const bool aligned = n > 0 && aligned16(x_prox) && aligned16(x_new);
  const hipError_t e = dppo::launch_ewma_step(x_prox, x_new, dtype == DPPO_BF16, n, beta, tau,
                                              patience, normalized != 0, stats, state, aligned,
                                              (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "ewma step launch");
  return DPPO_OK;
}

// ------------------------------------------------------------------ vocabulary shards
namespace {
// Shard geometry shared by the two per-row shard calls: columns [vstart, vstart + Vs) of a
// V-column vocabulary, with 16-byte offsets inside one row kept within int range.
dppo_status check_shard(const void* logits, int32_t dtype, int64_t T, int64_t Vs, int64_t ld,
                        int64_t vstart, int64_t V) {
  dppo_status s = check_matrix(logits, dtype, T, Vs, ld, "logits_shard");
  if (s != DPPO_OK) return s;
  if (Vs * esize_of(dtype) > (int64_t)1 << 30)
    return fail(DPPO_ERR_INVALID_ARG, "shard row of %lld elements exceeds 1 GiB", (long long)Vs);
  if (vstart < 0 || V < 1 || vstart + Vs > V)
    return fail(DPPO_ERR_INVALID_ARG, "shard columns [%lld, %lld) outside [0, V = %lld)",
                (long long)vstart, (long long)(vstart + Vs), (long long)V);
  return DPPO_OK;
}
}  // namespace

dppo_status vocab_shard_stats(const void* logits_shard, int32_t dtype, int64_t T, int64_t Vs,
                              int64_t ld, int64_t vocab_start, int64_t V,
                              const int64_t* token_ids, const uint8_t* loss_mask,
                              float* shard_lse, float* shard_zy, void* stream) {
  dppo_status s = check_shard(logits_shard, dtype, T, Vs, ld, vocab_start, V);
  if (s != DPPO_OK) return s;
  if (T > 0 && (!token_ids || !shard_lse || !shard_zy))
    return fail(DPPO_ERR_INVALID_ARG, "token_ids, shard_lse and shard_zy are required");
  if (T == 0) return DPPO_OK;
  const int es = esize_of(dtype);
  dppo::ShardArgs a{};
  a.a.logits = logits_shard;
  a.a.ld = ld;
  a.a.ids = token_ids;
  a.a.mask = loss_mask;
  a.a.T = (int32_t)T;
  a.a.V = (int32_t)Vs;
  a.vstart = vocab_start;
  a.vtot = V;
  a.lse_out = shard_lse;
  a.zy_out = shard_zy;
  const bool vec = aligned16(logits_shard) && (ld * es) % 16 == 0;
  auto* ev = timer_slot();
  if (ev) (void)hipEventRecord(ev->first, (hipStream_t)stream);
  const hipError_t e = dppo::launch_shard_stats(a, dtype == DPPO_BF16, vec, (hipStream_t)stream);
  if (ev) (void)hipEventRecord(ev->second, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "shard stats launch");
  return DPPO_OK;
}

dppo_status vocab_shard_combine(const float* shard_lse, int32_t P, int64_t T, float* lse,
                                void* stream) {
  if (P < 1) return fail(DPPO_ERR_INVALID_ARG, "P = %d shards < 1", (int)P);
  if (T < 0 || T > 0x7FFFFFFF) return fail(DPPO_ERR_INVALID_ARG, "T = %lld out of [0, 2^31)", (long long)T);
  if (T > 0 && (!shard_lse || !lse)) return fail(DPPO_ERR_INVALID_ARG, "shard_lse and lse are required");
  if (T > 0 && overlaps(span_of(shard_lse, P, T, T, 4), span_of(lse, 1, T, T, 4)))
    return fail(DPPO_ERR_INVALID_ARG, "lse overlaps shard_lse");
  if (T == 0) return DPPO_OK;
  const hipError_t e = dppo::launch_shard_combine(shard_lse, P, T, lse, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "shard combine launch");
  return DPPO_OK;
}

dppo_status decoupled_ppo_loss_shard_fwd_bwd(
    const void* logits_shard, int32_t dtype, int64_t T, int64_t Vs, int64_t ld,
    int64_t vocab_start, int64_t V, const int64_t* token_ids, const float* lse, const float* zy,
    const float* logp_mu_old, const float* logp_ref, const float* advantages,
    const uint8_t* loss_mask, const float* token_scale, const dppo_params* p, float* logp_out,
    float* loss_tok_out, float* loss_out, uint8_t* flags_out, void* dlogits_shard,
    int64_t ld_dlogits, int32_t* stats_out, void* stream) {
  dppo_status s = check_shard(logits_shard, dtype, T, Vs, ld, vocab_start, V);
  if (s != DPPO_OK) return s;
  if (!p) return fail(DPPO_ERR_INVALID_ARG, "params pointer is NULL");
  if (!loss_out || !stats_out) return fail(DPPO_ERR_INVALID_ARG, "loss_out and stats_out are required");
  s = check_token_args(p, T, token_ids, logp_mu_old, logp_ref, advantages, logp_out, loss_tok_out);
  if (s != DPPO_OK) return s;
  if (T > 0 && (!lse || !zy)) return fail(DPPO_ERR_INVALID_ARG, "lse and zy are required");
  const int es = esize_of(dtype);
  if (dlogits_shard && T > 0) {
    if (ld_dlogits < Vs)
      return fail(DPPO_ERR_INVALID_ARG, "dlogits stride %lld < Vs = %lld", (long long)ld_dlogits, (long long)Vs);
    const bool same = dlogits_shard == logits_shard && ld_dlogits == ld;
    if (!same && overlaps(span_of(logits_shard, T, Vs, ld, es), span_of(dlogits_shard, T, Vs, ld_dlogits, es)))
      return fail(DPPO_ERR_INVALID_ARG, "dlogits overlaps logits without aliasing them exactly");
  }
  hipStream_t st = (hipStream_t)stream;
  dppo::launch_prep_stats(loss_mask, T, stats_out, st);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, "prep_stats launch");
  if (T > 0) {
    dppo::ShardArgs a{};
    dppo::RowArgs& r = a.a;
    r.logits = logits_shard;
    r.ld = ld;
    r.dlogits = dlogits_shard;
    r.ldd = ld_dlogits;
    r.ids = token_ids;
    r.lp_mu = logp_mu_old;
    r.lp_ref = p->ref_mode == DPPO_REF_GIVEN ? logp_ref : nullptr;
    r.ref_mode = p->ref_mode;
    r.alpha = p->alpha;
    r.adv = advantages;
    r.mask = loss_mask;
    r.tscale = token_scale;
    r.lp_out = logp_out;
    r.loss_tok = loss_tok_out;
    r.flags = flags_out;
    r.stats = stats_out;
    r.T = (int32_t)T;
    r.V = (int32_t)Vs;
    r.mode = dppo::kModeLoss;
    r.band_lo = p->band_lo;
    r.band_hi = p->band_hi;
    r.clip_lo = 1.0f - p->clip_eps_lo;
    r.clip_hi = 1.0f + p->clip_eps_hi;
    r.loss_scale = p->loss_scale;
    r.rd_mode = p->rd_mode;
    r.scale_mode = p->scale_mode;
    a.vstart = vocab_start;
    a.vtot = V;
    a.lse_in = lse;
    a.zy_in = zy;
    const bool vec = aligned16(logits_shard) && (ld * es) % 16 == 0 &&
                     (!dlogits_shard || (aligned16(dlogits_shard) && (ld_dlogits * es) % 16 == 0));
    auto* ev = timer_slot();
    if (ev) (void)hipEventRecord(ev->first, st);
    e = dppo::launch_shard_loss(a, dtype == DPPO_BF16, vec, st);
    if (ev) (void)hipEventRecord(ev->second, st);
    if (e != hipSuccess) return hip_fail(e, "shard loss launch");
  }
  dppo::launch_loss_sum(loss_tok_out, loss_mask, token_scale, stats_out, T, p->loss_scale,
                        p->scale_mode, loss_out, st);
  e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, "loss_sum launch");
  return DPPO_OK;
}

}  // extern "C"
