/*
 * dppo.h -- C ABI of the MI355X (gfx950) library for the per-token loss stage of
 * decoupled off-policy PPO (Guan et al., "Missing Old Logits in Asynchronous Agentic RL",
 * arXiv 2605.12070).
 *
 * Notation (the paper's): z = current-policy logits [T, V]; y = sampled token ids;
 * lp_theta = log pi_theta(y); lp_ref = log pi_old(y) (exact old logits, Sec. 5.1), or
 * log pi_prox(y) (PPO-EWMA proxy, Sec. 5.2), or log pi_async(y) (Table 1, last row);
 * lp_mu = log mu_old(y), the inference engine's log-prob of the sampled token (Sec. 3.2);
 * A = advantages; m = loss mask.
 *
 * Conventions shared by every entry point
 *  - All array pointers are DEVICE pointers owned by the caller (for example PyTorch
 *    tensors). The library keeps no pointer after a call returns and allocates no device
 *    memory in these calls. Host pointers are marked "host".
 *  - `stream` is a hipStream_t passed as void*; NULL means the default stream. Kernels are
 *    enqueued on it in order; no call synchronises the device or the stream.
 *  - Argument checks run on the host before any HIP call. A failed check returns
 *    DPPO_ERR_INVALID_ARG (or DPPO_ERR_UNSUPPORTED) and enqueues nothing;
 *    dppo_last_error() then describes the failure. A launch failure returns DPPO_ERR_HIP.
 *    Nothing throws across the ABI.
 *  - Data errors are reported on the device, not in the return code (see below).
 *  - A loss mask ([T] uint8, where a call takes one) is read in aligned 4-byte words (and,
 *    to count its tokens, in the aligned 16-byte chunks that cover it), so its allocation
 *    must be readable from the 16-byte boundary at or below mask up to the next 4-byte
 *    boundary past mask + T (true of any hipMalloc or PyTorch allocation, and of views into
 *    one); the bytes outside [mask, mask + T) are ignored.
 *  - Row strides (`ld`, `ld_dlogits`) are in elements. bf16 rows that do not start on a
 *    16-byte boundary, or whose length is not a multiple of 8, are read as the aligned
 *    16-byte chunks that cover them: the logits allocation must be readable from the 16-byte
 *    boundary at or below the first row to the one after the last row (true of any
 *    hipMalloc or PyTorch allocation, and of views into one); only the rows' own entries
 *    are written. This needs dlogits (if any) at the logits' offset within 16 bytes on
 *    every row (the same pointer residue mod 16 and strides that differ by a multiple of 8
 *    entries, as in place or for a tensor of the logits' layout). Other layouts, fp32 rows
 *    that are not aligned, and rows longer than the resident kernels hold take a slower
 *    streaming path; none of this is an error.
 *  - Thread safety: calls may be issued from several host threads; the kernel timer
 *    (dppo_timer_*) is process-global and meant for one profiling thread.
 */
#ifndef DPPO_H
#define DPPO_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  DPPO_OK = 0,
  DPPO_ERR_INVALID_ARG = 1, /* null required pointer, bad size, bad enum, bad parameter */
  DPPO_ERR_UNSUPPORTED = 2, /* valid request the library does not implement */
  DPPO_ERR_HIP = 3          /* a HIP runtime call or kernel launch failed */
} dppo_status;

/* Storage type of logits / dlogits / EWMA buffers. Arithmetic is float32 throughout. */
typedef enum { DPPO_F32 = 0, DPPO_BF16 = 1 } dppo_dtype;

/* How the discrepancy ratio r_d = pi_ref / mu_old enters the objective.
 *  NONE:        wd = 1          (PPO-clip on r_s only; Table 1 rows with r_d = 1)
 *  MASK:        wd = M(r_d)     (band mask of Eq. 4, the MIS weight without the ratio)
 *  WEIGHT:      wd = r_d        (down-weighting; the r2 factor of Table 5)
 *  MASK_WEIGHT: wd = M(r_d) r_d (Eq. 4's mask with the total ratio r = r_d r_s of the MIS
 *                                gradient, Sec. 3.1 and Sec. 3.2; the default)          */
typedef enum {
  DPPO_RD_NONE = 0,
  DPPO_RD_MASK = 1,
  DPPO_RD_WEIGHT = 2,
  DPPO_RD_MASK_WEIGHT = 3
} dppo_rd_mode;

/* Per-token scale s_t = scale * token_scale_t with
 *  CONST:      scale = loss_scale
 *  TOKEN_MEAN: scale = loss_scale / max(1, sum_t m_t)   (the E_t of Eq. 2 read as a mean
 *              over loss-mask-valid tokens; band- and clip-removed tokens stay counted)  */
typedef enum { DPPO_SCALE_CONST = 0, DPPO_SCALE_TOKEN_MEAN = 1 } dppo_scale_mode;

/* Per-token flags (uint8), written when flags_out is non-NULL. */
#define DPPO_FLAG_VALID 1u  /* m_t = 1: the row was evaluated                           */
#define DPPO_FLAG_BAND 2u   /* band_lo <= r_d <= band_hi (Eq. 4)                         */
#define DPPO_FLAG_PPO 4u    /* Eq. 3 active mask holds on r_s (not clipped)              */
#define DPPO_FLAG_BAD_ID 8u /* valid row whose token id is outside [0, V)                */

/* stats_out layout (int32[5]). rho_t = stats[3] / stats[0] is the Train-Infer Mask value
 * that drives the PPO-EWMA automatic reset (Sec. 5.2).                                   */
#define DPPO_STAT_N_VALID 0  /* sum_t m_t                                                 */
#define DPPO_STAT_N_BAND 1   /* valid, good-id tokens inside the r_d band                  */
#define DPPO_STAT_N_PPO 2    /* valid, good-id tokens with the PPO mask active             */
#define DPPO_STAT_N_ACTIVE 3 /* PPO-active and (for MASK, MASK_WEIGHT) inside the band     */
#define DPPO_STAT_N_BAD 4    /* valid rows with an out-of-range token id                   */
#define DPPO_N_STATS 5

/* Where pi_ref, the policy between mu_old and pi_theta that splits the ratio, comes from.
 *  GIVEN:      logp_ref is an input (exact old log-probs, Sec. 5.1, or the PPO-EWMA proxy,
 *              Sec. 5.2).
 *  LOGLINEAR:  token-wise log-linear interpolation (App. A):
 *                log pi_ref = alpha log mu_old + (1 - alpha) log pi_theta.
 *  LINEAR:     arithmetic interpolation (App. A): pi_ref = alpha mu_old + (1 - alpha) pi_theta.
 * alpha in (0, 1) is the behaviour-policy weight (1 / (n + 1) for version gap n, Table 4).
 * An interpolated pi_ref is evaluated on the current log-prob and, like any reference, is a
 * constant with respect to theta. logp_ref is not read (may be NULL) unless GIVEN.         */
typedef enum { DPPO_REF_GIVEN = 0, DPPO_REF_LOGLINEAR = 1, DPPO_REF_LINEAR = 2 } dppo_ref_mode;

/* Knobs of the decoupled MIS objective (Eq. 2, Eq. 3, Eq. 4; Table 1).
 *  band_lo, band_hi:         r_d is kept iff band_lo <= r_d <= band_hi (inclusive, as in
 *                            Eq. 4: M_[1/c, c] is band_lo = 1/c, band_hi = c; App. A's
 *                            [1 - eps_1, 1 + eps_1] is the same with other bounds).
 *                            0 <= band_lo <= band_hi; band_hi may be +inf.
 *  clip_eps_lo, clip_eps_hi: PPO interval [1 - eps_lo, 1 + eps_hi] on r_s (Eq. 2; the
 *                            asymmetric form of App. A). Both >= 0, finite.
 *  rd_mode:                  a dppo_rd_mode.
 *  scale_mode, loss_scale:   a dppo_scale_mode and a finite multiplier.
 *  ref_mode, alpha:          a dppo_ref_mode; alpha in (0, 1) unless ref_mode is GIVEN. */
typedef struct dppo_params {
  float band_lo, band_hi;
  float clip_eps_lo, clip_eps_hi;
  int32_t rd_mode;
  int32_t scale_mode;
  float loss_scale;
  int32_t ref_mode;
  float alpha;
} dppo_params;

/*
 * logprob_fwd -- sampled-token log-probabilities log pi(y_t) = z[t, y_t] - lse_t with
 * lse_t = log sum_v exp z[t, v] over the whole vocabulary (the token probabilities whose
 * ratios Sec. 3.2 and Eq. 1 take). Also produces lp_ref from an old or proxy model's
 * logits (Sec. 5.1 exact routes, Sec. 5.2 proxy).
 *
 *  logits     [T, ld] of `dtype` (DPPO_F32 or DPPO_BF16), row t at logits + t*ld; only
 *             the first V entries of a row are read.
 *  T >= 0, V >= 1, ld >= V; T < 2^31.
 *  token_ids  [T] int64.
 *  logp_out   [T] float32: log pi(y_t); NaN when y_t is outside [0, V).
 *  lse_out    [T] float32 or NULL.
 * Non-finite logits follow IEEE arithmetic: a row holding NaN or +inf, or only -inf, has
 * lse = NaN. T = 0 enqueues nothing.
 */
dppo_status logprob_fwd(const void* logits, int32_t dtype, int64_t T, int64_t V, int64_t ld,
                        const int64_t* token_ids, float* logp_out, float* lse_out,
                        void* stream);

/* Most policy versions one logprob_fwd_versioned call can read. */
#define DPPO_MAX_VERSIONS 8

/*
 * logprob_fwd_versioned -- logprob_fwd for a batch whose tokens were generated by different
 * policy versions (partial rollouts): token t's log-prob is read from the logits of the
 * version that produced it, version_ids[t]. These are the exact old log-probs of the
 * snapshot route (Sec. 5.1): one forward pass per stored version, then the per-token
 * log-prob under the right one.
 *
 *  logits       host array of K device pointers; logits[v] is version v's [T, ld] matrix of
 *               `dtype` (all K share dtype, T, V and ld). 1 <= K <= DPPO_MAX_VERSIONS.
 *  version_ids  [T] int32 device array. A token whose version lies outside [0, K) gets
 *               log-prob NaN (like an out-of-range token id).
 *  Other arguments as logprob_fwd. Only the selected version's row of each token is read.
 */
dppo_status logprob_fwd_versioned(const void* const* logits, int32_t K, int32_t dtype, int64_t T,
                                  int64_t V, int64_t ld, const int32_t* version_ids,
                                  const int64_t* token_ids, float* logp_out, float* lse_out,
                                  void* stream);

/*
 * decoupled_ppo_loss_fwd_bwd -- the fused loss stage: log-prob through a vocabulary-wide
 * log-sum-exp, ratios r_s = pi_theta / pi_ref and r_d = pi_ref / mu_old (Eq. 1, Sec. 3.2),
 * the band decision M(r_d) (Eq. 4), the sign-dependent PPO decision on r_s (Eq. 3), the
 * per-token loss l_t = -wd_t * min(r_s A, clip(r_s, 1-eps_lo, 1+eps_hi) A) (Eq. 2), and,
 * when dlogits is non-NULL, the gradient of L = sum_t m_t s_t l_t with respect to the
 * logits in MIS form (Sec. 3.1):
 *     dlogits[t, v] = w_t * (softmax(z_t)[v] - 1{v = y_t}),
 *     w_t = m_t * s_t * wd_t * r_s * A_t  if PPO-active (and, for MASK modes, in band),
 *     w_t = 0                              otherwise.
 * r_d, the band and lp_ref are constants with respect to theta.
 *
 *  logits        [T, ld] of dtype; dlogits (if non-NULL) [T, ld_dlogits] of the same
 *                dtype. dlogits may alias logits only exactly (same pointer and stride);
 *                any other overlap is DPPO_ERR_INVALID_ARG.
 *  token_ids     [T] int64.   logp_mu_old, logp_ref, advantages: [T] float32; logp_ref
 *                only with ref_mode GIVEN (NULL allowed otherwise).
 *  loss_mask     [T] uint8 or NULL (all 1). Rows with m_t = 0 are not read: lp 0, loss 0,
 *                flags 0, and a zero dlogits row.
 *  token_scale   [T] float32 or NULL (all 1).
 *  p             host pointer to the parameters.
 *  logp_out      [T] float32: lp_theta (0 on masked rows, NaN on bad ids).
 *  loss_tok_out  [T] float32: l_t (before m_t and s_t).
 *  loss_out      [1] float32: L = sum_t m_t s_t l_t, summed in a fixed order in float64
 *                (bitwise reproducible run to run).
 *  flags_out     [T] uint8 or NULL.
 *  stats_out     [5] int32 (see DPPO_STAT_*); overwritten by the call.
 * A valid row with y_t outside [0, V) gets lp NaN, l_t = 0, w_t = 0, a zero dlogits row,
 * flags VALID|BAD_ID, and counts in stats[4] only. T = 0 writes loss 0 and zero stats.
 */
dppo_status decoupled_ppo_loss_fwd_bwd(
    const void* logits, int32_t dtype, int64_t T, int64_t V, int64_t ld,
    const int64_t* token_ids, const float* logp_mu_old, const float* logp_ref,
    const float* advantages, const uint8_t* loss_mask, const float* token_scale,
    const dppo_params* p, float* logp_out, float* loss_tok_out, float* loss_out,
    uint8_t* flags_out, void* dlogits, int64_t ld_dlogits, int32_t* stats_out, void* stream);

/*
 * fused_lm_head_loss_fwd_bwd -- decoupled_ppo_loss_fwd_bwd on logits z = hidden weight^T
 * that are never written to memory, with the gradients of L for both factors:
 *     d L / d hidden = G weight,   d L / d weight = G^T hidden,
 *     G[t, v] = w_t (softmax(z_t)[v] - 1{v = y_t})   (the dlogits of the row entry point,
 *     the MIS gradient of Sec. 3.1 chained through the LM head).
 * The logits exist only as 256 x 256 tiles in registers and LDS, formed with bf16
 * matrix-core products and fp32 accumulation; the forward pass reduces each tile to
 * per-token partial log-sum-exps. All four products run in the library's own matrix-core
 * kernels. lp, loss, flags, stats and the parameters are as in decoupled_ppo_loss_fwd_bwd
 * (ref_mode included).
 *
 * Two ways to form G, chosen by vocab_chunk:
 *  - vocab_chunk <= 0 or >= V (one pass, the default): the forward tiles also store their
 *    exponentials 2^(z log2 e - m) (m the maximum of each 128-entry vocabulary group) as
 *    fp16 into the workspace; once every token's log-sum-exp is known, a row pass scales
 *    them into G in bf16 in place. The logits are formed once.
 *  - 0 < vocab_chunk < V (chunked, for a smaller workspace): the backward recomputes the
 *    logit tiles one vocabulary chunk at a time and writes that chunk of G in bf16; the two
 *    gradient products then run on the chunk. The logits are formed twice.
 *
 *  hidden       [T, d] bf16, row-major, 16-byte aligned.
 *  weight       [V, d] bf16, row-major (an LM head in the [out, in] layout), 16-byte aligned.
 *  dtype        DPPO_BF16 (DPPO_F32 is DPPO_ERR_UNSUPPORTED).
 *  d            multiple of 8, at most 2^20; 1 <= V <= 2^21; T < 2^31.
 *  dhidden      [T, d] float32 or NULL (not computed); overwritten.
 *  dweight      [V, d] float32 or NULL (not computed); overwritten.
 *  vocab_chunk  see above; a chunk is rounded up to a multiple of 256 vocabulary rows.
 *  workspace    device buffer of at least fused_lm_head_workspace_bytes(T, d, V, vocab_chunk)
 *               bytes, 256-byte aligned, owned by the caller; its contents are scratch.
 * Masked rows and bad ids behave as in the row entry point (their G rows are zero). The
 * computation of rows with loss mask 0 is not skipped: a caller whose batch has many of them
 * passes only the rows it trains on (hidden, ids and the per-token inputs gathered), which
 * gives the same loss, counters and token-mean scale, and dweight up to the order of its
 * sum over tokens; the dhidden rows of the dropped tokens are zero. The call allocates
 * nothing.
 */
dppo_status fused_lm_head_loss_fwd_bwd(
    const void* hidden, const void* weight, int32_t dtype, int64_t T, int64_t d, int64_t V,
    const int64_t* token_ids, const float* logp_mu_old, const float* logp_ref,
    const float* advantages, const uint8_t* loss_mask, const float* token_scale,
    const dppo_params* p, float* logp_out, float* loss_tok_out, float* loss_out,
    uint8_t* flags_out, int32_t* stats_out, float* dhidden, float* dweight,
    int64_t vocab_chunk, void* workspace, int64_t workspace_bytes, void* stream);

/* Workspace bytes fused_lm_head_loss_fwd_bwd needs for these sizes (-1 if they are out of
 * range): per-token partial sums of every 128-entry vocabulary group (8 B per token and
 * group), four per-token vectors, and either [T, V rounded up to 256] of 2 bytes (one
 * pass) or one bf16 [T, chunk] gradient chunk (chunked). */
int64_t fused_lm_head_workspace_bytes(int64_t T, int64_t d, int64_t V, int64_t vocab_chunk);

/*
 * fused_lm_head_loss_fwd_bwd_noalloc -- fused_lm_head_loss_fwd_bwd for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid allocation): the workspace is the library's own static device scratch of
 * fused_lm_head_noalloc_scratch_bytes() = 64 MiB, one copy on every device the library runs
 * on, held until the process ends. The call allocates nothing (no hipMalloc, no allocating
 * library routine); the caller still passes every input and output.
 *  - It runs one pass (vocab_chunk 0) when that workspace fits the scratch, else the
 *    largest chunk of 256-row multiples that fits; *vocab_chunk_used (host, nullable)
 *    receives that value, and fused_lm_head_loss_fwd_bwd with the same vocab_chunk gives
 *    the same bits. Sizes whose 256-row chunked workspace exceeds the scratch return
 *    DPPO_ERR_UNSUPPORTED and enqueue nothing.
 *  - Every call on a device shares that device's scratch, which keeps the last call's
 *    contents (nothing in it needs clearing: every call writes what it reads). Calls that
 *    overlap on one device (other streams, other host threads) race on it and must be
 *    serialised by the caller.
 * Every other argument and the error behaviour are those of fused_lm_head_loss_fwd_bwd.
 */
dppo_status fused_lm_head_loss_fwd_bwd_noalloc(
    const void* hidden, const void* weight, int32_t dtype, int64_t T, int64_t d, int64_t V,
    const int64_t* token_ids, const float* logp_mu_old, const float* logp_ref,
    const float* advantages, const uint8_t* loss_mask, const float* token_scale,
    const dppo_params* p, float* logp_out, float* loss_tok_out, float* loss_out,
    uint8_t* flags_out, int32_t* stats_out, float* dhidden, float* dweight,
    int64_t* vocab_chunk_used, void* stream);

/* Bytes of the no-allocation variant's per-device scratch. */
int64_t fused_lm_head_noalloc_scratch_bytes(void);

/*
 * ewma_proxy_update -- one step of the PPO-EWMA reference (Sec. 5.2, Eq. 5; App. B) on a
 * flat buffer of n elements (proxy parameters, or per-token log-probs).
 *  normalized = 1: w_t = 1 + beta * w_{t-1};
 *                  x_prox <- x_new / w_t + beta * (w_{t-1} / w_t) * x_prox.
 *                  With w_{t-1} = 0 (first step) x_prox <- x_new and x_prox is not read.
 *  normalized = 0: fixed-decay form of Table 1: x_prox <- beta x_prox + (1 - beta) x_new;
 *                  `w` is not used and may be NULL.
 *  reset = 1:      automatic reset (Sec. 5.2): x_prox <- x_new, and *w = 1 when normalized.
 *  x_prox, x_new   [n] device buffers of `dtype` (float32 math, bf16 stored with RNE);
 *                  x_prox may not overlap x_new unless identical.
 *  beta            in [0, 1).
 *  w               host pointer: in w_{t-1} (0 before the first step), out w_t.
 * n = 0 only updates *w.
 */
dppo_status ewma_proxy_update(void* x_prox, const void* x_new, int32_t dtype, int64_t n,
                              float beta, double* w, int32_t reset, int32_t normalized,
                              void* stream);

/*
 * Vocabulary shards. The training engine's LM head may split the vocabulary over GPUs
 * (tensor parallelism, one of the training-side implementations Sec. 1 names). A GPU then
 * holds the column block [vocab_start, vocab_start + Vs) of the logits, and the per-token
 * log-prob of Sec. 3.2 needs a log-sum-exp over every shard. The three calls below are one
 * GPU's share of that path, at the shard's own shape:
 *   1. vocab_shard_stats on every shard: the shard's row log-sum-exp and z[y] where it
 *      holds column y;
 *   2. an exchange across the shards, done by the caller: all-gather of shard_lse into
 *      [P, T] (shard order), all-reduce sum of shard_zy (exactly one shard holds z[y]);
 *      then vocab_shard_combine on every shard, which gives the same lse everywhere;
 *   3. decoupled_ppo_loss_shard_fwd_bwd on every shard: the token math of Eq. 1-4 from
 *      the global lse and z[y] (every shard computes the same per-token outputs, loss and
 *      stats), and the shard's own columns of dlogits = w (softmax - onehot).
 * With P = 1 and vocab_start = 0 the three calls compute decoupled_ppo_loss_fwd_bwd (up to
 * rounding: the logits are read twice, not once).
 */

/*
 * vocab_shard_stats -- per row t of a shard [T, Vs] (row stride ld elements):
 *    shard_lse[t] = log sum_{v < Vs} exp z[t, v]   (-inf when every entry is -inf),
 *    shard_zy[t]  = z[t, y_t - vocab_start] if vocab_start <= y_t < vocab_start + Vs, else 0.
 *  Rows with loss_mask = 0 (nullable: all valid) are not read: shard_lse = -inf, shard_zy = 0.
 *  V is the whole vocabulary: vocab_start >= 0 and vocab_start + Vs <= V, else INVALID_ARG.
 *  NaN or +inf entries make shard_lse NaN.
 */
dppo_status vocab_shard_stats(const void* logits_shard, int32_t dtype, int64_t T, int64_t Vs,
                              int64_t ld, int64_t vocab_start, int64_t V,
                              const int64_t* token_ids, const uint8_t* loss_mask,
                              float* shard_lse, float* shard_zy, void* stream);

/*
 * vocab_shard_combine -- lse[t] = log sum_p exp shard_lse[p][t] over P gathered shard
 * statistics ([P, T] float32, shard-major), summed in shard order around their maximum.
 * A token whose shards are all -inf (its row masked, or all of its logits -inf) gets NaN,
 * as the unsharded log-sum-exp gives for a row of -inf. lse may not overlap shard_lse.
 */
dppo_status vocab_shard_combine(const float* shard_lse, int32_t P, int64_t T, float* lse,
                                void* stream);

/*
 * decoupled_ppo_loss_shard_fwd_bwd -- decoupled_ppo_loss_fwd_bwd on one shard, with the row
 * statistics given: lp = zy - lse per token, then the ratios, band, PPO clip, loss and MIS
 * weight w exactly as decoupled_ppo_loss_fwd_bwd computes them (Eq. 1-4, Sec. 3.1), and
 *    dlogits_shard[t, v] = w_t (exp(z[t, v] - lse_t) - 1{vocab_start + v = y_t}),  v < Vs.
 *  lse, zy      [T] float32: vocab_shard_combine's lse and the all-reduced shard_zy.
 *  token_ids    global ids; y outside [0, V) is a bad id (lp NaN, loss 0, a zero gradient
 *               row, stats[4]++), as in decoupled_ppo_loss_fwd_bwd.
 *  Every other argument, output, alias rule (dlogits_shard may be logits_shard with the same
 *  stride) and error convention is that of decoupled_ppo_loss_fwd_bwd with V replaced by Vs
 *  for the matrices. The per-token outputs, loss and stats are the same on every shard:
 *  they are not to be summed across shards.
 */
dppo_status decoupled_ppo_loss_shard_fwd_bwd(
    const void* logits_shard, int32_t dtype, int64_t T, int64_t Vs, int64_t ld,
    int64_t vocab_start, int64_t V, const int64_t* token_ids, const float* lse, const float* zy,
    const float* logp_mu_old, const float* logp_ref, const float* advantages,
    const uint8_t* loss_mask, const float* token_scale, const dppo_params* p, float* logp_out,
    float* loss_tok_out, float* loss_out, uint8_t* flags_out, void* dlogits_shard,
    int64_t ld_dlogits, int32_t* stats_out, void* stream);

/*
 * Device-resident state of the PPO-EWMA reference and of its automatic reset (Sec. 5.2,
 * App. B, App. E), for ewma_proxy_step. 40 bytes, 8-byte aligned, in device memory owned by
 * the caller; checkpoint it together with the proxy buffer. Initialise with the host: w as
 * for ewma_proxy_update (0 before the first step, 1 when the buffer already holds
 * theta^(0)), every other field 0.
 */
typedef struct {
  double w;           /* normaliser: w_{t-1} before a step, w_t after (normalized form)    */
  int32_t streak;     /* consecutive steps with rho_t < tau, reset to 0 when a reset fires */
  int32_t resets;     /* resets fired so far                                               */
  int32_t last_reset; /* 1 when the last step reset the buffer, else 0                     */
  int32_t error;      /* 1 when the last step found w negative or not finite; that step    */
                      /* left the buffer and the state (other than this field) unchanged  */
  float last_rho;     /* rho_t of the last step                                            */
  float ca, cb;       /* coefficients of the last step: x_prox <- ca x_new + cb x_prox      */
  int32_t reserved;
} dppo_ewma_state;

/*
 * ewma_proxy_step -- the reset controller and the PPO-EWMA update of ewma_proxy_update,
 * both on the device, so that a training step needs no device-to-host copy and no
 * synchronisation (the reset rule of Sec. 5.2 and App. E; the recursion of Eq. 5 / App. B).
 * The controller (one thread; for n <= 16384 in the same one-workgroup launch as the
 * update) reads the loss stage's counters and updates *state:
 *    rho_t = n_active / n_valid (1 when n_valid = 0);
 *    streak <- streak + 1 if rho_t < tau (compared in double), else 0;
 *    a reset fires when streak >= patience; the streak then restarts at 0;
 *    (stats NULL: rho_t = 1, no reset, the streak unchanged; dppo_reset_decision is the
 *    same rule on the host)
 *    w_t and (ca, cb) exactly as ewma_proxy_update computes them on the host, in double,
 *    then rounded to float.
 * The update then applies x_prox <- ca x_new + cb x_prox (x_prox not read when cb = 0) with
 * the arithmetic of ewma_proxy_update, so both entry points give bit-identical buffers for
 * the same sequence of reset decisions.
 *  x_prox, x_new  [n] device buffers of `dtype`, as for ewma_proxy_update.
 *  beta           in [0, 1); tau finite; patience >= 1.
 *  stats          device [5] int32 counters of the step (decoupled_ppo_loss_fwd_bwd's
 *                 stats_out), or NULL.
 *  state          device pointer, 8-byte aligned (see dppo_ewma_state).
 * n = 0 runs the controller only. The host checks the arguments above; w is checked on the
 * device (state->error).
 */
dppo_status ewma_proxy_step(void* x_prox, const void* x_new, int32_t dtype, int64_t n,
                            float beta, double tau, int32_t patience, int32_t normalized,
                            const int32_t* stats, dppo_ewma_state* state, void* stream);

/*
 * Host side of the PPO-EWMA reference (Sec. 5.2; App. B; App. E). Pure host arithmetic in
 * double, no HIP call; `stats` here is a HOST copy of the five counters a loss call wrote
 * (see DPPO_STAT_*). ewma_proxy_step runs the same rule on the device.
 *
 * dppo_beta_from_window: the staleness-aware decay beta = W / (W + 2) for a version window
 *   of width W (App. B), which puts the EWMA's centre of mass beta / (1 - beta) at W / 2.
 *   INVALID_ARG for W negative or not finite, or a NULL beta.
 * dppo_train_infer_mask_value: rho_t = n_active / n_valid, the fraction of valid tokens the
 *   decoupled mask keeps (Sec. 5.2); 1 when no token is valid.
 * dppo_ppo_clip_ratio: 1 - n_ppo / n_valid, the fraction of valid tokens the PPO clip
 *   removes; 0 when no token is valid.
 * dppo_reset_decision: one step of the automatic reset (Sec. 5.2; App. E). *streak (host,
 *   in/out, >= 0) counts consecutive steps with rho_t < tau, compared in double; *fire = 1
 *   when the streak reaches `patience` (>= 1), and the streak then restarts at 0. rho
 *   (nullable) receives rho_t. stats = NULL means no decision input, as in
 *   ewma_proxy_step: rho_t = 1, no reset, the streak unchanged. tau must be finite. On
 *   INVALID_ARG nothing is written.
 */
dppo_status dppo_beta_from_window(double window, double* beta);
dppo_status dppo_train_infer_mask_value(const int32_t* stats, double* rho);
dppo_status dppo_ppo_clip_ratio(const int32_t* stats, double* ratio);
dppo_status dppo_reset_decision(const int32_t* stats, double tau, int32_t patience,
                                int32_t* streak, double* rho, int32_t* fire);

/* Row-kernel policy, a testing and benchmarking hook, two bits. Bit 0: clear = automatic
 * (the register-resident kernel when the row fits, the two-pass streaming kernel
 * otherwise), set = always the streaming kernel. Bit 1: decoupled_ppo_loss_fwd_bwd counts
 * its statistics with a counting kernel and atomics even where it would otherwise take them
 * from the flags (same results). Process-global; a value outside 0..3 is INVALID_ARG. */
dppo_status dppo_set_path_policy(int32_t policy);

/* Name of the per-row kernel (as profilers print it) that a call with this logits dtype,
 * row length V and row stride ld (elements) launches under the current path policy,
 * assuming 16-byte-aligned base pointers; with_dlogits != 0 for the fused backward.
 * Pure host logic, no HIP call. The string is owned by the library and valid until the
 * next call on this host thread. NULL for an invalid dtype or V < 1 or ld < V. */
const char* dppo_row_kernel_name(int32_t dtype, int64_t V, int64_t ld, int32_t with_dlogits);

/* Effective bounds on the total ratio r = pi_theta / mu_old that an interpolated
 * reference induces (Prop. 1; App. A; Table 4): with the band [mask_lo, mask_hi] on r_d
 * and the PPO interval [clip_lo, clip_hi] on r_s,
 *   out[0], out[1]: the band as bounds on r;
 *   out[2]:         the clip lower bound on r (applies to A < 0);
 *   out[3]:         the clip upper bound on r (applies to A >= 0).
 * ref_mode LOGLINEAR: r_d = r^(1-alpha), r_s = r^alpha.
 * ref_mode LINEAR:    r_d = alpha + (1-alpha) r, r_s = r / (alpha + (1-alpha) r); a clip
 *                     bound b with (1-alpha) b >= 1 is unreachable and reported as +inf.
 * Pure host arithmetic in double. INVALID_ARG for ref_mode GIVEN or unknown, alpha outside
 * (0, 1), bounds that are negative or out of order, or a NULL out.                      */
dppo_status dppo_effective_thresholds(double mask_lo, double mask_hi, double clip_lo,
                                      double clip_hi, double alpha, int32_t ref_mode,
                                      double* out);

/* Static description of a status code. */
const char* dppo_strerror(dppo_status s);

/* Message of the last failed call on this host thread ("" if none). */
const char* dppo_last_error(void);

/* ABI version of this header (incremented on incompatible changes). */
#define DPPO_ABI_VERSION 6
int32_t dppo_abi_version(void);

/*
 * Kernel timer for profiling. While enabled, the library records a pair of HIP events on
 * the call's stream around every launch of the per-row loss-stage kernel (the one that
 * streams the logits; for the vocabulary-shard calls, the shard kernel; for the fused LM
 * head, its logit-tile kernels and each gradient product) and, on dppo_timer_read,
 * synchronises those events and returns the summed elapsed time in milliseconds and the
 * number of launches timed, then clears the record. Enabling allocates host-side event objects; it is process-global state, meant
 * for one profiling thread.
 */
dppo_status dppo_timer_enable(int32_t on);
dppo_status dppo_timer_read(double* total_ms, int64_t* launches);

#ifdef __cplusplus
}
#endif

#endif /* DPPO_H */
