"""Plain float64 CPU oracle for the per-token loss stage of decoupled off-policy PPO.

TEST INFRASTRUCTURE. This module is the checker, not the product. Only the tests, the
smoke check and the benchmark's CPU-baseline leg may import or run it; the library path
never does. It shares no code, constant or helper with the HIP path and imports nothing
from the package.

Source: Guan et al., "Missing Old Logits in Asynchronous Agentic RL: Semantic Mismatch and
Repair Methods for Off-Policy Correction" (arXiv 2605.12070).

Everything here is a definition evaluated in float64 with numpy, written to be read
against the paper:

* sampled-token log-probability, log pi(y) = z[y] - log sum_v exp z[v]: the quantity whose
  ratios the paper takes (Sec. 3.2); evaluated with the usual max shift;
* the ratio decomposition r = pi_theta/mu_old = r_d * r_s (Eq. 1, Sec. 3.2);
* the discrepancy band mask M_[lo,hi](r_d) = 1{lo <= r_d <= hi} (Eq. 4; Table 1);
* the sign-dependent PPO active mask (Eq. 3) on r_s, with separate lower and upper clip
  widths (App. A, "Numerical effective thresholds");
* the clipped surrogate min(r A, clip(r, 1-eps_lo, 1+eps_hi) A) (Eq. 2);
* the MIS gradient form E[MIS * r * A * grad log pi] (Sec. 3.1), pushed through
  d log pi(y) / dz = onehot(y) - softmax(z);
* the PPO-EWMA proxy recursion, its closed form, its centre of mass and the
  staleness-aware decay (Sec. 5.2, Eq. 5; App. B);
* the Train-Infer Mask value rho_t and the automatic reset rule (Sec. 5.2; App. E);
* the effective thresholds that interpolation proxies induce on the total ratio
  (Prop. 1; App. A; Table 4).

Readings where the paper is silent, each with its reason:

* The loss value is L = sum_t m_t * s_t * l_t with l_t = -wd_t * min(r_s A, clip(r_s) A),
  s_t = scale * token_scale_t, and scale = loss_scale (constant mode) or
  loss_scale / max(1, sum_t m_t) (token-mean mode). The expectation E_t of Eq. 2 is not
  pinned to a normaliser by the paper: the loss normalisation is "parity unpinned".
* wd_t, how r_d enters, is one of: none (1), mask (band), weight (r_d), mask_weight
  (band * r_d). mask_weight is the main-text reading: Eq. 4's mask times the MIS
  gradient's total ratio r = r_d * r_s (Sec. 3.1, Sec. 3.2).
* Ties are inclusive, as in Eq. 3 and Eq. 4. A = 0 takes the A >= 0 branch.
* r_d, the band decision and the reference log-probs are constants with respect to theta.
* Rows with loss mask m_t = 0 are not evaluated: log-prob 0, loss 0, flags 0, a zero
  dlogits row. A valid row whose token id is outside [0, V) gets log-prob NaN, loss 0,
  weight 0, a zero dlogits row, flags VALID|BAD_ID, and is counted in n_bad_ids only.
* Non-finite logits follow IEEE arithmetic through the max-shifted log-sum-exp: a row with
  a NaN or +inf logit, or with every logit -inf, has lse = NaN, so log-prob, r_s and
  loss are NaN, the PPO decision is false (the band decision on r_d is unaffected), the
  weight is 0 and the dlogits row is NaN.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

# ---------------------------------------------------------------------------------------
# Flags and stats layout (per token, uint8; per call, five counts)
# ---------------------------------------------------------------------------------------
FLAG_VALID = 1       # m_t = 1: the row was evaluated
FLAG_BAND = 2        # lo <= r_d <= hi (Eq. 4 band), valid rows with a good id only
FLAG_PPO = 4         # Eq. 3 active mask holds on r_s, valid rows with a good id only
FLAG_BAD_ID = 8      # valid row with token id outside [0, V)

STAT_N_VALID, STAT_N_BAND, STAT_N_PPO, STAT_N_ACTIVE, STAT_N_BAD = range(5)

RD_MODES = ("none", "mask", "weight", "mask_weight")
SCALE_MODES = ("const", "token_mean")


@dataclass(frozen=True)
class Params:
    """Knobs of the decoupled MIS objective.

    band_lo, band_hi: discrepancy band on r_d (Eq. 4 with lo = 1/c, hi = c; App. A uses
    [1 - eps_1, 1 + eps_1]). clip_eps_lo, clip_eps_hi: the PPO interval
    [1 - eps_lo, 1 + eps_hi] on r_s (Eq. 2, Eq. 3; App. A allows them to differ).
    """

    band_lo: float = 0.5
    band_hi: float = 2.0
    clip_eps_lo: float = 0.2
    clip_eps_hi: float = 0.2
    rd_mode: str = "mask_weight"
    scale_mode: str = "token_mean"
    loss_scale: float = 1.0


# ---------------------------------------------------------------------------------------
# Input decoding
# ---------------------------------------------------------------------------------------
def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact value of bfloat16 numbers given as their uint16 bit patterns.

    A bfloat16 value is the float32 whose upper 16 bits are the pattern and whose lower
    16 bits are zero; float32 -> float64 is exact.
    """
    b = np.ascontiguousarray(bits).view(np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


def as_f64(x: np.ndarray) -> np.ndarray:
    """float32 / float64 arrays -> float64 (exact)."""
    return np.asarray(x, dtype=np.float64)


# ---------------------------------------------------------------------------------------
# Sampled-token log-probability (the quantity whose ratios Sec. 3.2 takes)
# ---------------------------------------------------------------------------------------
def row_logsumexp(z: np.ndarray) -> np.ndarray:
    """log sum_v exp z[t, v] for each row t, with the standard max shift.

    lse = M + log sum_v exp(z - M), M = max_v z. IEEE semantics: NaN anywhere in a row,
    +inf in a row, or an all -inf row give NaN.
    """
    z = np.asarray(z, dtype=np.float64)
    with np.errstate(invalid="ignore", over="ignore"):
        m = np.max(z, axis=1, keepdims=True)
        s = np.sum(np.exp(z - m), axis=1)
        return m[:, 0] + np.log(s)


def token_logprob(z: np.ndarray, ids: np.ndarray, lse: np.ndarray) -> np.ndarray:
    """log pi(y_t) = z[t, y_t] - lse_t; NaN where y_t is outside [0, V)."""
    T, V = z.shape
    ids = np.asarray(ids, dtype=np.int64)
    good = (ids >= 0) & (ids < V)
    lp = np.full(T, np.nan)
    rows = np.nonzero(good)[0]
    lp[rows] = z[rows, ids[rows]] - lse[rows]
    return lp


def logprob_fwd(logits: np.ndarray, ids: np.ndarray, chunk: int = 256):
    """Sampled-token log-probs and row log-sum-exps of float logits [T, V].

    Returns (lp [T], lse [T]) in float64.
    """
    z_all = np.asarray(logits)
    T = z_all.shape[0]
    lp = np.empty(T)
    lse = np.empty(T)
    for a in range(0, T, chunk):
        z = as_f64(z_all[a:a + chunk])
        lse[a:a + chunk] = row_logsumexp(z)
        lp[a:a + chunk] = token_logprob(z, ids[a:a + chunk], lse[a:a + chunk])
    return lp, lse


# ---------------------------------------------------------------------------------------
# Ratios and decisions (Eq. 1, Eq. 2, Eq. 3, Eq. 4)
# ---------------------------------------------------------------------------------------
def ratios(lp_theta, lp_ref, lp_mu):
    """r_s = pi_theta / pi_ref, r_d = pi_ref / mu_old and r = pi_theta / mu_old (Eq. 1).

    pi_ref is pi_old (exact old logits), pi_prox (PPO-EWMA, Eq. 5), or pi_async
    (Table 1, last row); the algebra is the same.
    """
    with np.errstate(invalid="ignore", over="ignore"):
        r_s = np.exp(lp_theta - lp_ref)
        r_d = np.exp(lp_ref - lp_mu)
        r = np.exp(lp_theta - lp_mu)
    return r_s, r_d, r


def band_mask(r_d, lo, hi):
    """M_[lo,hi](r_d) = 1{lo <= r_d <= hi} (Eq. 4, inclusive)."""
    with np.errstate(invalid="ignore"):
        return (lo <= r_d) & (r_d <= hi)


def ppo_active_mask(r, adv, eps_lo, eps_hi):
    """Eq. 3: 1{A >= 0} 1{r <= 1 + eps_hi} + 1{A < 0} 1{r >= 1 - eps_lo}."""
    with np.errstate(invalid="ignore"):
        return (((adv >= 0) & (r <= 1.0 + eps_hi)) |
                ((adv < 0) & (r >= 1.0 - eps_lo)))


def clipped_surrogate(r, adv, eps_lo, eps_hi):
    """Eq. 2 summand: min(r A, clip(r, 1 - eps_lo, 1 + eps_hi) A)."""
    with np.errstate(invalid="ignore"):
        return np.minimum(r * adv, np.clip(r, 1.0 - eps_lo, 1.0 + eps_hi) * adv)


def discrepancy_weight(r_d, band, rd_mode):
    """How r_d enters the objective: 1, M(r_d), r_d or M(r_d) r_d."""
    if rd_mode == "none":
        return np.ones_like(r_d)
    if rd_mode == "mask":
        return band.astype(np.float64)
    if rd_mode == "weight":
        return r_d.copy()
    if rd_mode == "mask_weight":
        return band * r_d
    raise ValueError(f"unknown rd_mode {rd_mode!r}")


def token_mean_scale(mask, loss_scale):
    """Token-mean normaliser loss_scale / max(1, sum_t m_t) (a reading of E_t in Eq. 2)."""
    n = int(np.count_nonzero(np.asarray(mask)))
    return float(loss_scale) / max(1, n)


def batch_scale(mask, params: Params) -> float:
    if params.scale_mode == "const":
        return float(params.loss_scale)
    if params.scale_mode == "token_mean":
        return token_mean_scale(mask, params.loss_scale)
    raise ValueError(f"unknown scale_mode {params.scale_mode!r}")


# ---------------------------------------------------------------------------------------
# The fused stage: forward values, MIS weights and dlogits
# ---------------------------------------------------------------------------------------
def token_terms(lp, valid, good, lp_mu, lp_ref, adv, ts, params: Params, scale: float):
    """Everything the objective derives from a token's log-prob (float64 arrays [n]).

    Ratios (Eq. 1), band (Eq. 4) and PPO (Eq. 3) decisions, the per-token loss (Eq. 2), the
    MIS weight of the Sec. 3.1 gradient and the flags. Rows that are not valid, or whose id
    is out of range, carry no loss, no weight and no decision bits.
    """
    ev = valid & good
    r_s, r_d, _ = ratios(lp, lp_ref, lp_mu)
    band = band_mask(r_d, params.band_lo, params.band_hi) & ev
    ppo = ppo_active_mask(r_s, adv, params.clip_eps_lo, params.clip_eps_hi) & ev
    uses_mask = params.rd_mode in ("mask", "mask_weight")
    gate = ppo & (band if uses_mask else ev)
    wd = discrepancy_weight(r_d, band, params.rd_mode)

    with np.errstate(invalid="ignore", over="ignore"):
        sur = clipped_surrogate(r_s, adv, params.clip_eps_lo, params.clip_eps_hi)
        loss_tok = np.where(ev, -wd * sur, 0.0)
        s = scale * ts
        # MIS gradient form (Sec. 3.1) with r = r_d r_s: d(loss)/d(lp_theta) = -s wd r_s A
        # on active tokens, 0 elsewhere.
        w = np.where(gate, s * wd * r_s * adv, 0.0)

    flags = np.zeros(len(lp), np.uint8)
    flags[valid] |= FLAG_VALID
    flags[valid & ~good] |= FLAG_BAD_ID
    flags[band] |= FLAG_BAND
    flags[ppo] |= FLAG_PPO
    return dict(r_s=r_s, r_d=r_d, band=band, ppo=ppo, gate=gate, loss_tok=loss_tok, w=w, s=s,
                flags=flags)


def per_token(z, ids, lp_mu, lp_ref, adv, mask, token_scale, params: Params, scale: float,
              want_dlogits: bool = True):
    """Evaluate the decoupled MIS objective on a block of rows (float64).

    z: float64 logits [n, V] (rows with m = 0 may hold anything; they are not read).
    scale: the batch scale (batch_scale over the whole batch the rows belong to).
    Returns a dict with lp, lse, r_s, r_d, band, ppo, gate, loss_tok, w, s, flags and
    (optionally) dlogits [n, V] float64.
    """
    n, V = z.shape
    ids = np.asarray(ids, dtype=np.int64)
    lp_mu = as_f64(lp_mu)
    lp_ref = as_f64(lp_ref)
    adv = as_f64(adv)
    valid = np.ones(n, bool) if mask is None else (np.asarray(mask) != 0)
    ts = np.ones(n) if token_scale is None else as_f64(token_scale)
    good = (ids >= 0) & (ids < V)
    ev = valid & good                      # rows that carry a loss and a gradient

    lse = np.zeros(n)
    lp = np.zeros(n)
    vr = np.nonzero(valid)[0]
    if vr.size:
        lse[vr] = row_logsumexp(z[vr])
        lp[vr] = token_logprob(z[vr], ids[vr], lse[vr])

    out = token_terms(lp, valid, good, lp_mu, lp_ref, adv, ts, params, scale)
    out.update(lp=np.where(valid, lp, 0.0), lse=lse, valid=valid, good=good)
    w = out["w"]
    if want_dlogits:
        d = np.zeros((n, V))
        er = np.nonzero(ev)[0]
        if er.size:
            with np.errstate(invalid="ignore", over="ignore"):
                p = np.exp(z[er] - lse[er, None])
            d[er] = w[er, None] * p
            d[er, ids[er]] -= w[er]
        out["dlogits"] = d
    return out


def stats_of(flags: np.ndarray, params: Params) -> np.ndarray:
    """[n_valid, n_band, n_ppo_active, n_active, n_bad_ids] from per-token flags.

    n_active counts tokens active after discrepancy masking and PPO clipping (the
    numerator of the Train-Infer Mask value, Sec. 5.2); without a mask it counts PPO only.
    """
    f = flags.astype(np.int64)
    valid = (f & FLAG_VALID) != 0
    band = (f & FLAG_BAND) != 0
    ppo = (f & FLAG_PPO) != 0
    bad = (f & FLAG_BAD_ID) != 0
    uses_mask = params.rd_mode in ("mask", "mask_weight")
    active = ppo & band if uses_mask else ppo
    return np.array([valid.sum(), band.sum(), ppo.sum(), active.sum(), bad.sum()], np.int64)


def decoupled_ppo_loss(logits, ids, lp_mu, lp_ref, adv, mask=None, token_scale=None,
                       params: Params = Params(), want_dlogits: bool = True,
                       chunk: int = 256):
    """The whole loss stage over a batch of T rows, float64.

    logits: float array [T, V] (float32 or float64; decode bfloat16 with bf16_bits_to_f64).
    Returns dict: lp [T], loss_tok [T], flags [T] u8, w [T], loss (float), stats [5],
    and dlogits [T, V] float64 when want_dlogits.
    """
    z_all = np.asarray(logits)
    T = z_all.shape[0]
    mask_arr = np.ones(T, np.uint8) if mask is None else np.asarray(mask)
    scale = batch_scale(mask_arr, params)
    parts = []
    for a in range(0, T, chunk):
        b = min(T, a + chunk)
        parts.append(per_token(
            as_f64(z_all[a:b]), ids[a:b], lp_mu[a:b], lp_ref[a:b], adv[a:b],
            mask_arr[a:b], None if token_scale is None else token_scale[a:b],
            params, scale, want_dlogits))
    out = {}
    for k in ("lp", "lse", "loss_tok", "w", "s", "flags", "r_s", "r_d", "band", "ppo",
              "gate", "valid", "good"):
        out[k] = np.concatenate([p[k] for p in parts]) if parts else np.zeros(0)
    out["flags"] = out["flags"].astype(np.uint8)
    if want_dlogits:
        out["dlogits"] = (np.concatenate([p["dlogits"] for p in parts]) if parts
                          else np.zeros((0, z_all.shape[1] if z_all.ndim == 2 else 0)))
    valid = out["valid"].astype(bool) if T else np.zeros(0, bool)
    with np.errstate(invalid="ignore"):
        out["loss"] = float(np.sum(np.where(valid, out["s"] * out["loss_tok"], 0.0)))
    out["stats"] = stats_of(out["flags"], params)
    out["scale"] = scale
    return out


# ---------------------------------------------------------------------------------------
# Vocabulary shards: the same stage when the vocabulary columns are split over devices
# ---------------------------------------------------------------------------------------
def vocab_shard_stats(z_shard, ids, vocab_start, mask=None):
    """One shard's row statistics: (lse_s, zy_s) float64 [n].

    lse_s = log sum over the shard's columns of exp z (-inf for a shard of -inf only, which
    then adds nothing to the global sum); zy_s = z[y] where the shard holds column y, else 0.
    Rows with m = 0 are not evaluated: lse_s = -inf, zy_s = 0.
    """
    z = as_f64(z_shard)
    n, Vs = z.shape
    ids = np.asarray(ids, dtype=np.int64)
    valid = np.ones(n, bool) if mask is None else (np.asarray(mask) != 0)
    lse = np.full(n, -np.inf)
    zy = np.zeros(n)
    vr = np.nonzero(valid)[0]
    if vr.size and Vs:
        all_neg_inf = np.all(z[vr] == -np.inf, axis=1)
        lse[vr] = np.where(all_neg_inf, -np.inf, row_logsumexp(z[vr]))
    yl = ids - vocab_start
    own = np.nonzero(valid & (yl >= 0) & (yl < Vs))[0]
    zy[own] = z[own, yl[own]]
    return lse, zy


def vocab_shard_combine(shard_lse):
    """Global lse = log sum_p exp lse_p over the shards ([P, n]); NaN where every shard is
    -inf (a row of -inf logits, as row_logsumexp gives, or a masked row)."""
    l = np.asarray(shard_lse, dtype=np.float64)
    with np.errstate(invalid="ignore", over="ignore", divide="ignore"):
        m = np.max(l, axis=0)
        out = m + np.log(np.sum(np.exp(l - m[None]), axis=0))
    return np.where(m == -np.inf, np.nan, out)


def vocab_shard_loss(z_shard, ids, vocab_start, V, lse, zy, lp_mu, lp_ref, adv, mask,
                     token_scale, params: Params, scale: float, want_dlogits: bool = True):
    """The loss stage on one shard given the global lse and z[y]: lp = z[y] - lse and the
    token terms as in per_token; dlogits for the shard's columns v (global v + vocab_start):
    w (exp(z - lse) - 1{v + vocab_start = y})."""
    z = as_f64(z_shard)
    n, Vs = z.shape
    ids = np.asarray(ids, dtype=np.int64)
    valid = np.ones(n, bool) if mask is None else (np.asarray(mask) != 0)
    good = (ids >= 0) & (ids < V)
    ts = np.ones(n) if token_scale is None else as_f64(token_scale)
    lse = as_f64(lse)
    lp = np.full(n, np.nan)
    ev = valid & good
    lp[ev] = as_f64(zy)[ev] - lse[ev]
    out = token_terms(lp, valid, good, as_f64(lp_mu), as_f64(lp_ref), as_f64(adv), ts, params,
                      scale)
    out.update(lp=np.where(valid, lp, 0.0), lse=lse, valid=valid, good=good)
    if want_dlogits:
        w = out["w"]
        d = np.zeros((n, Vs))
        er = np.nonzero(ev)[0]
        if er.size:
            with np.errstate(invalid="ignore", over="ignore"):
                d[er] = w[er, None] * np.exp(z[er] - lse[er, None])
            yl = ids[er] - vocab_start
            own = (yl >= 0) & (yl < Vs)
            d[er[own], yl[own]] -= w[er[own]]
        out["dlogits"] = d
    return out


# ---------------------------------------------------------------------------------------
# PPO-EWMA proxy (Sec. 5.2, Eq. 5; App. B) and its reset rule
# ---------------------------------------------------------------------------------------
def ewma_normalized_step(x_prox, x_new, beta, w_prev):
    """One step of the normalised recursion of App. B.

    w_t = 1 + beta w_{t-1};  x_prox_t = x_new / w_t + beta (w_{t-1} / w_t) x_prox_{t-1}.
    With w_{t-1} = 0 (no history) the closed form has the single term x_new, so the old
    buffer is not used. Returns (x_prox_t, w_t).
    """
    x_new = as_f64(x_new)
    w = 1.0 + beta * w_prev
    if w_prev == 0.0:
        return x_new.copy(), w
    return x_new / w + beta * (w_prev / w) * as_f64(x_prox), w


def ewma_fixed_step(x_prox, x_new, beta):
    """Fixed-decay form of Table 1 / Table 5: beta x_prox + (1 - beta) x_new."""
    return beta * as_f64(x_prox) + (1.0 - beta) * as_f64(x_new)


def ewma_reset():
    """Automatic reset (Sec. 5.2): x_prox <- x_new, and the normaliser restarts at w = 1."""
    return 1.0


def ewma_closed_form(history, beta):
    """Eq. 5 / App. B closed form: sum_k beta^(t-k) x_k / sum_k beta^(t-k), k = 0..t."""
    h = [as_f64(x) for x in history]
    t = len(h) - 1
    num = sum((beta ** (t - k)) * h[k] for k in range(t + 1))
    den = sum(beta ** (t - k) for k in range(t + 1))
    return num / den


def ewma_center_of_mass(beta):
    """Stationary centre of mass of the EWMA history, beta / (1 - beta) (App. B)."""
    return beta / (1.0 - beta)


def beta_from_window(w_stale):
    """Staleness-aware decay beta = W / (W + 2) (Sec. 5.2; App. B)."""
    return w_stale / (w_stale + 2.0)


def train_infer_mask_value(stats) -> float:
    """rho_t: fraction of valid tokens active after discrepancy masking and PPO clipping.

    With no valid tokens there is no evidence of collapse; rho is taken as 1.
    """
    n_valid = int(stats[STAT_N_VALID])
    return 1.0 if n_valid == 0 else int(stats[STAT_N_ACTIVE]) / n_valid


def ppo_clip_ratio(stats) -> float:
    """Fraction of valid tokens that PPO clipping removes, 1 - n_ppo_active / n_valid."""
    n_valid = int(stats[STAT_N_VALID])
    return 0.0 if n_valid == 0 else 1.0 - int(stats[STAT_N_PPO]) / n_valid


def reset_schedule(rhos, tau=0.9, patience=1):
    """Reset decisions for a sequence of rho_t values (Sec. 5.2; App. E).

    A reset fires when rho_t < tau has held for `patience` consecutive steps; the streak
    then restarts from zero.
    """
    out = []
    streak = 0
    for rho in rhos:
        streak = streak + 1 if rho < tau else 0
        fire = streak >= patience
        if fire:
            streak = 0
        out.append(fire)
    return out


# ---------------------------------------------------------------------------------------
# Interpolation proxies (Prop. 1; App. A; Table 4)
# ---------------------------------------------------------------------------------------
def log_linear_proxy_logprob(lp_mu, lp_theta, alpha):
    """Token-wise log-linear proxy: log pi_prox = alpha log mu_old + (1 - alpha) log pi_theta."""
    return alpha * as_f64(lp_mu) + (1.0 - alpha) * as_f64(lp_theta)


def linear_proxy_logprob(lp_mu, lp_theta, alpha):
    """Arithmetic proxy: pi_prox = alpha mu_old + (1 - alpha) pi_theta, as a log-prob."""
    return np.log(alpha * np.exp(as_f64(lp_mu)) + (1.0 - alpha) * np.exp(as_f64(lp_theta)))


def effective_thresholds(mask_lo, mask_hi, clip_lo, clip_hi, alpha, kind):
    """Bounds on the total ratio r_theta = pi_theta / mu_old that a proxy induces (App. A).

    mask_lo, mask_hi: the band [lo, hi] applied to r_d; clip_lo, clip_hi: the PPO interval
    [1 - eps_lo, 1 + eps_hi] applied to r_s; alpha: behaviour-policy weight.
    kind "log_linear": r_d = r_theta^(1-alpha), r_s = r_theta^alpha.
    kind "linear": r_d = alpha + (1 - alpha) r_theta, r_s = r_theta / (alpha + (1-alpha) r_theta).
    Returns ((mask bounds on r_theta), (clip bounds on r_theta)); the clip upper bound
    applies to A >= 0 and the lower one to A < 0.
    """
    if kind == "log_linear":
        m = (mask_lo ** (1.0 / (1.0 - alpha)), mask_hi ** (1.0 / (1.0 - alpha)))
        c = (clip_lo ** (1.0 / alpha), clip_hi ** (1.0 / alpha))
    elif kind == "linear":
        m = ((mask_lo - alpha) / (1.0 - alpha), (mask_hi - alpha) / (1.0 - alpha))
        # r_s = x / (alpha + (1 - alpha) x) = b  <=>  x = alpha b / (1 - (1 - alpha) b)
        c = tuple(alpha * b / (1.0 - (1.0 - alpha) * b) for b in (clip_lo, clip_hi))
    else:
        raise ValueError(f"unknown interpolation kind {kind!r}")
    return m, c


# ---------------------------------------------------------------------------------------
# Loss stage with the LM head folded in
# ---------------------------------------------------------------------------------------
def lm_head_loss(hidden, weight, ids, lp_mu, lp_ref, adv, mask=None, token_scale=None,
                 params: Params = Params(), want_grads: bool = True):
    """The loss stage on logits z = hidden @ weight^T, with gradients for both factors.

    hidden [T, d] and weight [V, d] are float arrays (decode bfloat16 with
    bf16_bits_to_f64); weight is the LM head in the [out, in] layout, so row v of weight
    produces logit v. The logits are formed with one float64 matrix product, the loss stage
    is decoupled_ppo_loss on them, and the chain rule through z = hidden weight^T gives
        d L / d hidden = dlogits @ weight,     d L / d weight = dlogits^T @ hidden.
    Returns decoupled_ppo_loss's dict plus "dhidden" [T, d] and "dweight" [V, d] when
    want_grads. lp_ref may be an interpolated proxy computed by the caller (App. A).
    """
    h = as_f64(hidden)
    wt = as_f64(weight)
    z = h @ wt.T
    out = decoupled_ppo_loss(z, ids, lp_mu, lp_ref, adv, mask, token_scale, params,
                             want_dlogits=want_grads)
    out["logits"] = z
    if want_grads:
        g = out["dlogits"]
        out["dhidden"] = g @ wt
        out["dweight"] = g.T @ h
    return out


def versioned_logprob(logits_by_version, version, ids):
    """Exact old log-probs of a partial rollout (Sec. 5.1, snapshot route): token t's
    log-prob under the policy version that generated it, log pi_{v_t}(y_t), with v_t =
    version[t]; NaN where v_t is not one of the given versions (or y_t is out of range)."""
    version = np.asarray(version)
    ids = np.asarray(ids)
    T = ids.shape[0]
    out = np.full(T, np.nan)
    for v, z in enumerate(logits_by_version):
        rows = np.nonzero(version == v)[0]
        if rows.size:
            lp, _ = logprob_fwd(as_f64(np.asarray(z)[rows]), ids[rows])
            out[rows] = lp
    return out
