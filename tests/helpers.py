"""Shared helpers of the GPU parity tests: oracle runs on the same input bits, and the
comparison rules.

Tolerances, each with the arithmetic it follows from:
  * decisions (band, PPO, flags): bit-exact on every token whose oracle log-ratio is more
    than DELTA = 1e-4 from a threshold (the float32 log-prob error is ~1e-6);
  * lp, lse, l_t: |gpu - ref| <= rtol * max(|ref|, 1), rtol = 1e-5 (fp32 logits) or 2e-3
    (bf16 logits) as the contract states, and a tight implementation bound TIGHT = 2e-5
    that a dropped or doubled vocabulary element would break;
  * scalar loss: |gpu - ref| <= 1e-5 * sum_t |m_t s_t l_t| + 1e-30;
  * dlogits: |gpu - ref| <= DREL * |ref| + 2^-22 * |w_t| per element. For bf16 output
    DREL = 2^-8 + 2^-11: rounding to nearest bf16 (8 significant bits) is off by at most
    2^-8 |ref|, and the exponentials the resident kernels keep as fp16 (11 significant
    bits) add at most 2^-11 before that rounding. The floor covers exponentials in fp16's
    subnormal range, absolute error <= 2^-25 each, scaled by w_t 2^(n_c - lse2) < 2 w_t:
    <= 2^-24 |w_t|, with a factor 4 to spare. For fp32 output DREL = 2e-5 (the fp32
    log-sum-exp's error, ~1e-6, moves every softmax entry by that much relatively). Plus
    the contract's absolute bound 1e-3 on bf16 dlogits wherever a correctly rounded value
    can meet it: |ref| <= 1/4, where half a bf16 ulp is <= 2^-11 and the fp16 step adds
    <= 2^-13.
"""
from __future__ import annotations

import math

import numpy as np
import torch

import oracle

DELTA = 1e-4
TIGHT = 2e-5


def bits_of(t: torch.Tensor) -> np.ndarray:
    """Host copy of a tensor's values as the oracle reads them (float64)."""
    t = t.detach().cpu()
    if t.dtype == torch.bfloat16:
        return oracle.bf16_bits_to_f64(t.view(torch.int16).numpy().view(np.uint16))
    return t.double().numpy()


def rtol_for(dtype):
    return 2e-3 if dtype == torch.bfloat16 else 1e-5


def oracle_params(band, eps, rd_mode, scale_mode, loss_scale):
    f = lambda x: float(np.float32(x))  # the kernel receives float32 parameters
    return oracle.Params(f(band[0]), f(band[1]), f(eps[0]), f(eps[1]), rd_mode, scale_mode,
                         f(loss_scale))


def tie_mask(ref, params: oracle.Params):
    """Tokens within DELTA (in log-ratio) of a band or clip threshold."""
    with np.errstate(divide="ignore", invalid="ignore"):
        ls = np.log(ref["r_s"])
        ld = np.log(ref["r_d"])
        th_s = np.log([max(1.0 - params.clip_eps_lo, 1e-300), 1.0 + params.clip_eps_hi])
        th_d = np.log([max(params.band_lo, 1e-300), params.band_hi])
        near_s = np.min(np.abs(ls[:, None] - th_s[None]), axis=1) <= DELTA
        near_d = np.min(np.abs(ld[:, None] - th_d[None]), axis=1) <= DELTA
    return near_s | near_d


def assert_close_rel(gpu, ref, rtol, what, floor=1.0, mask=None):
    gpu = np.asarray(gpu, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    if mask is not None:
        gpu, ref = gpu[mask], ref[mask]
    both_nan = np.isnan(gpu) & np.isnan(ref)
    assert np.array_equal(np.isnan(gpu), np.isnan(ref)), f"{what}: NaN pattern differs"
    g, r = gpu[~both_nan], ref[~both_nan]
    if g.size == 0:
        return 0.0
    err = np.abs(g - r) / np.maximum(np.abs(r), floor)
    worst = float(err.max())
    assert worst <= rtol, f"{what}: max rel err {worst:.3e} > {rtol:.1e}"
    return worst


def check_dlogits_rows(gpu_rows, ref_rows, w, out_dtype, what="dlogits", lp=None):
    """gpu_rows: float64 values of the kernel's dlogits rows; ref_rows: oracle float64.
    With lp (the oracle's log-probs of the rows), the sampled entry w (p_y - 1), the one entry
    whose sign is opposite to w's, may also be off by |w| p_y TIGHT max(|lp|, 1): it carries
    the log-prob's own absolute error (the TIGHT bound of the lp check) through p_y, which a
    bound relative to |p_y - 1| does not cover once p_y is close to 1 (a vocabulary of a
    few entries, or a confident token)."""
    drel = 2.0 ** -8 + 2.0 ** -11 if out_dtype == torch.bfloat16 else 2e-5
    bound = drel * np.abs(ref_rows) + 2.0 ** -22 * np.abs(w)[:, None] + 1e-30
    if lp is not None:
        wy = np.asarray(w)[:, None]
        ysel = (ref_rows * wy) < 0
        p_y = np.exp(np.minimum(np.nan_to_num(np.asarray(lp, dtype=np.float64)), 0.0))[:, None]
        ytol = np.abs(wy) * p_y * TIGHT * np.maximum(np.abs(np.nan_to_num(np.asarray(lp)))[:, None], 1.0)
        bound = bound + np.where(ysel, ytol, 0.0)
    nan_ref = np.isnan(ref_rows)
    assert np.array_equal(np.isnan(gpu_rows), nan_ref), f"{what}: NaN pattern differs"
    err = np.where(nan_ref, 0.0, np.abs(gpu_rows - ref_rows))
    bad = err > np.where(nan_ref, 0.0, bound)
    assert not bad.any(), (f"{what}: {int(bad.sum())} elements out of bound, worst excess "
                           f"{float((err - bound).max()):.3e}")
    if out_dtype == torch.bfloat16:
        # The contract's absolute bound, where a correctly rounded value can meet it.
        small = np.abs(np.where(nan_ref, 0.0, ref_rows)) <= 0.25
        worst = float(np.max(np.where(small, err, 0.0), initial=0.0))
        assert worst <= 1e-3, f"{what}: absolute error {worst:.3e} > 1e-3"


def run_oracle(logits, ids, lp_mu, lp_ref, adv, mask, tscale, params, want_dlogits=True):
    return oracle.decoupled_ppo_loss(
        bits_of(logits), ids.cpu().numpy(), lp_mu.cpu().double().numpy(),
        lp_ref.cpu().double().numpy(), adv.cpu().double().numpy(),
        None if mask is None else mask.cpu().numpy(),
        None if tscale is None else tscale.cpu().double().numpy(),
        params=params, want_dlogits=want_dlogits)


def oracle_anchor(logits, ids):
    """Sampled-token log-probs from the oracle, used only to synthesise reference inputs."""
    lp, _ = oracle.logprob_fwd(bits_of(logits), ids.cpu().numpy())
    return torch.from_numpy(lp)


def torch_anchor(logits, ids, chunk=1024):
    """Sampled-token log-probs from PyTorch (float32, on the logits' device), used only to
    synthesise reference inputs for workloads too large for the oracle."""
    T = logits.shape[0]
    out = torch.empty(T, dtype=torch.float64, device=logits.device)
    for a in range(0, T, chunk):
        z = logits[a:a + chunk].float()
        lse = torch.logsumexp(z, dim=1)
        out[a:a + chunk] = (z.gather(1, ids[a:a + chunk, None])[:, 0] - lse).double()
    return out


def compare_loss(res, ref, params, logits_dtype, dl_dtype=None, check_dlogits=True,
                 rows=None):
    """Compare a LossResult with an oracle result (optionally on a subset of rows)."""
    sel = slice(None) if rows is None else rows
    ties = tie_mask(ref, params)
    ok = ~ties
    rt = rtol_for(logits_dtype)
    lp = res.logp.cpu().double().numpy()[sel]
    assert_close_rel(lp, ref["lp"], rt, "lp")
    assert_close_rel(lp, ref["lp"], TIGHT, "lp (tight)")
    lt = res.loss_tok.cpu().double().numpy()[sel]
    assert_close_rel(lt, ref["loss_tok"], rt, "loss_tok", mask=ok)
    assert_close_rel(lt, ref["loss_tok"], 1e-4, "loss_tok (tight)", mask=ok)
    if res.flags is not None:
        fl = res.flags.cpu().numpy()[sel]
        assert np.array_equal(fl[ok], ref["flags"][ok]), "flags differ away from ties"
    if check_dlogits and res.dlogits is not None:
        g = bits_of(res.dlogits)[sel] if rows is None else bits_of(res.dlogits[rows])
        w = ref["w"].copy()
        w[ties] = np.maximum(np.abs(w[ties]), 1.0)      # tie tokens: allow either decision
        tie_rows = np.nonzero(ties)[0]
        g2 = g.copy()
        r2 = ref["dlogits"].copy()
        g2[tie_rows] = 0.0
        r2[tie_rows] = 0.0
        check_dlogits_rows(g2, r2, w, dl_dtype or logits_dtype, lp=ref["lp"])
    return int(ties.sum())
