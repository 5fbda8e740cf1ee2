"""MI355X (gfx950) loss stage of decoupled off-policy PPO (arXiv 2605.12070).

Thin Python binding over libdppo.so: every function here only checks tensors and passes
device pointers and the current HIP stream to the C ABI (include/dppo.h); all arithmetic
runs in the library's kernels. PyTorch supplies device memory and streams.

    from paper_2605_12070_amd import decoupled_ppo_loss_fwd_bwd
    res = decoupled_ppo_loss_fwd_bwd(logits, ids, lp_mu, lp_ref, adv)
    res.loss, res.logp, res.dlogits, res.stats
"""
from __future__ import annotations

import ctypes as C
from dataclasses import dataclass

import torch

from . import _lib
from ._lib import (DppoError, FLAG_BAD_ID, FLAG_BAND, FLAG_PPO, FLAG_VALID,  # noqa: F401
                   RD_MODES, REF_MODES, SCALE_MODES, STAT_N_ACTIVE, STAT_N_BAD, STAT_N_BAND, STAT_N_PPO,
                   STAT_N_VALID)

__all__ = [
    "logprob_fwd", "decoupled_ppo_loss_fwd_bwd", "decoupled_ppo_loss", "ewma_proxy_update",
    "LossResult",
    "EwmaProxy", "beta_from_window", "train_infer_mask_value", "ppo_clip_ratio",
    "DecoupledPPOLoss", "DppoError", "set_path_policy", "KernelTimer", "row_kernel_name", "effective_thresholds",
    "fused_lm_head_loss_fwd_bwd", "LmHeadResult", "lm_head_workspace_bytes",
    "fused_lm_head_loss_fwd_bwd_noalloc",
    "logprob_fwd_versioned", "EwmaProxyDevice", "vocab_shard_stats", "vocab_shard_combine",
    "decoupled_ppo_loss_shard_fwd_bwd", "FusedLMHeadLoss",
]


def _stream(dev: torch.device) -> int:
    return torch.cuda.current_stream(dev).cuda_stream


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return _lib.DPPO_BF16
    if t.dtype == torch.float32:
        return _lib.DPPO_F32
    raise TypeError(f"logits must be bfloat16 or float32, got {t.dtype}")


def _matrix(t: torch.Tensor, name: str):
    if t.dim() != 2 or t.stride(1) != 1:
        raise ValueError(f"{name} must be a 2-D tensor with unit stride in its last dim")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    return t.data_ptr(), t.shape[0], t.shape[1], t.stride(0)


def _vec(t, T, dtype, name, dev, optional=False):
    if t is None:
        if optional:
            return None
        raise ValueError(f"{name} is required")
    if t.dtype != dtype or t.dim() != 1 or t.shape[0] != T or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous [{T}] {dtype} tensor")
    if t.device != dev:
        raise ValueError(f"{name} must live on {dev}")
    return t.data_ptr()


def logprob_fwd(logits: torch.Tensor, token_ids: torch.Tensor, with_lse: bool = False):
    """log pi(y_t) for every row of logits [T, V] (bf16 or fp32). Returns lp [T] fp32,
    or (lp, lse) when with_lse."""
    ptr, T, V, ld = _matrix(logits, "logits")
    dev = logits.device
    ids = _vec(token_ids, T, torch.int64, "token_ids", dev)
    lp = torch.empty(T, dtype=torch.float32, device=dev)
    lse = torch.empty(T, dtype=torch.float32, device=dev) if with_lse else None
    st = _lib.lib().logprob_fwd(ptr, _dtype_code(logits), T, V, ld, ids, lp.data_ptr(),
                                lse.data_ptr() if lse is not None else None, _stream(dev))
    _lib.check(st, "logprob_fwd")
    return (lp, lse) if with_lse else lp


def logprob_fwd_versioned(logits_by_version, version_ids: torch.Tensor, token_ids: torch.Tensor,
                          with_lse: bool = False):
    """log pi_{v_t}(y_t) for tokens produced by different policy versions: token t reads row t
    of logits_by_version[version_ids[t]] (exact old log-probs of a partial rollout)."""
    mats = list(logits_by_version)
    if not mats or len(mats) > _lib.MAX_VERSIONS:
        raise ValueError(f"between 1 and {_lib.MAX_VERSIONS} versions")
    infos = [_matrix(z, f"logits[{i}]") for i, z in enumerate(mats)]
    _, T, V, ld = infos[0]
    if any(i[1:] != (T, V, ld) for i in infos) or any(z.dtype != mats[0].dtype for z in mats):
        raise ValueError("all versions must share dtype, shape and row stride")
    dev = mats[0].device
    ver = _vec(version_ids, T, torch.int32, "version_ids", dev)
    ids = _vec(token_ids, T, torch.int64, "token_ids", dev)
    lp = torch.empty(T, dtype=torch.float32, device=dev)
    lse = torch.empty(T, dtype=torch.float32, device=dev) if with_lse else None
    arr = (C.c_void_p * len(mats))(*[i[0] for i in infos])
    st = _lib.lib().logprob_fwd_versioned(arr, len(mats), _dtype_code(mats[0]), T, V, ld, ver, ids,
                                          lp.data_ptr(), lse.data_ptr() if lse is not None else None,
                                          _stream(dev))
    _lib.check(st, "logprob_fwd_versioned")
    return (lp, lse) if with_lse else lp


@dataclass
class LossResult:
    loss: torch.Tensor          # [1] fp32: sum_t m_t s_t l_t
    logp: torch.Tensor          # [T] fp32: log pi_theta(y_t)
    loss_tok: torch.Tensor      # [T] fp32: l_t
    flags: torch.Tensor | None  # [T] uint8
    stats: torch.Tensor         # [5] int32
    dlogits: torch.Tensor | None


def decoupled_ppo_loss_fwd_bwd(logits, token_ids, logp_mu_old, logp_ref, advantages,
                               loss_mask=None, token_scale=None, *, band=(0.5, 2.0),
                               clip_eps=(0.2, 0.2), rd_mode="mask_weight",
                               scale_mode="token_mean", loss_scale=1.0, ref_mode="given",
                               alpha=0.5, want_dlogits=True, dlogits=None, want_flags=True,
                               out: LossResult | None = None) -> LossResult:
    """Fused loss stage: log-prob, ratios, band and clip decisions, per-token loss, stats and
    dlogits = w (softmax - onehot). `dlogits` may be the logits tensor itself (in place) or
    a preallocated tensor; `out` reuses all output buffers. ref_mode "log_linear" or
    "linear" interpolates the reference between mu_old (weight alpha) and the current
    policy instead of reading logp_ref (which may then be None)."""
    ptr, T, V, ld = _matrix(logits, "logits")
    dev = logits.device
    ids = _vec(token_ids, T, torch.int64, "token_ids", dev)
    mu = _vec(logp_mu_old, T, torch.float32, "logp_mu_old", dev)
    if ref_mode not in REF_MODES:
        raise ValueError(f"ref_mode in {list(REF_MODES)}")
    ref = _vec(logp_ref, T, torch.float32, "logp_ref", dev, optional=ref_mode != "given")
    adv = _vec(advantages, T, torch.float32, "advantages", dev)
    msk = _vec(loss_mask, T, torch.uint8, "loss_mask", dev, optional=True)
    tsc = _vec(token_scale, T, torch.float32, "token_scale", dev, optional=True)
    if rd_mode not in RD_MODES or scale_mode not in SCALE_MODES:
        raise ValueError(f"rd_mode in {list(RD_MODES)}, scale_mode in {list(SCALE_MODES)}")
    if out is None:
        f32 = dict(dtype=torch.float32, device=dev)
        out = LossResult(
            loss=torch.empty(1, **f32), logp=torch.empty(T, **f32),
            loss_tok=torch.empty(T, **f32),
            flags=torch.empty(T, dtype=torch.uint8, device=dev) if want_flags else None,
            stats=torch.empty(_lib.N_STATS, dtype=torch.int32, device=dev), dlogits=None)
    if want_dlogits:
        if dlogits is None:
            dlogits = out.dlogits if out.dlogits is not None else torch.empty_like(logits)
        if dlogits.dtype != logits.dtype or dlogits.shape != logits.shape or dlogits.stride(1) != 1:
            raise ValueError("dlogits must match logits in dtype and shape, unit last stride")
        out.dlogits = dlogits
        d_ptr, ldd = dlogits.data_ptr(), dlogits.stride(0)
    else:
        out.dlogits = None
        d_ptr, ldd = None, 0
    p = _lib.DppoParams(float(band[0]), float(band[1]), float(clip_eps[0]), float(clip_eps[1]),
                        RD_MODES[rd_mode], SCALE_MODES[scale_mode], float(loss_scale),
                        REF_MODES[ref_mode], float(alpha))
    st = _lib.lib().decoupled_ppo_loss_fwd_bwd(
        ptr, _dtype_code(logits), T, V, ld, ids, mu, ref, adv, msk, tsc, C.byref(p),
        out.logp.data_ptr(), out.loss_tok.data_ptr(), out.loss.data_ptr(),
        out.flags.data_ptr() if out.flags is not None else None, d_ptr, ldd,
        out.stats.data_ptr(), _stream(dev))
    _lib.check(st, "decoupled_ppo_loss_fwd_bwd")
    return out


def decoupled_ppo_loss(logits, y, lp_mu, lp_ref, adv, mask=None, band=(0.5, 2.0),
                       eps=(0.2, 0.2), rd_mode="mask_weight", scale="token_mean"):
    """The loss stage in the short form: returns (loss, lp, dlogits, stats), the scalar loss
    as a 0-d tensor. Argument marshalling over decoupled_ppo_loss_fwd_bwd."""
    r = decoupled_ppo_loss_fwd_bwd(logits, y, lp_mu, lp_ref, adv, mask, band=band, clip_eps=eps,
                                   rd_mode=rd_mode, scale_mode=scale)
    return r.loss[0], r.logp, r.dlogits, r.stats


def vocab_shard_stats(logits_shard, token_ids, vocab_start: int, vocab_size: int,
                      loss_mask=None):
    """One vocabulary shard's row statistics: (shard_lse [T], shard_zy [T]) float32, the
    log-sum-exp over the shard's columns and z[y] where the shard holds column y (0 else).
    logits_shard [T, Vs] holds columns [vocab_start, vocab_start + Vs) of a vocab_size-
    column vocabulary."""
    ptr, T, Vs, ld = _matrix(logits_shard, "logits_shard")
    dev = logits_shard.device
    ids = _vec(token_ids, T, torch.int64, "token_ids", dev)
    msk = _vec(loss_mask, T, torch.uint8, "loss_mask", dev, optional=True)
    lse = torch.empty(T, dtype=torch.float32, device=dev)
    zy = torch.empty(T, dtype=torch.float32, device=dev)
    st = _lib.lib().vocab_shard_stats(ptr, _dtype_code(logits_shard), T, Vs, ld, int(vocab_start),
                                      int(vocab_size), ids, msk, lse.data_ptr(), zy.data_ptr(),
                                      _stream(dev))
    _lib.check(st, "vocab_shard_stats")
    return lse, zy


def vocab_shard_combine(shard_lse: torch.Tensor) -> torch.Tensor:
    """Global per-token log-sum-exp from the gathered shard statistics [P, T] (shard order)."""
    if not (shard_lse.is_cuda and shard_lse.dtype == torch.float32 and shard_lse.dim() == 2
            and shard_lse.is_contiguous()):
        raise ValueError("shard_lse must be a contiguous [P, T] float32 GPU tensor")
    P, T = shard_lse.shape
    lse = torch.empty(T, dtype=torch.float32, device=shard_lse.device)
    st = _lib.lib().vocab_shard_combine(shard_lse.data_ptr(), P, T, lse.data_ptr(),
                                        _stream(shard_lse.device))
    _lib.check(st, "vocab_shard_combine")
    return lse


def decoupled_ppo_loss_shard_fwd_bwd(logits_shard, vocab_start: int, vocab_size: int, lse, zy,
                                     token_ids, logp_mu_old, logp_ref, advantages,
                                     loss_mask=None, token_scale=None, *, band=(0.5, 2.0),
                                     clip_eps=(0.2, 0.2), rd_mode="mask_weight",
                                     scale_mode="token_mean", loss_scale=1.0, ref_mode="given",
                                     alpha=0.5, want_dlogits=True, dlogits=None,
                                     want_flags=True) -> LossResult:
    """decoupled_ppo_loss_fwd_bwd on one vocabulary shard, from the global lse and z[y]
    (vocab_shard_combine's lse, the all-reduced shard_zy): the per-token outputs, loss and
    stats (the same on every shard) and this shard's columns of dlogits."""
    ptr, T, Vs, ld = _matrix(logits_shard, "logits_shard")
    dev = logits_shard.device
    ids = _vec(token_ids, T, torch.int64, "token_ids", dev)
    lse_p = _vec(lse, T, torch.float32, "lse", dev)
    zy_p = _vec(zy, T, torch.float32, "zy", dev)
    mu = _vec(logp_mu_old, T, torch.float32, "logp_mu_old", dev)
    if ref_mode not in REF_MODES:
        raise ValueError(f"ref_mode in {list(REF_MODES)}")
    ref = _vec(logp_ref, T, torch.float32, "logp_ref", dev, optional=ref_mode != "given")
    adv = _vec(advantages, T, torch.float32, "advantages", dev)
    msk = _vec(loss_mask, T, torch.uint8, "loss_mask", dev, optional=True)
    tsc = _vec(token_scale, T, torch.float32, "token_scale", dev, optional=True)
    if rd_mode not in RD_MODES or scale_mode not in SCALE_MODES:
        raise ValueError(f"rd_mode in {list(RD_MODES)}, scale_mode in {list(SCALE_MODES)}")
    f32 = dict(dtype=torch.float32, device=dev)
    out = LossResult(
        loss=torch.empty(1, **f32), logp=torch.empty(T, **f32), loss_tok=torch.empty(T, **f32),
        flags=torch.empty(T, dtype=torch.uint8, device=dev) if want_flags else None,
        stats=torch.empty(_lib.N_STATS, dtype=torch.int32, device=dev), dlogits=None)
    d_ptr, ldd = None, 0
    if want_dlogits:
        if dlogits is None:
            dlogits = torch.empty_like(logits_shard)
        if (dlogits.dtype != logits_shard.dtype or dlogits.shape != logits_shard.shape
                or dlogits.stride(1) != 1):
            raise ValueError("dlogits must match logits_shard in dtype and shape, unit last stride")
        out.dlogits = dlogits
        d_ptr, ldd = dlogits.data_ptr(), dlogits.stride(0)
    p = _lib.DppoParams(float(band[0]), float(band[1]), float(clip_eps[0]), float(clip_eps[1]),
                        RD_MODES[rd_mode], SCALE_MODES[scale_mode], float(loss_scale),
                        REF_MODES[ref_mode], float(alpha))
    st = _lib.lib().decoupled_ppo_loss_shard_fwd_bwd(
        ptr, _dtype_code(logits_shard), T, Vs, ld, int(vocab_start), int(vocab_size), ids, lse_p,
        zy_p, mu, ref, adv, msk, tsc, C.byref(p), out.logp.data_ptr(), out.loss_tok.data_ptr(),
        out.loss.data_ptr(), out.flags.data_ptr() if out.flags is not None else None, d_ptr, ldd,
        out.stats.data_ptr(), _stream(dev))
    _lib.check(st, "decoupled_ppo_loss_shard_fwd_bwd")
    return out


@dataclass
class LmHeadResult:
    loss: torch.Tensor          # [1] fp32
    logp: torch.Tensor          # [T] fp32
    loss_tok: torch.Tensor      # [T] fp32
    flags: torch.Tensor | None  # [T] uint8
    stats: torch.Tensor         # [5] int32
    dhidden: torch.Tensor | None  # [T, d] fp32
    dweight: torch.Tensor | None  # [V, d] fp32
    workspace: torch.Tensor | None  # scratch, reusable by the next call (out=)


def lm_head_workspace_bytes(T: int, d: int, V: int, vocab_chunk: int = 0) -> int:
    n = _lib.lib().fused_lm_head_workspace_bytes(T, d, V, vocab_chunk)
    if n < 0:
        raise ValueError(f"sizes out of range: T={T}, d={d}, V={V}")
    return n


def fused_lm_head_loss_fwd_bwd(hidden, weight, token_ids, logp_mu_old, logp_ref, advantages,
                               loss_mask=None, token_scale=None, *, band=(0.5, 2.0),
                               clip_eps=(0.2, 0.2), rd_mode="mask_weight",
                               scale_mode="token_mean", loss_scale=1.0, ref_mode="given",
                               alpha=0.5, want_grads=True, vocab_chunk=0, want_flags=True,
                               out: LmHeadResult | None = None) -> LmHeadResult:
    """The loss stage on logits hidden @ weight.T (never materialised), with d L / d hidden
    and d L / d weight. hidden [T, d] and weight [V, d] are contiguous bf16 GPU tensors."""
    for t, name in ((hidden, "hidden"), (weight, "weight")):
        if t.dtype != torch.bfloat16 or t.dim() != 2 or not t.is_contiguous() or not t.is_cuda:
            raise ValueError(f"{name} must be a contiguous 2-D bf16 GPU tensor")
    T, d = hidden.shape
    V = weight.shape[0]
    if weight.shape[1] != d:
        raise ValueError("hidden and weight disagree on d")
    dev = hidden.device
    ids = _vec(token_ids, T, torch.int64, "token_ids", dev)
    mu = _vec(logp_mu_old, T, torch.float32, "logp_mu_old", dev)
    if ref_mode not in REF_MODES:
        raise ValueError(f"ref_mode in {list(REF_MODES)}")
    ref = _vec(logp_ref, T, torch.float32, "logp_ref", dev, optional=ref_mode != "given")
    adv = _vec(advantages, T, torch.float32, "advantages", dev)
    msk = _vec(loss_mask, T, torch.uint8, "loss_mask", dev, optional=True)
    tsc = _vec(token_scale, T, torch.float32, "token_scale", dev, optional=True)
    if rd_mode not in RD_MODES or scale_mode not in SCALE_MODES:
        raise ValueError(f"rd_mode in {list(RD_MODES)}, scale_mode in {list(SCALE_MODES)}")
    nws = lm_head_workspace_bytes(T, d, V, vocab_chunk)
    if out is None:
        f32 = dict(dtype=torch.float32, device=dev)
        out = LmHeadResult(
            loss=torch.empty(1, **f32), logp=torch.empty(T, **f32), loss_tok=torch.empty(T, **f32),
            flags=torch.empty(T, dtype=torch.uint8, device=dev) if want_flags else None,
            stats=torch.empty(_lib.N_STATS, dtype=torch.int32, device=dev),
            dhidden=torch.empty(T, d, **f32) if want_grads else None,
            dweight=torch.empty(V, d, **f32) if want_grads else None,
            workspace=torch.empty(max(nws, 1), dtype=torch.uint8, device=dev))
    if out.workspace.numel() < nws:
        out.workspace = torch.empty(nws, dtype=torch.uint8, device=dev)
    p = _lib.DppoParams(float(band[0]), float(band[1]), float(clip_eps[0]), float(clip_eps[1]),
                        RD_MODES[rd_mode], SCALE_MODES[scale_mode], float(loss_scale),
                        REF_MODES[ref_mode], float(alpha))
    st = _lib.lib().fused_lm_head_loss_fwd_bwd(
        hidden.data_ptr(), weight.data_ptr(), _lib.DTYPE_BF16, T, d, V, ids, mu, ref, adv, msk,
        tsc, C.byref(p), out.logp.data_ptr(), out.loss_tok.data_ptr(), out.loss.data_ptr(),
        out.flags.data_ptr() if out.flags is not None else None, out.stats.data_ptr(),
        out.dhidden.data_ptr() if out.dhidden is not None else None,
        out.dweight.data_ptr() if out.dweight is not None else None,
        int(vocab_chunk), out.workspace.data_ptr(), out.workspace.numel(), _stream(dev))
    _lib.check(st, "fused_lm_head_loss_fwd_bwd")
    return out


def fused_lm_head_loss_fwd_bwd_noalloc(hidden, weight, token_ids, logp_mu_old, logp_ref,
                                       advantages, loss_mask=None, token_scale=None, *,
                                       band=(0.5, 2.0), clip_eps=(0.2, 0.2),
                                       rd_mode="mask_weight", scale_mode="token_mean",
                                       loss_scale=1.0, ref_mode="given", alpha=0.5,
                                       want_grads=True, want_flags=True):
    """fused_lm_head_loss_fwd_bwd with the library's static device scratch as workspace (the
    C call allocates nothing). Returns (LmHeadResult, vocab_chunk_used); the result's
    workspace field is None. Output tensors are allocated here, by the caller's side."""
    for t, name in ((hidden, "hidden"), (weight, "weight")):
        if t.dtype != torch.bfloat16 or t.dim() != 2 or not t.is_contiguous() or not t.is_cuda:
            raise ValueError(f"{name} must be a contiguous 2-D bf16 GPU tensor")
    T, d = hidden.shape
    V = weight.shape[0]
    if weight.shape[1] != d:
        raise ValueError("hidden and weight disagree on d")
    dev = hidden.device
    ids = _vec(token_ids, T, torch.int64, "token_ids", dev)
    mu = _vec(logp_mu_old, T, torch.float32, "logp_mu_old", dev)
    if ref_mode not in REF_MODES:
        raise ValueError(f"ref_mode in {list(REF_MODES)}")
    ref = _vec(logp_ref, T, torch.float32, "logp_ref", dev, optional=ref_mode != "given")
    adv = _vec(advantages, T, torch.float32, "advantages", dev)
    msk = _vec(loss_mask, T, torch.uint8, "loss_mask", dev, optional=True)
    tsc = _vec(token_scale, T, torch.float32, "token_scale", dev, optional=True)
    if rd_mode not in RD_MODES or scale_mode not in SCALE_MODES:
        raise ValueError(f"rd_mode in {list(RD_MODES)}, scale_mode in {list(SCALE_MODES)}")
    f32 = dict(dtype=torch.float32, device=dev)
    out = LmHeadResult(
        loss=torch.empty(1, **f32), logp=torch.empty(T, **f32), loss_tok=torch.empty(T, **f32),
        flags=torch.empty(T, dtype=torch.uint8, device=dev) if want_flags else None,
        stats=torch.empty(_lib.N_STATS, dtype=torch.int32, device=dev),
        dhidden=torch.empty(T, d, **f32) if want_grads else None,
        dweight=torch.empty(V, d, **f32) if want_grads else None, workspace=None)
    p = _lib.DppoParams(float(band[0]), float(band[1]), float(clip_eps[0]), float(clip_eps[1]),
                        RD_MODES[rd_mode], SCALE_MODES[scale_mode], float(loss_scale),
                        REF_MODES[ref_mode], float(alpha))
    used = C.c_int64(-1)
    st = _lib.lib().fused_lm_head_loss_fwd_bwd_noalloc(
        hidden.data_ptr(), weight.data_ptr(), _lib.DTYPE_BF16, T, d, V, ids, mu, ref, adv, msk,
        tsc, C.byref(p), out.logp.data_ptr(), out.loss_tok.data_ptr(), out.loss.data_ptr(),
        out.flags.data_ptr() if out.flags is not None else None, out.stats.data_ptr(),
        out.dhidden.data_ptr() if out.dhidden is not None else None,
        out.dweight.data_ptr() if out.dweight is not None else None, C.byref(used), _stream(dev))
    _lib.check(st, "fused_lm_head_loss_fwd_bwd_noalloc")
    return out, used.value


def ewma_proxy_update(x_prox: torch.Tensor, x_new: torch.Tensor, beta: float, w: float = 0.0,
                      reset: bool = False, normalized: bool = True) -> float:
    """One PPO-EWMA step on a flat buffer (in place on x_prox). Returns the new normaliser
    w_t (normalized form) or w unchanged (fixed-decay form)."""
    if x_prox.dtype != x_new.dtype or x_prox.numel() != x_new.numel():
        raise ValueError("x_prox and x_new must have the same dtype and size")
    if not (x_prox.is_contiguous() and x_new.is_contiguous() and x_prox.is_cuda and x_new.is_cuda):
        raise ValueError("x_prox and x_new must be contiguous GPU tensors")
    code = _dtype_code(x_prox)
    wv = C.c_double(float(w))
    st = _lib.lib().ewma_proxy_update(x_prox.data_ptr(), x_new.data_ptr(), code, x_prox.numel(),
                                      float(beta), C.byref(wv), int(bool(reset)),
                                      int(bool(normalized)), _stream(x_prox.device))
    _lib.check(st, "ewma_proxy_update")
    return wv.value


def set_path_policy(policy: str):
    """'auto' (register-resident rows when they fit) or 'stream' (always two-pass); with
    '+atomics' appended the loss call counts its statistics with its counting kernel and
    atomics even where it would take them from the flags (a testing hook: same results)."""
    code = {"auto": 0, "stream": 1, "auto+atomics": 2, "stream+atomics": 3}[policy]
    _lib.check(_lib.lib().dppo_set_path_policy(code), "dppo_set_path_policy")


def effective_thresholds(band, clip, alpha: float, kind: str):
    """Bounds on the total ratio pi_theta / mu_old that an interpolated reference induces
    (Prop. 1, App. A): returns ((band_lo, band_hi), (clip_lo, clip_hi)) on the total ratio
    for the band `band` on r_d and the PPO interval `clip` = (1 - eps_lo, 1 + eps_hi) on r_s;
    the clip lower bound applies to A < 0, the upper one to A >= 0."""
    out = (C.c_double * 4)()
    _lib.check(_lib.lib().dppo_effective_thresholds(float(band[0]), float(band[1]),
                                                    float(clip[0]), float(clip[1]),
                                                    float(alpha), REF_MODES[kind], out),
               "dppo_effective_thresholds")
    return (out[0], out[1]), (out[2], out[3])


def row_kernel_name(dtype: torch.dtype, V: int, ld: int | None = None,
                    with_dlogits: bool = True) -> str:
    """Profiler name of the per-row kernel a call with these shapes launches."""
    code = {torch.float32: 0, torch.bfloat16: 1}[dtype]
    name = _lib.lib().dppo_row_kernel_name(code, V, V if ld is None else ld, int(with_dlogits))
    if name is None:
        raise ValueError(f"no row kernel for dtype={dtype}, V={V}, ld={ld}")
    return name.decode()


class KernelTimer:
    """HIP-event timing of the per-row kernel launches made while the timer is on."""

    def __enter__(self):
        _lib.check(_lib.lib().dppo_timer_enable(1), "dppo_timer_enable")
        return self

    def read(self):
        ms = C.c_double(0.0)
        n = C.c_int64(0)
        _lib.check(_lib.lib().dppo_timer_read(C.byref(ms), C.byref(n)), "dppo_timer_read")
        return ms.value, n.value

    def __exit__(self, *exc):
        _lib.lib().dppo_timer_enable(0)


# ------------------------------------------------------------------ host-side controller
def _host_stats(stats):
    """The five counters as a host int32 array (a device tensor is copied once)."""
    if isinstance(stats, torch.Tensor):
        stats = stats.tolist()
    vals = [int(v) for v in stats]
    if len(vals) < _lib.N_STATS:
        raise ValueError(f"stats must hold {_lib.N_STATS} counters")
    return (C.c_int32 * _lib.N_STATS)(*vals[:_lib.N_STATS])


def beta_from_window(w_stale: float) -> float:
    """Staleness-aware decay beta = W / (W + 2) (App. B), computed by the library."""
    out = C.c_double(0.0)
    _lib.check(_lib.lib().dppo_beta_from_window(float(w_stale), C.byref(out)),
               "dppo_beta_from_window")
    return out.value


def train_infer_mask_value(stats) -> float:
    """rho_t = n_active / n_valid (1 when no token is valid), computed by the library."""
    out = C.c_double(0.0)
    _lib.check(_lib.lib().dppo_train_infer_mask_value(_host_stats(stats), C.byref(out)),
               "dppo_train_infer_mask_value")
    return out.value


def ppo_clip_ratio(stats) -> float:
    """Fraction of valid tokens removed by PPO clipping, computed by the library."""
    out = C.c_double(0.0)
    _lib.check(_lib.lib().dppo_ppo_clip_ratio(_host_stats(stats), C.byref(out)),
               "dppo_ppo_clip_ratio")
    return out.value


class EwmaProxy:
    """PPO-EWMA reference with automatic reset (Sec. 5.2; App. B; App. E), host-driven.

    Holds the proxy buffer (parameters or per-token log-probs), the normaliser w and the
    low-rho streak. `step(x_new, stats)` passes the loss stage's counters (one small
    device-to-host copy) to the library's reset rule (dppo_reset_decision) and then to
    ewma_proxy_update, which applies the reset or the normalised recursion. Its state
    (buffer, w, streak) is what a checkpoint must save.
    """

    def __init__(self, x0: torch.Tensor, beta: float, tau: float = 0.9, patience: int = 1,
                 normalized: bool = True):
        if not 0.0 <= beta < 1.0:
            raise ValueError("beta must lie in [0, 1)")
        self.x = x0.clone()
        self.beta = float(beta)
        self.tau = float(tau)
        self.patience = int(patience)
        self.normalized = normalized
        self.w = 1.0          # x0 is theta^(0): one step of history
        self.streak = 0
        self.resets = 0
        self.last_rho = 1.0

    def decide_reset(self, stats) -> bool:
        streak = C.c_int32(self.streak)
        rho = C.c_double(1.0)
        fire = C.c_int32(0)
        _lib.check(_lib.lib().dppo_reset_decision(_host_stats(stats), self.tau, self.patience,
                                                  C.byref(streak), C.byref(rho), C.byref(fire)),
                   "dppo_reset_decision")
        self.streak = streak.value
        self.last_rho = rho.value
        return bool(fire.value)

    def step(self, x_new: torch.Tensor, stats=None) -> bool:
        reset = self.decide_reset(stats) if stats is not None else False
        self.w = ewma_proxy_update(self.x, x_new, self.beta, self.w, reset=reset,
                                   normalized=self.normalized)
        if reset:
            self.resets += 1
        return reset

    def state_dict(self):
        return dict(x=self.x, w=self.w, streak=self.streak, resets=self.resets,
                    beta=self.beta, tau=self.tau, patience=self.patience,
                    normalized=self.normalized)

    def load_state_dict(self, sd):
        self.x.copy_(sd["x"])
        for k in ("w", "streak", "resets", "beta", "tau", "patience", "normalized"):
            setattr(self, k, sd[k])


class EwmaProxyDevice:
    """PPO-EWMA reference with automatic reset, both on the device (Sec. 5.2; App. B;
    App. E): `step(x_new, stats)` takes the loss stage's stats tensor as it lies in device
    memory and enqueues the reset rule and the update on the stream, with no
    device-to-host copy and no synchronisation. The decisions and the buffer are those of
    EwmaProxy; `read_state()` copies the 40-byte state to the host (one synchronisation).
    """

    STATE_BYTES = C.sizeof(_lib.DppoEwmaState)

    def __init__(self, x0: torch.Tensor, beta: float, tau: float = 0.9, patience: int = 1,
                 normalized: bool = True, w0: float = 1.0):
        if not 0.0 <= beta < 1.0:
            raise ValueError("beta must lie in [0, 1)")
        if not x0.is_cuda:
            raise ValueError("the proxy buffer must be a GPU tensor")
        self.x = x0.clone()
        self.beta = float(beta)
        self.tau = float(tau)
        self.patience = int(patience)
        self.normalized = normalized
        # int64 storage keeps the 40-byte state 8-byte aligned
        self.state = torch.zeros(self.STATE_BYTES // 8, dtype=torch.int64, device=x0.device)
        self.write_state(w=w0)

    def write_state(self, w: float, streak: int = 0, resets: int = 0):
        st = _lib.DppoEwmaState(w=float(w), streak=int(streak), resets=int(resets))
        host = torch.frombuffer(bytearray(C.string_at(C.addressof(st), self.STATE_BYTES)),
                                dtype=torch.int64)
        self.state.copy_(host)

    def read_state(self) -> dict:
        raw = self.state.cpu().numpy().tobytes()
        st = _lib.DppoEwmaState.from_buffer_copy(raw)
        return {k: getattr(st, k) for k, _ in _lib.DppoEwmaState._fields_ if k != "reserved"}

    def step(self, x_new: torch.Tensor, stats: torch.Tensor = None):
        if x_new.dtype != self.x.dtype or x_new.numel() != self.x.numel():
            raise ValueError("x_new must match the proxy buffer's dtype and size")
        if not (x_new.is_contiguous() and x_new.is_cuda):
            raise ValueError("x_new must be a contiguous GPU tensor")
        sp = None
        if stats is not None:
            if not (stats.is_cuda and stats.dtype == torch.int32 and stats.numel() >= _lib.N_STATS
                    and stats.is_contiguous()):
                raise ValueError("stats must be the loss stage's int32 device tensor")
            sp = stats.data_ptr()
        st = _lib.lib().ewma_proxy_step(self.x.data_ptr(), x_new.data_ptr(), _dtype_code(self.x),
                                        self.x.numel(), self.beta, self.tau, self.patience,
                                        int(bool(self.normalized)), sp, self.state.data_ptr(),
                                        _stream(self.x.device))
        _lib.check(st, "ewma_proxy_step")

    def state_dict(self):
        return dict(x=self.x, state=self.state.clone(), beta=self.beta, tau=self.tau,
                    patience=self.patience, normalized=self.normalized)

    def load_state_dict(self, sd):
        self.x.copy_(sd["x"])
        self.state.copy_(sd["state"])
        for k in ("beta", "tau", "patience", "normalized"):
            setattr(self, k, sd[k])


class DecoupledPPOLoss(torch.autograd.Function):
    """Autograd wrapper: forward runs the fused kernel (loss and dlogits at once); backward
    returns grad_output * dlogits (one extra elementwise pass when grad_output != 1)."""

    @staticmethod
    def forward(ctx, logits, token_ids, logp_mu_old, logp_ref, advantages, loss_mask,
                token_scale, kwargs):
        res = decoupled_ppo_loss_fwd_bwd(logits, token_ids, logp_mu_old, logp_ref, advantages,
                                         loss_mask, token_scale, **(kwargs or {}))
        ctx.save_for_backward(res.dlogits)
        ctx.mark_non_differentiable(res.logp, res.stats)
        return res.loss[0], res.logp, res.stats

    @staticmethod
    def backward(ctx, g_loss, g_lp, g_stats):
        (d,) = ctx.saved_tensors
        return (d * g_loss.to(d.dtype), None, None, None, None, None, None, None)


class FusedLMHeadLoss(torch.autograd.Function):
    """Autograd wrapper of the fused LM head: forward runs fused_lm_head_loss_fwd_bwd (the
    loss and both gradients at once, logits never materialised); backward returns
    grad_output * dL/dhidden and grad_output * dL/dweight in the dtypes of hidden and weight
    (one extra elementwise pass each)."""

    @staticmethod
    def forward(ctx, hidden, weight, token_ids, logp_mu_old, logp_ref, advantages, loss_mask,
                token_scale, kwargs):
        res = fused_lm_head_loss_fwd_bwd(hidden.detach(), weight.detach(), token_ids,
                                         logp_mu_old, logp_ref, advantages, loss_mask,
                                         token_scale, want_grads=True, **(kwargs or {}))
        ctx.save_for_backward(res.dhidden, res.dweight)
        ctx.dtypes = (hidden.dtype, weight.dtype)
        ctx.mark_non_differentiable(res.logp, res.stats)
        return res.loss[0], res.logp, res.stats

    @staticmethod
    def backward(ctx, g_loss, g_lp, g_stats):
        dh, dw = ctx.saved_tensors
        th, tw = ctx.dtypes
        gh = (dh * g_loss).to(th) if ctx.needs_input_grad[0] else None
        gw = (dw * g_loss).to(tw) if ctx.needs_input_grad[1] else None
        return (gh, gw, None, None, None, None, None, None, None)

