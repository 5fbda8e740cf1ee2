"""Seeded synthetic workloads for the loss stage (random draws only).

This module draws the random inputs of the benchmark and test workloads and holds none of
the loss arithmetic: no log-sum-exp, no ratios, no clipping. Reference and inference-side
log-probs are synthesised by the caller as an *anchor* log-prob (the current policy's
sampled-token log-prob, computed by whoever consumes the workload) plus the noise drawn
here:

    lp_ref = anchor + e_ref        lp_mu = lp_ref + e_mu

The paper trains on an agentic corpus with Qwen3 backbones; neither is available, so these
draws stand in for them with the shapes of a Qwen3 vocabulary (V = 151936), GRPO-style
group-normalised advantages and partial-rollout loss masks.

Workloads (name: what it is):
  tiny          T=256 (8 x 32), V=1024, fp32 logits ~ N(0, 2^2); e_ref ~ N(0, 0.1^2),
                e_mu ~ N(0, 0.05^2); A ~ N(0, 1) per 32-token sequence.
  small_vocab   T=4096 (16 x 256), V=32000, bf16 logits ~ N(0, 3^2); 1% of rows get one
                logit +15; noise as tiny, plus +-1.0 on e_mu for 5% of tokens.
  large_vocab   T=16384 (32 x 512), V=151936, bf16 logits ~ N(0, 3^2); e_ref ~ N(0, 0.2^2)
                (staleness drift), e_mu ~ Laplace(0, 0.05) (train-inference discrepancy);
                A = +-1 per sequence, groups of 8 samples with 4 positive and 4 negative.
  lm_head       T=8192 (16 x 512), d=4096, V=151936: hidden ~ N(0, 1) and LM-head weight
                ~ N(0, 0.02^2), both bf16 (logit std about 1.28); noise and advantages as
                large_vocab. Built by make_lm_head_workload; the logits are formed (chunk by
                chunk, float32, on the device) only to sample the token ids.
  long_agentic  T=65536 (8 x 8192), V=151936, bf16 logits ~ N(0, 3^2); exactly 40% of
                positions are tool/observation tokens (mask 0) in alternating spans of mean
                length 200 (observation) / 300 (assistant); each sequence holds 1-4 policy
                version segments with staleness gap g in {0..3} and drift e_old ~
                N(0, (0.1 (g+1))^2); e_prev ~ N(0, 0.1^2) is the previous version's extra
                drift; e_mu ~ Laplace(0, 0.05); A ~ N(0, 1) per sequence.

Token ids are sampled from softmax(logits) with the Gumbel-max trick. Large arrays are
drawn with a torch generator on the target device; small structural choices (spans,
segments, spike positions, group permutations) with a numpy generator. Both are seeded.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np
import torch

WORKLOADS = {
    "tiny": dict(n_seq=8, seq_len=32, V=1024, dtype="f32", sigma=2.0, seed=0,
                 ref_std=0.1, mu_std=0.05, mu_laplace=0.0, flip_frac=0.0, spike_frac=0.0,
                 adv="normal", mask_frac=0.0),
    "small_vocab": dict(n_seq=16, seq_len=256, V=32000, dtype="bf16", sigma=3.0, seed=1,
                        ref_std=0.1, mu_std=0.05, mu_laplace=0.0, flip_frac=0.05,
                        spike_frac=0.01, adv="normal", mask_frac=0.0),
    "large_vocab": dict(n_seq=32, seq_len=512, V=151936, dtype="bf16", sigma=3.0, seed=2,
                        ref_std=0.2, mu_std=0.0, mu_laplace=0.05, flip_frac=0.0,
                        spike_frac=0.0, adv="group_pm1", mask_frac=0.0),
    "long_agentic": dict(n_seq=8, seq_len=8192, V=151936, dtype="bf16", sigma=3.0, seed=3,
                         ref_std=None, mu_std=0.0, mu_laplace=0.05, flip_frac=0.0,
                         spike_frac=0.0, adv="normal", mask_frac=0.4),
}

# Band and clip used by every workload unless a test overrides them: r_d band [0.5, 2.0]
# (c = 2 in Eq. 4) and a symmetric clip of 0.2.
DEFAULT_BAND = (0.5, 2.0)
DEFAULT_EPS = (0.2, 0.2)


@dataclass
class Workload:
    name: str
    T: int
    V: int
    seq_len: int
    logits: torch.Tensor            # [T, V] float32 or bfloat16
    ids: torch.Tensor               # [T] int64
    adv: torch.Tensor               # [T] float32
    mask: torch.Tensor              # [T] uint8
    e_ref: torch.Tensor             # [T] float64 noise: lp_ref = anchor + e_ref
    e_mu: torch.Tensor              # [T] float64 noise: lp_mu = lp_ref + e_mu
    e_prev: torch.Tensor | None = None   # long_agentic: previous version's extra drift
    segments: np.ndarray | None = None   # long_agentic: per-token staleness gap
    meta: dict = field(default_factory=dict)
    hidden: torch.Tensor | None = None   # lm_head: [T, d] bf16 (logits is None)
    weight: torch.Tensor | None = None   # lm_head: [V, d] bf16, the [out, in] layout


def _laplace(gen, n, b, device):
    """Laplace(0, b) as b * (E1 - E2) with E1, E2 ~ Exp(1) (a standard construction)."""
    u1 = torch.rand(n, generator=gen, device=device, dtype=torch.float64)
    u2 = torch.rand(n, generator=gen, device=device, dtype=torch.float64)
    e1 = -torch.log1p(-u1)
    e2 = -torch.log1p(-u2)
    return b * (e1 - e2)


def gumbel_max_ids(logits: torch.Tensor, gen: torch.Generator, chunk: int = 1024):
    """Sample y_t ~ softmax(logits[t]) as argmax_v (z[t, v] + G[t, v]), G ~ Gumbel(0, 1)."""
    T, V = logits.shape
    out = torch.empty(T, dtype=torch.int64, device=logits.device)
    tiny = torch.finfo(torch.float32).tiny
    for a in range(0, T, chunk):
        b = min(T, a + chunk)
        u = torch.rand((b - a, V), generator=gen, device=logits.device, dtype=torch.float32)
        g = -torch.log(-torch.log(u.clamp_min(tiny)))
        out[a:b] = torch.argmax(logits[a:b].float() + g, dim=1)
        del u, g
    return out


def _group_pm1_advantages(rng, n_seq, group=8):
    """+-1 per sequence: each group of 8 samples of a prompt has 4 successes, 4 failures.

    Group normalisation of binary rewards with a 4/4 split gives exactly +-1.
    """
    assert n_seq % group == 0
    vals = []
    for _ in range(n_seq // group):
        g = np.array([1.0] * (group // 2) + [-1.0] * (group // 2))
        vals.append(rng.permutation(g))
    return np.concatenate(vals)


def _span_mask(rng, seq_len, n_zero, mean_obs=200.0, mean_asst=300.0):
    """One sequence's loss mask: alternating observation (0) / assistant (1) spans.

    Span lengths are geometric with the given means; observation and assistant span
    lengths are then rescaled so that exactly n_zero positions are observation tokens.
    """
    spans = []
    total = 0
    kind = 0
    while total < seq_len:
        mean = mean_obs if kind == 0 else mean_asst
        L = int(rng.geometric(1.0 / mean))
        spans.append([kind, L])
        total += L
        kind ^= 1
    spans[-1][1] -= total - seq_len
    if spans[-1][1] <= 0:
        spans.pop()
    if all(k == 0 for k, _ in spans):                # keep at least one assistant span
        spans[0][1] -= 1
        spans.append([1, 1])
    for want, k in ((n_zero, 0), (seq_len - n_zero, 1)):
        have = sum(L for kk, L in spans if kk == k)
        idx = [i for i, (kk, _) in enumerate(spans) if kk == k]
        scaled = [max(1, int(round(spans[i][1] * want / max(have, 1)))) for i in idx]
        # put the rounding residue on the longest span of this kind
        j = int(np.argmax(scaled))
        scaled[j] += want - sum(scaled)
        assert scaled[j] >= 1, "span rescaling failed"
        for i, L in zip(idx, scaled):
            spans[i][1] = L
    m = np.concatenate([np.full(L, k, np.uint8) for k, L in spans])
    assert m.size == seq_len and int((m == 0).sum()) == n_zero
    return m


def _segments(rng, seq_len, max_segments=4):
    """Per-token staleness gap for one partial-rollout sequence.

    The sequence is cut into 1..4 contiguous segments, each generated by a different
    policy version; the earliest segment is the stalest (gap up to 3).
    """
    k = int(rng.integers(1, max_segments + 1))
    cuts = np.sort(rng.choice(np.arange(1, seq_len), size=k - 1, replace=False)) if k > 1 else []
    bounds = [0, *list(cuts), seq_len]
    gap = np.empty(seq_len, np.int64)
    for s in range(k):
        gap[bounds[s]:bounds[s + 1]] = k - 1 - s
    return gap


def version_ids(T: int, seq_len: int, seed: int) -> np.ndarray:
    """Per-token policy version of a partial-rollout batch: sequences of seq_len tokens, each
    cut into 1..4 segments as in _segments, version id = staleness gap (0 = newest)."""
    rng = np.random.default_rng(seed)
    n_seq = -(-T // seq_len) if T > 0 else 0
    gaps = [_segments(rng, min(seq_len, T - i * seq_len)) for i in range(n_seq)]
    return (np.concatenate(gaps) if gaps else np.zeros(0, np.int64)).astype(np.int32)


def make_workload(name: str, device="cpu", T: int | None = None, V: int | None = None,
                  seed: int | None = None, seq_len: int | None = None) -> Workload:
    """Draw one named workload. T, V, seed and seq_len may be overridden (parity sizes)."""
    cfg = dict(WORKLOADS[name])
    seq_len = cfg["seq_len"] if seq_len is None else seq_len
    T = T if T is not None else cfg["n_seq"] * seq_len
    V = V if V is not None else cfg["V"]
    seed = cfg["seed"] if seed is None else seed
    seq_len = min(seq_len, T) if T > 0 else seq_len
    n_seq = -(-T // seq_len) if T > 0 else 0
    device = torch.device(device)
    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    rng = np.random.default_rng(seed)

    # logits
    z = torch.randn((T, V), generator=gen, device=device, dtype=torch.float32)
    z.mul_(cfg["sigma"])
    if cfg["spike_frac"] > 0 and T > 0:
        n_sp = max(1, int(round(cfg["spike_frac"] * T)))
        rows = rng.choice(T, size=n_sp, replace=False)
        cols = rng.integers(0, V, size=n_sp)
        z[torch.as_tensor(rows, device=device), torch.as_tensor(cols, device=device)] += 15.0
    logits = z.to(torch.bfloat16) if cfg["dtype"] == "bf16" else z
    del z
    ids = gumbel_max_ids(logits, gen) if T > 0 else torch.zeros(0, dtype=torch.int64,
                                                                  device=device)

    # advantages, one per sequence, broadcast over its tokens
    if cfg["adv"] == "group_pm1" and n_seq % 8 == 0:
        a_seq = _group_pm1_advantages(rng, n_seq)
    else:
        a_seq = rng.standard_normal(n_seq)
    adv = np.repeat(a_seq, seq_len)[:T].astype(np.float32)

    # loss mask
    if cfg["mask_frac"] > 0 and T > 0:
        total_zero = int(round(cfg["mask_frac"] * T))
        per = [total_zero // n_seq + (1 if i < total_zero % n_seq else 0) for i in range(n_seq)]
        lens = [min(seq_len, T - i * seq_len) for i in range(n_seq)]
        mask = np.concatenate([_span_mask(rng, L, min(nz, L - 1)) for L, nz in zip(lens, per)])
    else:
        mask = np.ones(T, np.uint8)

    # log-prob noise
    segments = None
    e_prev = None
    if cfg["ref_std"] is None:                       # long_agentic: version segments
        gaps = [_segments(rng, min(seq_len, T - i * seq_len)) for i in range(n_seq)]
        segments = np.concatenate(gaps) if gaps else np.zeros(0, np.int64)
        std = torch.as_tensor(0.1 * (segments + 1), dtype=torch.float64, device=device)
        e_ref = -std * torch.randn(T, generator=gen, device=device, dtype=torch.float64)
        e_prev = 0.1 * torch.randn(T, generator=gen, device=device, dtype=torch.float64)
    else:
        e_ref = cfg["ref_std"] * torch.randn(T, generator=gen, device=device,
                                             dtype=torch.float64)
    e_mu = torch.zeros(T, dtype=torch.float64, device=device)
    if cfg["mu_std"] > 0:
        e_mu += cfg["mu_std"] * torch.randn(T, generator=gen, device=device, dtype=torch.float64)
    if cfg["mu_laplace"] > 0:
        e_mu += _laplace(gen, T, cfg["mu_laplace"], device)
    if cfg["flip_frac"] > 0 and T > 0:
        n_fl = int(round(cfg["flip_frac"] * T))
        rows = rng.choice(T, size=n_fl, replace=False)
        signs = rng.choice([-1.0, 1.0], size=n_fl)
        e_mu[torch.as_tensor(rows, device=device)] += torch.as_tensor(signs, device=device)

    return Workload(
        name=name, T=T, V=V, seq_len=seq_len, logits=logits, ids=ids,
        adv=torch.as_tensor(adv, device=device), mask=torch.as_tensor(mask, device=device),
        e_ref=e_ref, e_mu=e_mu, e_prev=e_prev, segments=segments,
        meta=dict(cfg, seed=seed, T=T, V=V))


def reference_logprobs(anchor: torch.Tensor, wl: Workload):
    """lp_ref = anchor + e_ref and lp_mu = lp_ref + e_mu, as float32 (pure sums)."""
    a = anchor.to(torch.float64).to(wl.e_ref.device)
    lp_ref = a + wl.e_ref
    lp_mu = lp_ref + wl.e_mu
    return lp_ref.to(torch.float32), lp_mu.to(torch.float32)


def version_logprobs(anchor: torch.Tensor, wl: Workload):
    """long_agentic: (lp_old, lp_old_prev, lp_mu) for a segment-wise stale reference.

    lp_old = anchor + e_ref (e_ref drawn per version segment), lp_old_prev = lp_old + e_prev,
    lp_mu = lp_old + e_mu. The EWMA proxy over (lp_old_prev, lp_old) is left to the caller.
    """
    a = anchor.to(torch.float64).to(wl.e_ref.device)
    lp_old = a + wl.e_ref
    prev = lp_old + (wl.e_prev if wl.e_prev is not None else 0.0)
    lp_mu = lp_old + wl.e_mu
    return lp_old.to(torch.float32), prev.to(torch.float32), lp_mu.to(torch.float32)


LM_HEAD = dict(n_seq=16, seq_len=512, d=4096, V=151936, seed=4, hidden_std=1.0, weight_std=0.02,
               ref_std=0.2, mu_laplace=0.05)


def make_lm_head_workload(device="cpu", T: int | None = None, d: int | None = None,
                          V: int | None = None, seed: int | None = None,
                          seq_len: int | None = None, mask_frac: float = 0.0,
                          weight_std: float | None = None) -> Workload:
    """Draw the LM-head workload (hidden states, head weight, ids, noise, advantages)."""
    cfg = dict(LM_HEAD)
    seq_len = cfg["seq_len"] if seq_len is None else seq_len
    T = cfg["n_seq"] * seq_len if T is None else T
    d = cfg["d"] if d is None else d
    V = cfg["V"] if V is None else V
    seed = cfg["seed"] if seed is None else seed
    wstd = cfg["weight_std"] if weight_std is None else weight_std
    seq_len = min(seq_len, T) if T > 0 else seq_len
    n_seq = -(-T // seq_len) if T > 0 else 0
    device = torch.device(device)
    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    rng = np.random.default_rng(seed)
    hidden = (cfg["hidden_std"] * torch.randn((T, d), generator=gen, device=device)).to(torch.bfloat16)
    weight = torch.empty((V, d), dtype=torch.bfloat16, device=device)
    for a in range(0, V, 8192):                    # draw in float32 slices, store bf16
        b = min(V, a + 8192)
        weight[a:b] = (wstd * torch.randn((b - a, d), generator=gen, device=device)).to(torch.bfloat16)
    ids = torch.empty(T, dtype=torch.int64, device=device)
    tiny = torch.finfo(torch.float32).tiny
    for a in range(0, T, 512):                     # Gumbel-max over softmax(hidden weight^T)
        b = min(T, a + 512)
        z = hidden[a:b].float() @ weight.float().T if V * d <= (1 << 26) else \
            torch.cat([hidden[a:b].float() @ weight[c:c + 16384].float().T
                       for c in range(0, V, 16384)], dim=1)
        u = torch.rand(z.shape, generator=gen, device=device, dtype=torch.float32)
        ids[a:b] = torch.argmax(z - torch.log(-torch.log(u.clamp_min(tiny))), dim=1)
        del z, u
    if n_seq % 8 == 0 and n_seq > 0:
        a_seq = _group_pm1_advantages(rng, n_seq)
    else:
        a_seq = rng.standard_normal(n_seq)
    adv = np.repeat(a_seq, seq_len)[:T].astype(np.float32)
    mask = (rng.random(T) >= mask_frac).astype(np.uint8)
    e_ref = cfg["ref_std"] * torch.randn(T, generator=gen, device=device, dtype=torch.float64)
    e_mu = _laplace(gen, T, cfg["mu_laplace"], device)
    return Workload(name="lm_head", T=T, V=V, seq_len=seq_len, logits=None, ids=ids,
                    adv=torch.as_tensor(adv, device=device), mask=torch.as_tensor(mask, device=device),
                    e_ref=e_ref, e_mu=e_mu, meta=dict(cfg, seed=seed, T=T, V=V, d=d),
                    hidden=hidden, weight=weight)
