"""Pins of the oracle's decoupled MIS loss, weights and dlogits.

Independent references: a hand-derived worked example (closed-form rationals), torch
float64 autograd of the clipped surrogate of Eq. 2 (checks the MIS gradient form of
Sec. 3.1), central finite differences, the Eq. 1 identity against an independently
computed total ratio, the reductions to standard PPO-clip (Table 1, first row) and to the
policy gradient when pi_theta = pi_old, and inclusive ties (Eq. 3, Eq. 4).
"""
import json
import math
import os

import numpy as np
import pytest
import torch

import oracle
from oracle import Params

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "loss_worked_example.json")
MODES = ("none", "mask", "weight", "mask_weight")


def _worked_inputs():
    g = json.load(open(GOLDEN))
    z_row = [math.log(v) for v in g["logits_row"]["log_terms"]]
    toks = g["tokens"]
    T = len(toks)
    z = np.tile(np.array(z_row), (T, 1))
    ids = np.array([t["y"] for t in toks])
    lp_theta = np.array([math.log(g["lp_theta"][t["name"]][0]) for t in toks])
    lp_ref = np.array([lp_theta[i] - math.log(t["r_s"]) for i, t in enumerate(toks)])
    lp_mu = np.array([lp_ref[i] - math.log(t["r_d"]) for i, t in enumerate(toks)])
    adv = np.array([t["adv"] for t in toks])
    return g, z, ids, lp_theta, lp_ref, lp_mu, adv


@pytest.mark.parametrize("mode", MODES)
def test_worked_example(mode):
    g, z, ids, lp_theta, lp_ref, lp_mu, adv = _worked_inputs()
    p = Params(0.5, 2.0, 0.2, 0.2, mode, "const", 1.0)
    out = oracle.decoupled_ppo_loss(z, ids, lp_mu, lp_ref, adv, params=p)
    exp = g["modes"][mode]
    np.testing.assert_allclose(out["lp"], lp_theta, atol=1e-15)
    np.testing.assert_array_equal(out["band"].astype(int), g["band"])
    np.testing.assert_array_equal(out["ppo"].astype(int), g["ppo_active"])
    np.testing.assert_allclose(out["loss_tok"], exp["loss_tok"], atol=1e-12)
    np.testing.assert_allclose(out["w"], exp["w"], atol=1e-12)
    np.testing.assert_allclose(out["dlogits"], np.array(exp["dlogits"]), atol=1e-12)
    assert abs(out["loss"] - exp["loss"]) < 1e-12
    np.testing.assert_array_equal(out["stats"], exp["stats"])


def _random_batch(seed, T=96, V=48, zscale=3.0, ref_std=0.15, mu_std=0.3, away=True,
                  eps=(0.2, 0.2)):
    """Random inputs with every token at least 2e-3 (relative) away from each threshold."""
    rng = np.random.default_rng(seed)
    z = rng.normal(0.0, zscale, size=(T, V))
    ids = rng.integers(0, V, size=T)
    lp, _ = oracle.logprob_fwd(z, ids)
    lp_ref = lp + rng.normal(0.0, ref_std, size=T)
    lp_mu = lp_ref + rng.normal(0.0, mu_std, size=T)
    adv = rng.normal(0.0, 1.0, size=T)
    if away:
        p = Params(clip_eps_lo=eps[0], clip_eps_hi=eps[1])
        bounds_s = np.log([1 - p.clip_eps_lo, 1 + p.clip_eps_hi])
        bounds_d = np.log([p.band_lo, p.band_hi])
        ls = lp - lp_ref
        ld = lp_ref - lp_mu
        near = (np.min(np.abs(ls[:, None] - bounds_s[None]), 1) < 2e-3) | \
               (np.min(np.abs(ld[:, None] - bounds_d[None]), 1) < 2e-3)
        lp_ref[near] = lp[near]          # r_s = 1 exactly, r_d moves off the band edge too
        lp_mu[near] = lp_ref[near]
    return z, ids, lp_mu, lp_ref, adv


def test_total_ratio_identity():
    # r = r_d r_s with r computed independently from lp_theta - lp_mu (Eq. 1)
    z, ids, lp_mu, lp_ref, adv = _random_batch(20)
    lp, _ = oracle.logprob_fwd(z, ids)
    r_s, r_d, _ = oracle.ratios(lp, lp_ref, lp_mu)
    r_indep = np.array([math.exp(a - b) for a, b in zip(lp, lp_mu)])
    np.testing.assert_allclose(r_d * r_s, r_indep, rtol=1e-12)


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("scale_mode", ["const", "token_mean"])
@pytest.mark.parametrize("eps", [(0.2, 0.2), (0.1, 0.3)])
def test_mis_gradient_equals_autograd_of_clipped_surrogate(mode, scale_mode, eps):
    z, ids, lp_mu, lp_ref, adv = _random_batch(21, eps=eps)
    T, V = z.shape
    rng = np.random.default_rng(5)
    mask = (rng.random(T) > 0.2).astype(np.uint8)
    ts = rng.uniform(0.5, 2.0, size=T)
    p = Params(0.5, 2.0, eps[0], eps[1], mode, scale_mode, 0.7)
    out = oracle.decoupled_ppo_loss(z, ids, lp_mu, lp_ref, adv, mask, ts, params=p)

    # torch float64 autograd of L = sum_t m_t s_t * (-wd_t) * min(r_s A, clip(r_s) A)
    zt = torch.tensor(z, requires_grad=True)
    lp_t = torch.log_softmax(zt, 1)[torch.arange(T), torch.from_numpy(ids)]
    lpr = torch.from_numpy(lp_ref)
    lpm = torch.from_numpy(lp_mu)
    A = torch.from_numpy(adv)
    r_s = torch.exp(lp_t - lpr)
    r_d = torch.exp(lpr - lpm)
    band = ((r_d >= 0.5) & (r_d <= 2.0)).double()
    wd = {"none": torch.ones_like(r_d), "mask": band, "weight": r_d, "mask_weight": band * r_d}[mode]
    sur = torch.minimum(r_s * A, torch.clamp(r_s, 1 - eps[0], 1 + eps[1]) * A)
    m = torch.from_numpy(mask.astype(np.float64))
    n = max(1, int(mask.sum()))
    scale = 0.7 / n if scale_mode == "token_mean" else 0.7
    L = torch.sum(m * scale * torch.from_numpy(ts) * (-wd * sur))
    L.backward()
    assert abs(out["loss"] - L.item()) <= 1e-12 * max(1.0, abs(L.item()))
    np.testing.assert_allclose(out["dlogits"], zt.grad.numpy(), rtol=1e-10, atol=1e-14)


def test_dlogits_central_finite_differences():
    z, ids, lp_mu, lp_ref, adv = _random_batch(22, T=12, V=16)
    p = Params(0.5, 2.0, 0.2, 0.2, "mask_weight", "const", 1.0)

    def loss_of(zz):
        return oracle.decoupled_ppo_loss(zz, ids, lp_mu, lp_ref, adv, params=p,
                                         want_dlogits=False)["loss"]

    d = oracle.decoupled_ppo_loss(z, ids, lp_mu, lp_ref, adv, params=p)["dlogits"]
    h = 1e-6
    fd = np.zeros_like(z)
    for t in range(z.shape[0]):
        for v in range(z.shape[1]):
            zp = z.copy(); zp[t, v] += h
            zm = z.copy(); zm[t, v] -= h
            fd[t, v] = (loss_of(zp) - loss_of(zm)) / (2 * h)
    np.testing.assert_allclose(d, fd, rtol=1e-6, atol=1e-9)


def test_dlogits_rows_sum_to_zero():
    z, ids, lp_mu, lp_ref, adv = _random_batch(23, T=64, V=200)
    out = oracle.decoupled_ppo_loss(z, ids, lp_mu, lp_ref, adv,
                                    params=Params(scale_mode="const"))
    rs = out["dlogits"].sum(axis=1)
    assert np.all(np.abs(rs) <= 1e-12 * np.maximum(np.abs(out["w"]), 1e-300) + 1e-300)


def test_pi_theta_equals_pi_old_gives_policy_gradient():
    # lp_ref = lp_theta => r_s = 1: never clipped for eps > 0, loss = -sum m s wd A, and the
    # gradient is the policy gradient of -sum c_t log pi(y_t), c_t = m s wd A.
    rng = np.random.default_rng(24)
    T, V = 40, 30
    z = rng.normal(0, 2.0, size=(T, V))
    ids = rng.integers(0, V, size=T)
    lp, _ = oracle.logprob_fwd(z, ids)
    lp_mu = lp + rng.normal(0, 0.4, size=T)
    adv = rng.normal(size=T)
    p = Params(0.5, 2.0, 0.2, 0.2, "mask_weight", "token_mean", 1.0)
    out = oracle.decoupled_ppo_loss(z, ids, lp_mu, lp, adv, params=p)
    np.testing.assert_array_equal(out["r_s"], np.ones(T))
    assert out["ppo"].all()
    r_d = np.exp(lp - lp_mu)
    band = (r_d >= 0.5) & (r_d <= 2.0)
    c = band * r_d * adv / T
    assert abs(out["loss"] - (-np.sum(c))) < 1e-12
    zt = torch.tensor(z, requires_grad=True)
    pg = -torch.sum(torch.from_numpy(c) * torch.log_softmax(zt, 1)[torch.arange(T), torch.from_numpy(ids)])
    pg.backward()
    np.testing.assert_allclose(out["dlogits"], zt.grad.numpy(), rtol=1e-11, atol=1e-15)


def test_reduces_to_standard_ppo_clip():
    # Table 1, first row: r_d = 1 (lp_mu = lp_ref), band [0, inf): plain PPO-clip of Eq. 2.
    z, ids, _, lp_ref, adv = _random_batch(25)
    T = z.shape[0]
    p = Params(0.0, float("inf"), 0.2, 0.2, "mask_weight", "const", 1.0)
    out = oracle.decoupled_ppo_loss(z, ids, lp_ref, lp_ref, adv, params=p)
    zt = torch.tensor(z, requires_grad=True)
    lp_t = torch.log_softmax(zt, 1)[torch.arange(T), torch.from_numpy(ids)]
    r = torch.exp(lp_t - torch.from_numpy(lp_ref))
    A = torch.from_numpy(adv)
    L = -torch.sum(torch.minimum(r * A, torch.clamp(r, 0.8, 1.2) * A))
    L.backward()
    assert abs(out["loss"] - L.item()) < 1e-11
    np.testing.assert_allclose(out["dlogits"], zt.grad.numpy(), rtol=1e-10, atol=1e-14)
    assert out["band"].all()


def test_inclusive_ties():
    # Eq. 3 and Eq. 4 use <=: r = 1 exactly on a zero-width clip and a [1, 1] band is kept.
    z = np.zeros((2, 4))
    ids = np.array([1, 2])
    lp, _ = oracle.logprob_fwd(z, ids)
    adv = np.array([1.0, -1.0])
    p = Params(1.0, 1.0, 0.0, 0.0, "mask_weight", "const", 1.0)
    out = oracle.decoupled_ppo_loss(z, ids, lp, lp, adv, params=p)
    assert out["band"].all() and out["ppo"].all()
    np.testing.assert_allclose(out["w"], adv)


def test_masked_rows_and_bad_ids():
    rng = np.random.default_rng(26)
    T, V = 10, 12
    z = rng.normal(size=(T, V))
    z[3] = np.nan                              # masked: never read, so no NaN escapes
    ids = rng.integers(0, V, size=T)
    ids[5] = V                                  # bad id on a valid row
    ids[6] = -3                                 # bad id on a masked row
    mask = np.ones(T, np.uint8)
    mask[[3, 6]] = 0
    lp_ref = np.zeros(T) - 2.0
    out = oracle.decoupled_ppo_loss(z, ids, lp_ref, lp_ref, np.ones(T), mask,
                                    params=Params(scale_mode="token_mean"))
    assert out["lp"][3] == 0 and out["loss_tok"][3] == 0 and out["flags"][3] == 0
    assert np.all(out["dlogits"][3] == 0) and np.all(out["dlogits"][6] == 0)
    assert np.isnan(out["lp"][5]) and out["loss_tok"][5] == 0 and out["w"][5] == 0
    assert out["flags"][5] == oracle.FLAG_VALID | oracle.FLAG_BAD_ID
    assert np.all(out["dlogits"][5] == 0)
    st = out["stats"]
    assert st[oracle.STAT_N_VALID] == 8 and st[oracle.STAT_N_BAD] == 1
    assert st[oracle.STAT_N_BAND] <= 7 and np.isfinite(out["loss"])
    assert abs(out["scale"] - 1.0 / 8) < 1e-15


def test_nonfinite_logits_propagate_nan():
    z = np.zeros((3, 6))
    z[1, 2] = np.inf
    ids = np.array([0, 0, 0])
    lp_ref = np.full(3, -math.log(6))
    out = oracle.decoupled_ppo_loss(z, ids, lp_ref, lp_ref, np.ones(3),
                                    params=Params(scale_mode="const"))
    assert np.isnan(out["lp"][1]) and np.isnan(out["loss_tok"][1]) and np.isnan(out["loss"])
    # r_d = pi_ref / mu_old does not involve the logits, so the band decision stands;
    # the PPO decision on r_s = NaN is false.
    assert out["flags"][1] == oracle.FLAG_VALID | oracle.FLAG_BAND and out["w"][1] == 0
    assert np.isnan(out["dlogits"][1]).all() and np.isfinite(out["dlogits"][[0, 2]]).all()


def test_token_mean_and_const_scale_relation():
    z, ids, lp_mu, lp_ref, adv = _random_batch(27)
    T = z.shape[0]
    mask = (np.arange(T) % 3 != 0).astype(np.uint8)
    a = oracle.decoupled_ppo_loss(z, ids, lp_mu, lp_ref, adv, mask,
                                  params=Params(scale_mode="token_mean", loss_scale=2.0))
    b = oracle.decoupled_ppo_loss(z, ids, lp_mu, lp_ref, adv, mask,
                                  params=Params(scale_mode="const", loss_scale=1.0))
    n = int(mask.sum())
    assert abs(a["loss"] - 2.0 * b["loss"] / n) < 1e-13
    np.testing.assert_allclose(a["dlogits"], 2.0 * b["dlogits"] / n, rtol=1e-12, atol=1e-300)


def test_stats_and_rho():
    z, ids, lp_mu, lp_ref, adv = _random_batch(28, T=200)
    out = oracle.decoupled_ppo_loss(z, ids, lp_mu, lp_ref, adv, params=Params())
    st = out["stats"]
    assert st[0] == 200
    assert st[1] == int(out["band"].sum()) and st[2] == int(out["ppo"].sum())
    assert st[3] == int((out["band"] & out["ppo"]).sum())
    rho = oracle.train_infer_mask_value(st)
    assert 0.0 <= rho <= 1.0 and abs(rho - st[3] / 200) < 1e-15
    assert abs(oracle.ppo_clip_ratio(st) - (1 - st[2] / 200)) < 1e-15


def test_empty_batch():
    z = np.zeros((0, 16))
    out = oracle.decoupled_ppo_loss(z, np.zeros(0, np.int64), np.zeros(0), np.zeros(0),
                                    np.zeros(0), params=Params())
    assert out["loss"] == 0.0 and list(out["stats"]) == [0, 0, 0, 0, 0]
    assert out["dlogits"].shape == (0, 16)
