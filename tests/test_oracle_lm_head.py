"""Pins of the oracle's loss stage with the LM head folded in (chain rule through
z = hidden weight^T)."""
import numpy as np
import pytest
import torch

import oracle
from oracle import Params


def _case(T=24, d=16, V=40, seed=0, scale_w=0.3):
    rng = np.random.default_rng(seed)
    h = rng.standard_normal((T, d))
    w = rng.standard_normal((V, d)) * scale_w
    z = h @ w.T
    zs = z - z.max(1, keepdims=True)
    p = np.exp(zs) / np.exp(zs).sum(1, keepdims=True)
    ids = np.array([rng.choice(V, p=p[t]) for t in range(T)])
    lp = np.log(p[np.arange(T), ids])
    lp_ref = lp + rng.normal(0, 0.1, T)
    lp_mu = lp_ref + rng.normal(0, 0.05, T)
    adv = np.repeat(rng.standard_normal(T // 8), 8)
    mask = (rng.random(T) > 0.2).astype(np.uint8)
    return h, w, ids, lp_mu, lp_ref, adv, mask


@pytest.mark.parametrize("rd_mode", ["none", "mask", "weight", "mask_weight"])
def test_grads_equal_autograd_of_the_surrogate(rd_mode):
    """dhidden and dweight equal float64 autograd of L = sum_t m_t s_t l_t through
    log_softmax(hidden weight^T), the ratios, the band and the clipped surrogate (Eq. 2-4)
    with the reference and the band held constant (a separate implementation of the same
    objective, in torch)."""
    h, w, ids, lp_mu, lp_ref, adv, mask = _case(seed=3)
    params = Params(0.5, 2.0, 0.15, 0.25, rd_mode, "token_mean", 1.0)
    ref = oracle.lm_head_loss(h, w, ids, lp_mu, lp_ref, adv, mask, None, params)
    H = torch.tensor(h, requires_grad=True)
    W = torch.tensor(w, requires_grad=True)
    lp = torch.log_softmax(H @ W.T, dim=1)[torch.arange(len(ids)), torch.tensor(ids)]
    r_s = torch.exp(lp - torch.tensor(lp_ref))
    r_d = np.exp(lp_ref - lp_mu)
    band = (r_d >= 0.5) & (r_d <= 2.0)
    wd = {"none": np.ones_like(r_d), "mask": band * 1.0, "weight": r_d,
          "mask_weight": band * r_d}[rd_mode]
    A = torch.tensor(adv)
    sur = torch.minimum(r_s * A, torch.clamp(r_s, 1 - 0.15, 1 + 0.25) * A)
    s = 1.0 / max(1, int(mask.sum()))
    L = -(torch.tensor(mask * wd * s) * sur).sum()
    L.backward()
    # away from clip ties the surrogate is differentiable
    rs = ref["r_s"]
    far = np.minimum(np.abs(np.log(rs) - np.log(0.85)), np.abs(np.log(rs) - np.log(1.25))) > 1e-6
    assert far.all()
    np.testing.assert_allclose(ref["loss"], L.item(), rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(ref["dhidden"], H.grad.numpy(), rtol=1e-9, atol=1e-13)
    np.testing.assert_allclose(ref["dweight"], W.grad.numpy(), rtol=1e-9, atol=1e-13)


def test_finite_differences():
    """Central differences of the loss in a few entries of hidden and weight."""
    h, w, ids, lp_mu, lp_ref, adv, mask = _case(T=16, d=8, V=24, seed=5)
    params = Params(0.5, 2.0, 0.2, 0.2, "mask_weight", "const", 1.0)
    ref = oracle.lm_head_loss(h, w, ids, lp_mu, lp_ref, adv, mask, None, params)
    eps = 1e-6

    def loss(hh, ww):
        return oracle.lm_head_loss(hh, ww, ids, lp_mu, lp_ref, adv, mask, None, params,
                                   want_grads=False)["loss"]

    rng = np.random.default_rng(0)
    for _ in range(12):
        t, k = rng.integers(16), rng.integers(8)
        hp, hm = h.copy(), h.copy()
        hp[t, k] += eps
        hm[t, k] -= eps
        fd = (loss(hp, w) - loss(hm, w)) / (2 * eps)
        assert abs(fd - ref["dhidden"][t, k]) <= 1e-6 * max(1.0, abs(fd))
        v, k = rng.integers(24), rng.integers(8)
        wp, wm = w.copy(), w.copy()
        wp[v, k] += eps
        wm[v, k] -= eps
        fd = (loss(h, wp) - loss(h, wm)) / (2 * eps)
        assert abs(fd - ref["dweight"][v, k]) <= 1e-6 * max(1.0, abs(fd))


def test_identity_head_reduces_to_the_row_oracle():
    """With V = d and weight = I the logits are the hidden states: the loss and dlogits are
    the row oracle's, dhidden = dlogits and dweight = dlogits^T hidden."""
    h, _, ids, lp_mu, lp_ref, adv, mask = _case(T=16, d=12, V=12, seed=7)
    w = np.eye(12)
    params = Params()
    ref = oracle.lm_head_loss(h, w, ids, lp_mu, lp_ref, adv, mask, None, params)
    row = oracle.decoupled_ppo_loss(h, ids, lp_mu, lp_ref, adv, mask, None, params)
    assert ref["loss"] == row["loss"]
    np.testing.assert_array_equal(ref["dhidden"], row["dlogits"])
    np.testing.assert_allclose(ref["dweight"], row["dlogits"].T @ h, rtol=0, atol=0)
