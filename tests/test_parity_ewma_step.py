"""GPU parity of ewma_proxy_step (reset rule and PPO-EWMA update on the device, through the
C ABI) against the oracle's reset schedule and recursion, and bit-equality with
ewma_proxy_update driven by the same decisions."""
import numpy as np
import pytest
import torch

import oracle
import paper_2605_12070_amd as P
from paper_2605_12070_amd import workloads as W

from helpers import bits_of, oracle_params, tie_mask

pytestmark = pytest.mark.gpu
DEV = "cuda:0"

# rho_t sequence with isolated and consecutive collapses, and a step with no valid token
RHOS = [0.95, 0.70, 0.95, 0.70, 0.70, 0.70, 1.00, 0.50, 0.95, None, 0.80, 0.80]


def _say(*a):
    print("[case]", *a, flush=True)


def _stats_for(rho, n_valid=1000):
    """Counters [n_valid, n_band, n_ppo, n_active, n_bad] with n_active / n_valid = rho
    (rho None: no valid token)."""
    if rho is None:
        return [0, 0, 0, 0, 0]
    act = int(round(rho * n_valid))
    return [n_valid, act, act, act, 0]


def _rho_of(st):
    return 1.0 if st[0] == 0 else st[3] / st[0]


# buffers the one-workgroup step takes (controller and update in one launch; 4099 with a
# tail past its 16-byte vectors; 16384 its largest) and ones of several workgroups (the
# controller kernel, then the element kernel; 16385 the smallest)
@pytest.mark.parametrize("n", [1001, 4099, 16384, 16385, 140003])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("normalized", [True, False])
@pytest.mark.parametrize("patience", [1, 2])
def test_device_step_matches_oracle_and_host_path(dtype, normalized, patience, n):
    beta, tau = 0.75, 0.9
    _say("ewma step", dtype, normalized, patience, n)
    g = torch.Generator(device=DEV).manual_seed(11 + patience)
    x0 = torch.randn(n, generator=g, device=DEV).to(dtype)
    hist = [torch.randn(n, generator=g, device=DEV).to(dtype) for _ in RHOS]
    stats = [_stats_for(r) for r in RHOS]
    rhos = [_rho_of(s) for s in stats]
    fired_ref = oracle.reset_schedule(rhos, tau, patience)

    dev = P.EwmaProxyDevice(x0, beta, tau=tau, patience=patience, normalized=normalized, w0=1.0)
    host_x, host_w = x0.clone(), 1.0
    x_ref, w_ref = bits_of(x0), 1.0
    streak, resets = 0, 0
    tol = 2.0 ** -8 if dtype == torch.bfloat16 else 2e-6
    for t, (th, st) in enumerate(zip(hist, stats)):
        dev.step(th, torch.tensor(st, dtype=torch.int32, device=DEV))
        fire = fired_ref[t]
        host_w = P.ewma_proxy_update(host_x, th, beta, host_w, reset=fire, normalized=normalized)
        if fire:
            x_ref = bits_of(th)
            w_ref = oracle.ewma_reset() if normalized else w_ref
        elif normalized:
            x_ref, w_ref = oracle.ewma_normalized_step(x_ref, bits_of(th), beta, w_ref)
        else:
            x_ref = oracle.ewma_fixed_step(x_ref, bits_of(th), beta)
        streak = 0 if fire else (streak + 1 if rhos[t] < tau else 0)
        resets += int(fire)
        state = dev.read_state()
        got = bits_of(dev.x)
        # same decisions and arithmetic as the host-coefficient entry point: identical bits
        assert np.array_equal(dev.x.view(torch.int16 if dtype == torch.bfloat16 else torch.int32)
                              .cpu().numpy(),
                              host_x.view(torch.int16 if dtype == torch.bfloat16 else torch.int32)
                              .cpu().numpy()), f"step {t}: device and host paths differ"
        np.testing.assert_allclose(got, x_ref, rtol=tol * (t + 2), atol=tol * (t + 2))
        assert state["last_reset"] == int(fire), t
        assert state["streak"] == streak and state["resets"] == resets, (t, state)
        assert state["error"] == 0
        assert state["last_rho"] == np.float32(rhos[t])
        if normalized:
            assert abs(state["w"] - w_ref) < 1e-12 and state["w"] == host_w
        else:
            assert state["w"] == 1.0
    assert resets == sum(fired_ref) and resets >= 1


@pytest.mark.parametrize("n", [1000, 140003])
def test_device_step_bad_normaliser_leaves_everything_unchanged(n):
    _say("ewma step bad w", n)
    g = torch.Generator(device=DEV).manual_seed(5)
    x0 = torch.randn(n, generator=g, device=DEV)
    xn = torch.randn(n, generator=g, device=DEV)
    dev = P.EwmaProxyDevice(x0, 0.75, tau=0.9, patience=1)
    dev.write_state(w=float("nan"), streak=3, resets=2)
    before = bits_of(dev.x)
    dev.step(xn, torch.tensor(_stats_for(0.5), dtype=torch.int32, device=DEV))
    st = dev.read_state()
    assert st["error"] == 1 and np.isnan(st["w"]) and st["streak"] == 3 and st["resets"] == 2
    assert np.array_equal(bits_of(dev.x), before)
    # a valid normaliser clears the flag on the next step
    dev.write_state(w=-1.0)
    dev.step(xn, None)
    assert dev.read_state()["error"] == 1
    dev.write_state(w=1.0)
    dev.step(xn, None)
    st = dev.read_state()
    assert st["error"] == 0 and st["w"] == 1.75 and st["last_reset"] == 0 and st["last_rho"] == 1.0
    ref, _ = oracle.ewma_normalized_step(before, bits_of(xn), 0.75, 1.0)
    np.testing.assert_allclose(bits_of(dev.x), ref, rtol=2e-6, atol=2e-6)


@pytest.mark.parametrize("n", [1001, 4099])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_device_step_unaligned_and_empty(dtype, n):
    _say("ewma step unaligned", dtype, n)
    g = torch.Generator(device=DEV).manual_seed(9)
    xb = torch.randn(n + 1, generator=g, device=DEV).to(dtype)
    nb = torch.randn(n + 1, generator=g, device=DEV).to(dtype)
    dev = P.EwmaProxyDevice(xb[1:], 0.9, normalized=False)
    dev.x = xb[1:]                                 # operate on the misaligned slice itself
    x0 = bits_of(dev.x)
    dev.step(nb[1:], torch.tensor(_stats_for(0.95), dtype=torch.int32, device=DEV))
    tol = 2.0 ** -8 if dtype == torch.bfloat16 else 2e-6
    np.testing.assert_allclose(bits_of(dev.x), oracle.ewma_fixed_step(x0, bits_of(nb[1:]), 0.9),
                               rtol=tol, atol=tol)
    # n = 0 runs the controller only: the streak still counts
    e = P.EwmaProxyDevice(torch.zeros(0, device=DEV, dtype=dtype), 0.5, tau=0.9, patience=3)
    for _ in range(2):
        e.step(torch.zeros(0, device=DEV, dtype=dtype),
               torch.tensor(_stats_for(0.5), dtype=torch.int32, device=DEV))
    st = e.read_state()
    assert st["streak"] == 2 and st["resets"] == 0 and st["w"] == 1.0 + 0.5 * (1.0 + 0.5)


def test_collapse_of_the_loss_stage_triggers_the_reset():
    """End to end: the loss kernel's own counters drive both controllers. A healthy step,
    then two steps where lp_mu is shifted by +1 on 30 % of the tokens (r_d = e^-1 < 0.5,
    outside the band), then a healthy one. With patience 2 the reset fires on the second
    collapsed step, exactly where the oracle's counters put it."""
    T, V = 512, 4096
    _say("collapse -> reset", T, V)
    wl = W.make_workload("small_vocab", device=DEV, T=T, V=V)
    zb = bits_of(wl.logits)
    ids = wl.ids.cpu().numpy()
    anchor, _ = oracle.logprob_fwd(zb, ids)
    lp_ref, lp_mu = W.reference_logprobs(torch.from_numpy(anchor), wl)
    g = np.random.default_rng(4)
    shift = torch.zeros(T, device=DEV)
    shift[torch.from_numpy(g.choice(T, size=int(0.3 * T), replace=False)).to(DEV)] = 1.0
    plans = [0.0, 1.0, 1.0, 0.0]
    x0 = torch.zeros(T, device=DEV)
    dev_ctl = P.EwmaProxyDevice(x0, 0.75, tau=0.9, patience=2)
    host_ctl = P.EwmaProxy(x0, 0.75, tau=0.9, patience=2)
    params = oracle_params((0.5, 2.0), (0.2, 0.2), "mask_weight", "token_mean", 1.0)
    rhos, fired_dev, fired_host = [], [], []
    for k, amount in enumerate(plans):
        mu = (lp_mu + amount * shift).to(DEV)
        ref = lp_ref.to(DEV)
        out = P.decoupled_ppo_loss_fwd_bwd(wl.logits, wl.ids, mu, ref, wl.adv, wl.mask)
        o = oracle.decoupled_ppo_loss(zb, ids, mu.cpu().double().numpy(), ref.cpu().double().numpy(),
                                      wl.adv.cpu().double().numpy(), wl.mask.cpu().numpy(),
                                      params=params, want_dlogits=False)
        # counters agree exactly away from threshold ties (each tie may go either way)
        n_ties = int(tie_mask(o, params).sum())
        diff = np.abs(out.stats.cpu().numpy().astype(np.int64) - np.asarray(o["stats"], np.int64))
        assert diff[0] == 0 and diff[4] == 0 and np.all(diff <= n_ties), (k, diff, n_ties)
        rhos.append(oracle.train_infer_mask_value(out.stats.cpu().tolist()))
        x_new = torch.full((T,), float(k + 1), device=DEV)
        dev_ctl.step(x_new, out.stats)
        fired_dev.append(bool(dev_ctl.read_state()["last_reset"]))
        fired_host.append(host_ctl.step(x_new, out.stats))
    assert rhos[0] >= 0.9 and rhos[1] < 0.9 and rhos[2] < 0.9 and rhos[3] >= 0.9, rhos
    expect = oracle.reset_schedule(rhos, 0.9, 2)
    assert expect == [False, False, True, False]
    assert fired_dev == expect and fired_host == expect
    assert torch.equal(dev_ctl.x, host_ctl.x)
    assert dev_ctl.read_state()["w"] == host_ctl.w == 1.75


@pytest.mark.parametrize("device_side", [True, False])
def test_controller_checkpoint_resume(device_side):
    """Saving the controller's state mid-run and loading it into a fresh controller gives
    the same continuation, bit for bit (the state is the buffer plus a few scalars)."""
    n = 1000
    _say("checkpoint resume", device_side)
    g = torch.Generator(device=DEV).manual_seed(21)
    xs = [torch.randn(n, generator=g, device=DEV) for _ in range(7)]
    stats = [torch.tensor(_stats_for(r), dtype=torch.int32, device=DEV)
             for r in (0.95, 0.5, 0.95, 0.5, 0.5, 0.95, 0.5)]
    mk = (lambda: P.EwmaProxyDevice(xs[0], 0.8, tau=0.9, patience=2)) if device_side else \
         (lambda: P.EwmaProxy(xs[0], 0.8, tau=0.9, patience=2))
    a = mk()
    for t in range(3):
        a.step(xs[t], stats[t])
    saved = {k: (v.clone() if torch.is_tensor(v) else v) for k, v in a.state_dict().items()}
    for t in range(3, 7):
        a.step(xs[t], stats[t])
    b = mk()
    b.load_state_dict(saved)
    for t in range(3, 7):
        b.step(xs[t], stats[t])
    assert torch.equal(a.x, b.x)
    if device_side:
        assert a.read_state() == b.read_state()
    else:
        assert (a.w, a.streak, a.resets) == (b.w, b.streak, b.resets)
