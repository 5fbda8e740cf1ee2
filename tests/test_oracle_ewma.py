"""Pins of the oracle's PPO-EWMA proxy (Sec. 5.2, Eq. 5; App. B) and reset rule."""
import numpy as np
import pytest

import oracle


@pytest.mark.parametrize("beta", [0.0, 0.3, 0.5, 0.75, 0.9])
def test_recursion_equals_closed_form(beta):
    # App. B: the normalised recursion unrolls to the weighted average of Eq. 5.
    rng = np.random.default_rng(30)
    hist = [rng.normal(size=17) for _ in range(12)]
    x = np.full(17, np.nan)          # the first step must not read the old buffer
    w = 0.0
    for t, th in enumerate(hist):
        x, w = oracle.ewma_normalized_step(x, th, beta, w)
        np.testing.assert_allclose(x, oracle.ewma_closed_form(hist[:t + 1], beta),
                                   rtol=1e-12, atol=1e-13)
    # w_t is the sum of the weights, 1 + beta + ... + beta^t
    assert abs(w - sum(beta ** k for k in range(len(hist)))) < 1e-12


def test_stationary_limit_is_fixed_decay_form():
    # As t grows, 1/w_t -> 1 - beta and beta w_{t-1}/w_t -> beta: the fixed form of Table 1.
    beta = 0.75
    w = 0.0
    for _ in range(200):
        w_prev = w
        w = 1.0 + beta * w
    a = 1.0 / w
    b = beta * w_prev / w
    assert abs(a - (1 - beta)) < 1e-12 and abs(b - beta) < 1e-12
    x0 = np.array([1.0, -2.0])
    x1 = np.array([3.0, 5.0])
    np.testing.assert_allclose(oracle.ewma_fixed_step(x0, x1, beta), a * x1 + b * x0, rtol=1e-12)


def test_center_of_mass_matches_series():
    for beta in (0.2, 0.5, 0.75, 0.9):
        k = np.arange(20000, dtype=np.float64)
        series = np.sum(k * beta ** k) / np.sum(beta ** k)
        assert abs(oracle.ewma_center_of_mass(beta) - series) < 1e-9


def test_staleness_aware_decay():
    # beta = W / (W + 2) puts the centre of mass at W / 2 (App. B).
    assert oracle.beta_from_window(6) == 0.75
    assert oracle.beta_from_window(2) == 0.5
    for W in (1, 2, 3, 4, 6, 10):
        assert abs(oracle.ewma_center_of_mass(oracle.beta_from_window(W)) - W / 2) < 1e-12


def test_reset_restarts_history():
    rng = np.random.default_rng(31)
    hist = [rng.normal(size=5) for _ in range(6)]
    beta = 0.6
    x, w = hist[0], 1.0
    for th in hist[1:3]:
        x, w = oracle.ewma_normalized_step(x, th, beta, w)
    # reset at step 3: proxy <- theta^(3), w <- 1; later steps average from there on
    x, w = hist[3].copy(), oracle.ewma_reset()
    for th in hist[4:]:
        x, w = oracle.ewma_normalized_step(x, th, beta, w)
    np.testing.assert_allclose(x, oracle.ewma_closed_form(hist[3:], beta), rtol=1e-12)


def test_reset_schedule():
    rhos = [0.95, 0.85, 0.92, 0.80, 0.70, 0.60, 0.95, 0.89]
    assert oracle.reset_schedule(rhos, 0.9, 1) == [False, True, False, True, True, True, False, True]
    assert oracle.reset_schedule(rhos, 0.9, 2) == [False, False, False, False, True, False, False, False]
    assert oracle.reset_schedule(rhos, 0.8, 1) == [False, False, False, False, True, True, False, False]
