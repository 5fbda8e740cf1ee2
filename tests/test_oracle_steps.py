"""Direct pins of the oracle's step functions (each is also exercised through
decoupled_ppo_loss): textbook values of the PPO clipped surrogate (Eq. 2, Eq. 3), the
special cases of the four ways r_d enters (Eq. 4, Sec. 3.1), the sampled-token log-prob
against brute force, the token-mean scale against a count, and the exactness of the
float64 conversion."""
import math

import numpy as np

import oracle


def test_clipped_surrogate_textbook_values():
    cs = oracle.clipped_surrogate
    r = np.array([1.5, 0.5, 0.5, 1.5, 1.1, 0.95, 2.0])
    a = np.array([1.0, 1.0, -1.0, -1.0, 1.0, -1.0, 0.0])
    got = cs(r, a, 0.2, 0.2)
    # A > 0: the gain is capped at 1 + eps, not floored; A < 0: the loss is floored at
    # 1 - eps (pessimistic min), not capped; inside the interval the ratio is unclipped
    np.testing.assert_array_equal(got, [1.2, 0.5, -0.8, -1.5, 1.1, -0.95, 0.0])
    # asymmetric interval [1 - 0.1, 1 + 0.3]
    np.testing.assert_allclose(cs(np.array([1.5, 0.5]), np.array([1.0, -1.0]), 0.1, 0.3),
                               [1.3, -0.9], rtol=0, atol=1e-15)
    assert np.isnan(cs(np.array([np.nan]), np.array([1.0]), 0.2, 0.2))[0]


def test_discrepancy_weight_modes():
    r_d = np.array([0.4, 1.0, 3.0])
    band = np.array([False, True, False])
    dw = oracle.discrepancy_weight
    np.testing.assert_array_equal(dw(r_d, band, "none"), [1.0, 1.0, 1.0])
    np.testing.assert_array_equal(dw(r_d, band, "mask"), [0.0, 1.0, 0.0])
    np.testing.assert_array_equal(dw(r_d, band, "weight"), [0.4, 1.0, 3.0])
    np.testing.assert_array_equal(dw(r_d, band, "mask_weight"), [0.0, 1.0, 0.0])


def test_token_logprob_brute_force():
    z = np.array([[0.0, 0.0, math.log(2.0)], [1.0, -2.0, 0.5]])
    lse = np.array([math.log(sum(math.exp(v) for v in row)) for row in z])
    lp = oracle.token_logprob(z, np.array([2, 5]), lse)
    assert abs(lp[0] - math.log(2.0 / 4.0)) < 1e-15
    assert np.isnan(lp[1])                                  # id outside [0, V)
    lp = oracle.token_logprob(z, np.array([0, 1]), lse)
    assert abs(lp[0] - math.log(1.0 / 4.0)) < 1e-15
    assert abs(lp[1] - (-2.0 - math.log(math.e + math.exp(-2.0) + math.exp(0.5)))) < 1e-15


def test_token_mean_scale_counts_valid_tokens():
    assert oracle.token_mean_scale(np.array([1, 0, 1, 1], np.uint8), 2.0) == 2.0 / 3.0
    assert oracle.token_mean_scale(np.zeros(5, np.uint8), 0.5) == 0.5     # max(1, 0)
    assert oracle.token_mean_scale(np.zeros(0, np.uint8), 1.0) == 1.0


def test_as_f64_is_exact():
    x = np.array([1.0000001, 3.4e38, 1e-45, -0.1], dtype=np.float32)
    y = oracle.as_f64(x)
    assert y.dtype == np.float64
    np.testing.assert_array_equal(y.astype(np.float32).view(np.uint32), x.view(np.uint32))
