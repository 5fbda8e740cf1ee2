"""Pins of the oracle's sampled-token log-prob (the quantity whose ratios Sec. 3.2 takes).

Each pin comes from outside the oracle: an unshifted naive formula, an exactly rounded
pure-Python sum, torch's float64 log_softmax, bfloat16 decoding by torch, closed forms.
"""
import math

import numpy as np
import pytest
import torch

import oracle


def _rand_logits(rng, T, V, scale=5.0):
    return rng.uniform(-scale, scale, size=(T, V))


def test_lse_equals_unshifted_naive_sum():
    # |z| < 30 keeps exp(z) finite, so the unshifted log(sum(exp(z))) is a valid reference
    # for the max-shifted evaluation.
    rng = np.random.default_rng(10)
    z = _rand_logits(rng, 64, 48, scale=29.0)
    naive = np.log(np.exp(z).sum(axis=1))
    np.testing.assert_allclose(oracle.row_logsumexp(z), naive, rtol=1e-13, atol=1e-12)


def test_lse_equals_exactly_rounded_python_sum():
    rng = np.random.default_rng(11)
    z = _rand_logits(rng, 8, 37, scale=12.0)
    for t in range(z.shape[0]):
        ref = math.log(math.fsum(math.exp(v) for v in z[t]))
        assert abs(oracle.row_logsumexp(z[t:t + 1])[0] - ref) <= 1e-13 * max(1.0, abs(ref))


def test_logprob_matches_torch_log_softmax_f64():
    rng = np.random.default_rng(12)
    T, V = 33, 61
    z = _rand_logits(rng, T, V, scale=20.0)
    ids = rng.integers(0, V, size=T)
    lp, lse = oracle.logprob_fwd(z, ids)
    ref = torch.log_softmax(torch.from_numpy(z), dim=1)[torch.arange(T), torch.from_numpy(ids)]
    np.testing.assert_allclose(lp, ref.numpy(), rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(lse, torch.logsumexp(torch.from_numpy(z), 1).numpy(), rtol=1e-14)


def test_softmax_sums_to_one_over_vocab():
    rng = np.random.default_rng(13)
    T, V = 16, 40
    z = _rand_logits(rng, T, V, scale=8.0)
    lse = oracle.row_logsumexp(z)
    for v in range(V):
        lp_v, _ = oracle.logprob_fwd(z, np.full(T, v))
        if v == 0:
            acc = np.exp(lp_v)
        else:
            acc = acc + np.exp(lp_v)
    np.testing.assert_allclose(acc, 1.0, rtol=1e-13)
    assert np.all(np.isfinite(lse))


def test_closed_form_two_way_row():
    # z = [ln 3, 0] -> softmax [3/4, 1/4]
    z = np.array([[math.log(3.0), 0.0], [math.log(3.0), 0.0]])
    lp, lse = oracle.logprob_fwd(z, np.array([0, 1]))
    assert abs(lp[0] - math.log(0.75)) < 1e-15
    assert abs(lp[1] - math.log(0.25)) < 1e-15
    assert abs(lse[0] - math.log(4.0)) < 1e-15


def test_uniform_row_and_shift_invariance():
    V = 151936
    z = np.zeros((1, V))
    lp, lse = oracle.logprob_fwd(z, np.array([7]))
    assert abs(lp[0] + math.log(V)) < 1e-12
    # log pi is invariant to adding a constant to the row
    z2 = z + 1234.5
    lp2, lse2 = oracle.logprob_fwd(z2, np.array([7]))
    assert abs(lp2[0] - lp[0]) < 1e-10 and abs(lse2[0] - lse[0] - 1234.5) < 1e-10


def test_bf16_decoding_matches_torch():
    rng = np.random.default_rng(14)
    bits = rng.integers(0, 1 << 16, size=4096, dtype=np.uint16)
    bits = bits[((bits >> 7) & 0xFF) != 0xFF]        # finite patterns only
    ours = oracle.bf16_bits_to_f64(bits)
    ref = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(ours, ref)
    fixed = oracle.bf16_bits_to_f64(np.array([0x3F80, 0xC000, 0x7F80, 0x0001], np.uint16))
    assert fixed[0] == 1.0 and fixed[1] == -2.0 and fixed[2] == np.inf
    assert fixed[3] == 2.0 ** -133


@pytest.mark.parametrize("bad", ["nan", "posinf", "allneginf"])
def test_non_finite_rows_give_nan(bad):
    z = np.zeros((3, 8))
    if bad == "nan":
        z[1, 3] = np.nan
    elif bad == "posinf":
        z[1, 5] = np.inf
    else:
        z[1, :] = -np.inf
    lp, lse = oracle.logprob_fwd(z, np.array([0, 0, 0]))
    assert np.isnan(lse[1]) and np.isnan(lp[1])
    assert np.isfinite(lse[[0, 2]]).all()


def test_neg_inf_entries_are_zero_probability():
    z = np.array([[0.0, -np.inf, 0.0, -np.inf]])
    lp, lse = oracle.logprob_fwd(z, np.array([0]))
    assert abs(lse[0] - math.log(2.0)) < 1e-15 and abs(lp[0] + math.log(2.0)) < 1e-15
    lp1, _ = oracle.logprob_fwd(z, np.array([1]))
    assert lp1[0] == -np.inf


def test_out_of_range_ids_give_nan():
    z = np.zeros((3, 4))
    lp, _ = oracle.logprob_fwd(z, np.array([-1, 4, 3]))
    assert np.isnan(lp[0]) and np.isnan(lp[1]) and abs(lp[2] + math.log(4)) < 1e-15


def test_versioned_logprob_special_cases():
    """One version for every token reduces to the plain log-prob of that version's logits;
    identical versions reduce to the plain log-prob; unknown versions give NaN."""
    rng = np.random.default_rng(11)
    T, V = 40, 37
    zs = [rng.normal(0, 2, (T, V)) for _ in range(3)]
    ids = rng.integers(0, V, T)
    for v in range(3):
        lp, _ = oracle.logprob_fwd(zs[v], ids)
        np.testing.assert_array_equal(oracle.versioned_logprob(zs, np.full(T, v), ids), lp)
    lp0, _ = oracle.logprob_fwd(zs[0], ids)
    mixed = rng.integers(0, 3, T)
    np.testing.assert_array_equal(oracle.versioned_logprob([zs[0]] * 3, mixed, ids), lp0)
    bad = mixed.copy()
    bad[:5] = [-1, 3, 7, -2, 100]
    got = oracle.versioned_logprob(zs, bad, ids)
    assert np.isnan(got[:5]).all() and np.isfinite(got[5:]).all()
    # each token takes its own version's row, brute force on a tiny case
    for t in range(T):
        z = zs[mixed[t]][t]
        ref = z[ids[t]] - np.log(np.sum(np.exp(z)))
        assert abs(oracle.versioned_logprob(zs, mixed, ids)[t] - ref) < 1e-12
