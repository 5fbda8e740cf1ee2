"""Pins of the oracle's vocabulary-shard functions: the shard statistics against brute force,
the combine against numpy's logaddexp, and the whole sharded stage against the unsharded
oracle (the same objective, Eq. 1-4 and Sec. 3.1, whatever the column split)."""
import numpy as np
import pytest

import oracle


def _batch(n=48, V=200, seed=0):
    g = np.random.default_rng(seed)
    z = g.normal(0.0, 2.0, size=(n, V))
    z[3, 17] += 12.0                                    # a spiked row
    ids = g.integers(0, V, size=n)
    ids[5] = V + 3                                      # out-of-range id on a valid row
    ids[6] = -1
    mask = np.ones(n, np.uint8)
    mask[[1, 9, 20]] = 0
    lp_theta, _ = oracle.logprob_fwd(z, np.clip(ids, 0, V - 1))
    lp_ref = lp_theta + g.normal(0.0, 0.2, size=n)
    lp_mu = lp_ref + g.laplace(0.0, 0.3, size=n)
    adv = g.normal(size=n)
    ts = g.uniform(0.5, 1.5, size=n)
    return z, ids, mask, lp_mu, lp_ref, adv, ts


def test_shard_stats_brute_force():
    g = np.random.default_rng(1)
    z = g.normal(0.0, 1.5, size=(10, 30))
    ids = np.array([0, 5, 12, 29, 11, 40, -2, 13, 19, 20])
    mask = np.ones(10, np.uint8)
    mask[4] = 0
    lse, zy = oracle.vocab_shard_stats(z[:, 12:20], ids, 12, mask)
    for t in range(10):
        if t == 4:
            assert lse[t] == -np.inf and zy[t] == 0.0
            continue
        assert abs(lse[t] - np.log(np.sum(np.exp(z[t, 12:20])))) < 1e-12
        assert zy[t] == (z[t, ids[t]] if 12 <= ids[t] < 20 else 0.0)


def test_shard_stats_all_neg_inf_and_nan():
    z = np.zeros((3, 4))
    z[0] = -np.inf
    z[1, 2] = np.nan
    lse, _ = oracle.vocab_shard_stats(z, np.zeros(3, np.int64), 0)
    assert lse[0] == -np.inf and np.isnan(lse[1]) and abs(lse[2] - np.log(4.0)) < 1e-15


def test_combine_against_logaddexp():
    g = np.random.default_rng(2)
    a, b, c = g.normal(0, 5, size=(3, 100))
    got = oracle.vocab_shard_combine(np.stack([a, b, c]))
    np.testing.assert_allclose(got, np.logaddexp(np.logaddexp(a, b), c), rtol=1e-14, atol=1e-14)
    # one shard: identity; a -inf shard adds nothing; all -inf: NaN (as a row of -inf)
    np.testing.assert_array_equal(oracle.vocab_shard_combine(a[None]), a)
    np.testing.assert_allclose(oracle.vocab_shard_combine(np.stack([a, np.full(100, -np.inf)])),
                               a, rtol=1e-15)
    assert np.all(np.isnan(oracle.vocab_shard_combine(np.full((2, 5), -np.inf))))


@pytest.mark.parametrize("rd_mode", ["none", "mask", "weight", "mask_weight"])
@pytest.mark.parametrize("cuts", [(0, 200), (0, 1, 57, 130, 200), (0, 25, 50, 75, 100, 125, 150, 175, 200)])
def test_sharded_stage_equals_unsharded(rd_mode, cuts):
    z, ids, mask, lp_mu, lp_ref, adv, ts = _batch()
    n, V = z.shape
    params = oracle.Params(0.5, 2.0, 0.1, 0.3, rd_mode, "token_mean", 1.0)
    ref = oracle.decoupled_ppo_loss(z, ids, lp_mu, lp_ref, adv, mask, ts, params=params)
    shards = [(cuts[i], cuts[i + 1]) for i in range(len(cuts) - 1)]
    stats = [oracle.vocab_shard_stats(z[:, a:b], ids, a, mask) for a, b in shards]
    lse = oracle.vocab_shard_combine(np.stack([s[0] for s in stats]))
    zy = np.sum([s[1] for s in stats], axis=0)           # exactly one shard holds z[y]
    scale = oracle.batch_scale(mask, params)
    outs = [oracle.vocab_shard_loss(z[:, a:b], ids, a, V, lse, zy, lp_mu, lp_ref, adv, mask, ts,
                                    params, scale) for a, b in shards]
    ev = mask.astype(bool) & (ids >= 0) & (ids < V)
    np.testing.assert_allclose(lse[ev], ref["lse"][ev], rtol=1e-13)
    for o in outs:                                       # every shard: the same token outputs
        np.testing.assert_allclose(o["lp"], ref["lp"], rtol=1e-12, atol=1e-13)
        np.testing.assert_allclose(o["loss_tok"], ref["loss_tok"], rtol=1e-12, atol=1e-13)
        np.testing.assert_allclose(o["w"], ref["w"], rtol=1e-12, atol=1e-15)
        np.testing.assert_array_equal(o["flags"], ref["flags"])
        np.testing.assert_array_equal(oracle.stats_of(o["flags"], params), ref["stats"])
    d = np.concatenate([o["dlogits"] for o in outs], axis=1)
    np.testing.assert_allclose(d, ref["dlogits"], rtol=1e-11, atol=1e-16)
    # the gradient of every row still sums to zero across the shards
    assert np.all(np.abs(d.sum(axis=1)) <= 1e-12 * np.maximum(np.abs(ref["w"]), 1e-300) + 1e-16)
