"""Pins of the interpolation-proxy threshold map (Prop. 1; App. A; Table 4)."""
import csv
import os

import numpy as np
import pytest

import oracle
from oracle import Params

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "table4_effective_thresholds.csv")


def _rows():
    with open(GOLDEN) as f:
        lines = [l for l in f if not l.startswith("#")]
    return list(csv.DictReader(lines))


@pytest.mark.parametrize("row", _rows(), ids=lambda r: f"{r['mask_lo']}-{r['clip_hi']}-n{r['n']}-{r['kind']}")
def test_table4_row(row):
    alpha = 1.0 / (int(row["n"]) + 1)
    m, c = oracle.effective_thresholds(float(row["mask_lo"]), float(row["mask_hi"]),
                                       float(row["clip_lo"]), float(row["clip_hi"]),
                                       alpha, row["kind"])
    got = [m[0], m[1], c[0], c[1]]
    want = [float(row[k]) for k in ("eff_mask_lo", "eff_mask_hi", "eff_clip_lo", "eff_clip_hi")]
    for g, w in zip(got, want):
        assert abs(g - w) <= 0.5e-4 + 1e-12, (g, w)


@pytest.mark.parametrize("kind", ["linear", "log_linear"])
@pytest.mark.parametrize("n", [1, 2, 3])
def test_prop1_active_sets_coincide(kind, n):
    # Prop. 1 by brute force: masking r_d and clipping r_s of an interpolated proxy keeps
    # exactly the tokens whose total ratio lies inside the re-parameterised bounds.
    alpha = 1.0 / (n + 1)
    rng = np.random.default_rng(40 + n)
    N = 20000
    lp_theta = rng.uniform(-8, -0.01, size=N)
    lp_mu = lp_theta - rng.normal(0, 0.02, size=N)
    adv = rng.choice([-1.0, 1.0], size=N)
    proxy = (oracle.log_linear_proxy_logprob if kind == "log_linear"
             else oracle.linear_proxy_logprob)(lp_mu, lp_theta, alpha)
    band = (0.99, 1.01)
    clip = (0.997, 1.004)
    r_s, r_d, r = oracle.ratios(lp_theta, proxy, lp_mu)
    keep = oracle.band_mask(r_d, *band) & oracle.ppo_active_mask(r_s, adv, 1 - clip[0], clip[1] - 1)
    m, c = oracle.effective_thresholds(band[0], band[1], clip[0], clip[1], alpha, kind)
    keep2 = (r >= m[0]) & (r <= m[1]) & np.where(adv >= 0, r <= c[1], r >= c[0])
    # allow disagreement only within rounding distance of a bound
    edge = np.min(np.abs(np.log(r)[:, None] - np.log(np.array([*m, *c]))[None]), axis=1) < 1e-9
    assert np.array_equal(keep[~edge], keep2[~edge])
    assert keep.sum() > 100 and (~keep).sum() > 100
