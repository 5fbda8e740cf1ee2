"""Host-side checks of the seeded workload generators (shapes, recipe, determinism)."""
import numpy as np
import torch

from paper_2605_12070_amd import workloads as W


def test_tiny_shapes_and_determinism():
    a = W.make_workload("tiny")
    b = W.make_workload("tiny")
    assert a.logits.shape == (256, 1024) and a.logits.dtype == torch.float32
    assert torch.equal(a.logits, b.logits) and torch.equal(a.ids, b.ids)
    assert a.ids.min() >= 0 and a.ids.max() < 1024
    # one advantage per 32-token sequence
    adv = a.adv.view(8, 32)
    assert torch.all(adv == adv[:, :1])
    assert a.mask.sum().item() == 256


def test_small_vocab_recipe():
    wl = W.make_workload("small_vocab", T=1024, V=512)
    assert wl.logits.dtype == torch.bfloat16
    flips = (wl.e_mu.abs() > 0.5).sum().item()
    assert abs(flips - round(0.05 * 1024)) <= 2       # ~5% pushed off the band by +-1.0


def test_large_vocab_group_advantages():
    wl = W.make_workload("large_vocab", T=32 * 16, V=64, seq_len=16)
    a = wl.adv.view(32, 16)[:, 0].numpy()
    assert set(np.unique(a)) == {-1.0, 1.0}
    for g in range(4):
        assert a[g * 8:(g + 1) * 8].sum() == 0.0           # 4 successes, 4 failures


def test_long_agentic_mask_exactly_40_percent():
    wl = W.make_workload("long_agentic", T=2 * 8192, V=64)
    m = wl.mask.numpy()
    assert int((m == 0).sum()) == round(0.4 * 2 * 8192)
    # spans: far fewer transitions than tokens (contiguous observation/assistant spans)
    assert np.count_nonzero(np.diff(m.astype(int))) < 200
    assert wl.segments.min() >= 0 and wl.segments.max() <= 3
    lp_old, prev, lp_mu = W.version_logprobs(torch.zeros(wl.T), wl)
    assert lp_old.dtype == torch.float32 and prev.shape == (wl.T,)


def test_reference_logprobs_are_sums():
    wl = W.make_workload("tiny")
    anchor = torch.linspace(-5, -1, wl.T, dtype=torch.float64)
    lp_ref, lp_mu = W.reference_logprobs(anchor, wl)
    np.testing.assert_allclose(lp_ref.double().numpy(), (anchor + wl.e_ref).numpy(), rtol=1e-6)
    np.testing.assert_allclose(lp_mu.double().numpy(), (anchor + wl.e_ref + wl.e_mu).numpy(), rtol=1e-6)


def test_gumbel_max_follows_softmax():
    # a row with one dominant logit is sampled at that logit
    z = torch.full((64, 10), -20.0)
    z[:, 3] = 10.0
    g = torch.Generator().manual_seed(0)
    assert torch.all(W.gumbel_max_ids(z, g) == 3)
