"""GPU parity of fused_lm_head_loss_fwd_bwd (through the C ABI) against the float64 oracle.

The oracle forms z = hidden weight^T exactly from the same bf16 bits, runs the loss stage and
applies the chain rule. Tolerances:
  * lp, l_t: as the row entry point (bf16 contract 2e-3 relative, floor 1), plus a tight
    1e-4 bound (fp32 accumulation of d bf16 products);
  * decisions and stats: exact away from threshold ties;
  * dhidden, dweight: |gpu - ref| <= 2^-7 (|G| |W|) and 2^-7 (|G|^T |H|) elementwise, where G
    is the oracle's dlogits: G is rounded to bf16 (2^-9) after an fp32 exponential, and the
    products accumulate in fp32.
Every case prints its name and sizes before it touches the GPU.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2605_12070_amd as P
from paper_2605_12070_amd import workloads as W

from helpers import DELTA, assert_close_rel, bits_of, oracle_params, tie_mask

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _say(*a):
    print("[case]", *a, flush=True)


def _anchor(wl):
    """Oracle log-probs of the sampled tokens (only to synthesise lp_ref and lp_mu)."""
    z = bits_of(wl.hidden) @ bits_of(wl.weight).T
    lp, _ = oracle.logprob_fwd(z, wl.ids.cpu().numpy())
    return torch.from_numpy(lp)


def _grad_bound(G, other):
    return 2.0 ** -7 * (np.abs(G) @ np.abs(other)) + 1e-7


def _run(T, d, V, seed=0, mask_frac=0.2, rd_mode="mask_weight", scale_mode="token_mean",
         loss_scale=1.0, band=(0.5, 2.0), eps=(0.2, 0.2), ref_mode="given", alpha=0.5,
         vocab_chunk=0, weight_std=0.1, bad_ids=(), want_grads=True):
    _say("lm_head", T, d, V, seed, mask_frac, rd_mode, scale_mode, ref_mode, vocab_chunk)
    wl = W.make_lm_head_workload(DEV, T=T, d=d, V=V, seed=seed, seq_len=8,
                                 mask_frac=mask_frac, weight_std=weight_std)
    for t in bad_ids:
        wl.ids[t] = V + 3 if t % 2 else -1
    anchor = _anchor(wl)
    lp_ref, lp_mu = W.reference_logprobs(anchor, wl)
    if ref_mode == "given":
        ref_in = lp_ref
    else:
        f = oracle.log_linear_proxy_logprob if ref_mode == "log_linear" else oracle.linear_proxy_logprob
        ref_in = torch.from_numpy(f(lp_mu.cpu().double().numpy(), anchor.numpy(), alpha))
    res = P.fused_lm_head_loss_fwd_bwd(
        wl.hidden, wl.weight, wl.ids, lp_mu, lp_ref if ref_mode == "given" else None, wl.adv,
        wl.mask, band=band, clip_eps=eps, rd_mode=rd_mode, scale_mode=scale_mode,
        loss_scale=loss_scale, ref_mode=ref_mode, alpha=alpha, vocab_chunk=vocab_chunk,
        want_grads=want_grads)
    torch.cuda.synchronize()
    params = oracle_params(band, eps, rd_mode, scale_mode, loss_scale)
    H, Wt = bits_of(wl.hidden), bits_of(wl.weight)
    ref = oracle.lm_head_loss(H, Wt, wl.ids.cpu().numpy(), lp_mu.cpu().double().numpy(),
                              ref_in.cpu().double().numpy(), wl.adv.cpu().double().numpy(),
                              wl.mask.cpu().numpy(), None, params, want_grads=want_grads)
    ties = tie_mask(ref, params)
    lp = res.logp.cpu().double().numpy()
    assert_close_rel(lp, ref["lp"], 2e-3, "lp")
    assert_close_rel(lp, ref["lp"], 1e-4, "lp (tight)")
    lt = res.loss_tok.cpu().double().numpy()
    assert_close_rel(lt, ref["loss_tok"], 1e-4, "loss_tok", mask=~ties)
    fl = res.flags.cpu().numpy()
    assert np.array_equal(fl[~ties], ref["flags"][~ties]), "flags differ away from ties"
    st = res.stats.cpu().numpy()
    np.testing.assert_array_equal(st, oracle.stats_of(fl, params))
    if ties.sum() == 0:
        np.testing.assert_array_equal(st, ref["stats"])
        denom = np.nansum(np.abs(np.where(ref["valid"], ref["s"] * ref["loss_tok"], 0.0))) + 1e-30
        assert abs(res.loss.item() - ref["loss"]) <= 1e-5 * denom
    if want_grads:
        G = ref["dlogits"].copy()
        G[ties] = 0.0                      # tie rows may take either decision: excluded below
        keep = ~ties
        dh = res.dhidden.cpu().double().numpy()
        bound = _grad_bound(G, Wt)
        err = np.abs(dh - ref["dhidden"])
        assert np.all(err[keep] <= bound[keep]), f"dhidden: worst excess {np.max(err[keep] - bound[keep]):.3e}"
        if ties.sum() == 0:
            dw = res.dweight.cpu().double().numpy()
            bound = _grad_bound(G.T, H)
            err = np.abs(dw - ref["dweight"])
            assert np.all(err <= bound), f"dweight: worst excess {np.max(err - bound):.3e}"
    else:
        assert res.dhidden is None and res.dweight is None
    _say("lm_head ok", "ties", int(ties.sum()))
    return wl, res, ref


@pytest.mark.parametrize("rd_mode", ["none", "mask", "weight", "mask_weight"])
def test_small_ragged(rd_mode):
    # T and V not multiples of the 256 x 256 tile; d not a multiple of the 64-wide K step
    _run(200, 200, 1000, seed=1, rd_mode=rd_mode, bad_ids=(3, 4))


def test_several_token_tiles_odd_stage_count():
    # three token tiles (the last ragged), three vocabulary tiles, and d = 320: five K stages,
    # an odd count, so the two-stage ring runs one padded stage of zeros
    _run(600, 320, 700, seed=7)


def test_const_scale_and_unit_loss():
    _run(130, 256, 640, seed=2, scale_mode="const", loss_scale=1.0, mask_frac=0.0)


def test_vocab_chunks():
    # backward in vocabulary chunks of 256 rows (5 chunks, the last ragged)
    _run(256, 128, 1100, seed=3, vocab_chunk=256)


@pytest.mark.parametrize("kind", ["log_linear", "linear"])
def test_interpolated_reference(kind):
    _run(128, 128, 512, seed=4, ref_mode=kind, alpha=0.5, band=(0.99, 1.01), eps=(0.003, 0.004))


def test_forward_only():
    _run(96, 64, 300, seed=5, want_grads=False)


def test_single_token_single_tile():
    _run(1, 8, 5, seed=6, mask_frac=0.0)


def test_empty_batch():
    _say("lm_head empty")
    h = torch.zeros(0, 64, dtype=torch.bfloat16, device=DEV)
    w = torch.randn(300, 64, device=DEV).to(torch.bfloat16)
    e = torch.zeros(0, device=DEV)
    res = P.fused_lm_head_loss_fwd_bwd(h, w, torch.zeros(0, dtype=torch.int64, device=DEV), e, e, e)
    torch.cuda.synchronize()
    assert res.loss.item() == 0.0 and res.stats.sum().item() == 0
    assert res.dweight.abs().sum().item() == 0.0


def _fullsize_inputs():
    wl = W.make_lm_head_workload(DEV)
    T = wl.T
    lp_anchor = torch.empty(T, dtype=torch.float64)
    # anchor from a float32 torch pass (input synthesis only)
    for a in range(0, T, 512):
        z = wl.hidden[a:a + 512].float() @ wl.weight.float().T
        lse = torch.logsumexp(z, dim=1)
        lp_anchor[a:a + 512] = (z.gather(1, wl.ids[a:a + 512, None])[:, 0] - lse).double().cpu()
        del z
    lp_ref, lp_mu = W.reference_logprobs(lp_anchor, wl)
    return wl, lp_ref, lp_mu


def _z_rows(wl, rows, block=16384):
    """Oracle logits z[rows] = hidden[rows] weight^T in float64 from the bf16 bits."""
    H = bits_of(wl.hidden[torch.as_tensor(rows, device=DEV)])
    V = wl.V
    z = np.empty((len(rows), V))
    for a in range(0, V, block):
        z[:, a:a + block] = H @ bits_of(wl.weight[a:a + block]).T
    return H, z


def test_lm_head_workload_sampled_rows():
    """The full-size LM-head workload (T = 8192, d = 4096, V = 151936, every token valid), as
    the benchmark runs it: on 40 sampled rows (random, plus the first and the last), lp,
    loss_tok and flags against the oracle's row-level computation on z_t = hidden_t weight^T,
    and dhidden; on every row, the counters against the kernel's own flags; and dweight's
    columns summing to zero over the vocabulary (each G row sums to zero)."""
    _say("lm_head full size")
    wl, lp_ref, lp_mu = _fullsize_inputs()
    T, V = wl.T, wl.V
    res = P.fused_lm_head_loss_fwd_bwd(wl.hidden, wl.weight, wl.ids, lp_mu, lp_ref, wl.adv, wl.mask)
    torch.cuda.synchronize()
    rows = np.sort(np.concatenate([np.random.default_rng(0).choice(np.arange(1, T - 1), size=38,
                                                                   replace=False), [0, T - 1]]))
    H, z_rows = _z_rows(wl, rows)
    params = oracle_params((0.5, 2.0), (0.2, 0.2), "mask_weight", "token_mean", 1.0)
    scale = oracle.batch_scale(wl.mask.cpu().numpy(), params)
    ref = oracle.per_token(z_rows, wl.ids.cpu().numpy()[rows], lp_mu.cpu().double().numpy()[rows],
                           lp_ref.cpu().double().numpy()[rows], wl.adv.cpu().double().numpy()[rows],
                           wl.mask.cpu().numpy()[rows], None, params, scale, want_dlogits=True)
    ties = tie_mask(ref, params)
    lp = res.logp.cpu().double().numpy()[rows]
    assert_close_rel(lp, ref["lp"], 1e-4, "lp")
    lt = res.loss_tok.cpu().double().numpy()[rows]
    assert_close_rel(lt, ref["loss_tok"], 1e-4, "loss_tok", mask=~ties)
    fl_all = res.flags.cpu().numpy()
    assert np.array_equal(fl_all[rows][~ties], ref["flags"][~ties]), "flags differ away from ties"
    st = res.stats.cpu().numpy()
    np.testing.assert_array_equal(st, oracle.stats_of(fl_all, params))
    assert st[0] == T
    dh = res.dhidden[torch.as_tensor(rows, device=DEV)].cpu().double().numpy()
    G = ref["dlogits"].copy()
    G[ties] = 0.0
    dh_ref = np.zeros_like(dh)
    bound = np.zeros_like(dh)
    for a in range(0, V, 16384):
        Wb = bits_of(wl.weight[a:a + 16384])
        dh_ref += G[:, a:a + 16384] @ Wb
        bound += 2.0 ** -7 * (np.abs(G[:, a:a + 16384]) @ np.abs(Wb))
    keep = ~ties
    assert np.all(np.abs(dh - dh_ref)[keep] <= bound[keep] + 1e-7)
    # sum_v dweight[v] = sum_t (sum_v G[t, v]) hidden_t and every G row sums to zero; the
    # bf16 rounding of G leaves at most 2^-8 sum_v |G[t, v]| <= 2^-8 * 2 |w_t| per row, with
    # |w_t| <= s wd r_s |A| <= (1 / n_valid) * 2 * 1.2 * 1 here (band [0.5, 2], clip 0.2)
    col = res.dweight.double().sum(dim=0).cpu().numpy()
    n_valid = int(wl.mask.sum().item())
    habs = wl.hidden.float().abs().double().sum(dim=0).cpu().numpy()
    assert np.all(np.abs(col) <= 2.0 ** -7 * (4.8 / n_valid) * habs + 1e-9)
    _say("lm_head full size ok", st.tolist(), "ties", int(ties.sum()))


@pytest.mark.parametrize("vocab_chunk", [0, 38000])
def test_lm_head_fullsize_few_valid_tokens_every_gradient_entry(vocab_chunk):
    """The full-size launch (T = 8192, d = 4096, V = 151936: every tile of every kernel runs)
    with only 64 valid tokens, so that the oracle can form the whole gradient: every entry of
    dweight (all 151936 rows, including the last ragged vocabulary tile and the rows of the
    sampled ids) and of dhidden, plus the per-token outputs and the counters. The 64 valid
    tokens are drawn from candidates whose ratios lie away from every threshold, so no
    decision is a tie. vocab_chunk 38000 (rounded to 38144: four chunks, the last ragged)
    runs the chunked backward at this size; 0 runs the one-pass backward."""
    _say("lm_head full size, 64 valid tokens", vocab_chunk)
    wl, lp_ref, lp_mu = _fullsize_inputs()
    T, V = wl.T, wl.V
    params = oracle_params((0.5, 2.0), (0.2, 0.2), "mask_weight", "token_mean", 1.0)
    cand = np.sort(np.random.default_rng(5).choice(T, size=96, replace=False))
    H_c, z_c = _z_rows(wl, cand)
    probe = oracle.per_token(z_c, wl.ids.cpu().numpy()[cand], lp_mu.cpu().double().numpy()[cand],
                             lp_ref.cpu().double().numpy()[cand], wl.adv.cpu().double().numpy()[cand],
                             np.ones(len(cand), np.uint8), None, params, 1.0, want_dlogits=False)
    ok = np.nonzero(~tie_mask(probe, params))[0][:64]
    assert ok.size == 64
    rows = cand[ok]
    mask = torch.zeros(T, dtype=torch.uint8, device=DEV)
    mask[torch.as_tensor(rows, device=DEV)] = 1
    res = P.fused_lm_head_loss_fwd_bwd(wl.hidden, wl.weight, wl.ids, lp_mu, lp_ref, wl.adv, mask,
                                       vocab_chunk=vocab_chunk)
    torch.cuda.synchronize()
    H, z = H_c[ok], z_c[ok]
    m_np = mask.cpu().numpy()
    scale = oracle.batch_scale(m_np, params)
    ref = oracle.per_token(z, wl.ids.cpu().numpy()[rows], lp_mu.cpu().double().numpy()[rows],
                           lp_ref.cpu().double().numpy()[rows], wl.adv.cpu().double().numpy()[rows],
                           m_np[rows], None, params, scale, want_dlogits=True)
    assert not tie_mask(ref, params).any()
    lp = res.logp.cpu().double().numpy()
    assert_close_rel(lp[rows], ref["lp"], 1e-4, "lp")
    assert np.all(lp[m_np == 0] == 0.0)
    assert_close_rel(res.loss_tok.cpu().double().numpy()[rows], ref["loss_tok"], 1e-4, "loss_tok")
    fl = res.flags.cpu().numpy()
    assert np.array_equal(fl[rows], ref["flags"]) and np.all(fl[m_np == 0] == 0)
    np.testing.assert_array_equal(res.stats.cpu().numpy(), ref["stats"] if "stats" in ref
                                  else oracle.stats_of(ref["flags"], params))
    G = ref["dlogits"]
    dh = res.dhidden.cpu().double().numpy()
    assert np.all(dh[m_np == 0] == 0.0)
    dh_ref = np.zeros((64, H.shape[1]))
    dh_bound = np.zeros_like(dh_ref)
    dw = res.dweight
    worst = 0.0
    for a in range(0, V, 16384):
        b = min(V, a + 16384)
        Wb = bits_of(wl.weight[a:b])
        Gb = G[:, a:b]
        dh_ref += Gb @ Wb
        dh_bound += 2.0 ** -7 * (np.abs(Gb) @ np.abs(Wb))
        dw_ref = Gb.T @ H
        dw_bound = 2.0 ** -7 * (np.abs(Gb).T @ np.abs(H)) + 1e-7
        err = np.abs(dw[a:b].cpu().double().numpy() - dw_ref)
        assert np.all(err <= dw_bound), f"dweight rows {a}..{b}: worst excess {np.max(err - dw_bound):.3e}"
        worst = max(worst, float(np.max(err / dw_bound)))
    err = np.abs(dh[rows] - dh_ref)
    assert np.all(err <= dh_bound + 1e-7), f"dhidden: worst excess {np.max(err - dh_bound - 1e-7):.3e}"
    _say("lm_head 64 valid ok", vocab_chunk, "worst dW err / bound", round(worst, 4))


def test_lm_head_autograd_wrapper_returns_the_call_gradients():
    """FusedLMHeadLoss: loss.backward() gives hidden.grad and weight.grad equal to the direct
    call's dhidden and dweight times the upstream gradient, in the parameters' dtype."""
    T, d, V = 300, 64, 1000
    print(f"[case] lm head autograd T={T} d={d} V={V}", flush=True)
    g = torch.Generator(device=DEV).manual_seed(31)
    hidden = torch.randn(T, d, generator=g, device=DEV).to(torch.bfloat16)
    weight = (0.1 * torch.randn(V, d, generator=g, device=DEV)).to(torch.bfloat16)
    ids = torch.randint(0, V, (T,), generator=g, device=DEV)
    lp_ref = torch.full((T,), -7.0, device=DEV)
    lp_mu = lp_ref + 0.05 * torch.randn(T, generator=g, device=DEV)
    adv = torch.randn(T, generator=g, device=DEV)
    direct = P.fused_lm_head_loss_fwd_bwd(hidden, weight, ids, lp_mu, lp_ref, adv)
    h = hidden.clone().requires_grad_(True)
    w = weight.clone().requires_grad_(True)
    loss, lp, st = P.FusedLMHeadLoss.apply(h, w, ids, lp_mu, lp_ref, adv, None, None, None)
    (3.0 * loss).backward()
    torch.cuda.synchronize()
    assert torch.equal(loss.detach(), direct.loss[0]) and torch.equal(lp, direct.logp)
    assert h.grad.dtype == torch.bfloat16 and w.grad.dtype == torch.bfloat16
    assert torch.equal(h.grad, (3.0 * direct.dhidden).to(torch.bfloat16))
    assert torch.equal(w.grad, (3.0 * direct.dweight).to(torch.bfloat16))

