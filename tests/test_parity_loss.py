"""GPU parity of decoupled_ppo_loss_fwd_bwd (through the C ABI) against the float64 oracle.

Every case prints its name, shape and seed before it touches the GPU.
"""
import json
import math
import os

import numpy as np
import pytest
import torch

import oracle
import paper_2605_12070_amd as P
from paper_2605_12070_amd import workloads as W

from helpers import (TIGHT, assert_close_rel, bits_of, compare_loss, oracle_anchor,
                     oracle_params, run_oracle, tie_mask, torch_anchor)

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _say(*a):
    print("[case]", *a, flush=True)


def _run_case(wl_name, T=None, V=None, seed=None, seq_len=None, rd_mode="mask_weight",
              scale_mode="token_mean", loss_scale=1.0, band=(0.5, 2.0), eps=(0.2, 0.2),
              tscale=False, policy="auto", check_loss=True):
    _say(wl_name, T, V, seed, rd_mode, scale_mode, loss_scale, band, eps, tscale, policy)
    wl = W.make_workload(wl_name, device=DEV, T=T, V=V, seed=seed, seq_len=seq_len)
    anchor = oracle_anchor(wl.logits, wl.ids)
    lp_ref, lp_mu = W.reference_logprobs(anchor.to(DEV), wl)
    ts = None
    if tscale:
        g = torch.Generator(device=DEV).manual_seed(99)
        ts = torch.rand(wl.T, generator=g, device=DEV) * 1.5 + 0.25
    P.set_path_policy(policy)
    try:
        res = P.decoupled_ppo_loss_fwd_bwd(wl.logits, wl.ids, lp_mu, lp_ref, wl.adv, wl.mask, ts,
                                           band=band, clip_eps=eps, rd_mode=rd_mode,
                                           scale_mode=scale_mode, loss_scale=loss_scale)
        torch.cuda.synchronize()
    finally:
        P.set_path_policy("auto")
    params = oracle_params(band, eps, rd_mode, scale_mode, loss_scale)
    ref = run_oracle(wl.logits, wl.ids, lp_mu, lp_ref, wl.adv, wl.mask, ts, params)
    n_ties = compare_loss(res, ref, params, wl.logits.dtype)
    # stats: consistent with the kernel's own flags, equal to the oracle's without ties
    fl = res.flags.cpu().numpy()
    st = res.stats.cpu().numpy()
    np.testing.assert_array_equal(st, oracle.stats_of(fl, params))
    if n_ties == 0:
        np.testing.assert_array_equal(st, ref["stats"])
    if check_loss:
        denom = np.nansum(np.abs(np.where(ref["valid"], ref["s"] * ref["loss_tok"], 0.0))) + 1e-30
        if n_ties == 0:
            assert abs(res.loss.item() - ref["loss"]) <= 1e-5 * denom + 1e-30, \
                (res.loss.item(), ref["loss"])
        # the loss is the fixed-order sum of the kernel's own per-token values
        lt = res.loss_tok.cpu().double().numpy()
        s = ref["s"]
        own = float(np.sum(np.where(ref["valid"], s * lt, 0.0)))
        assert abs(res.loss.item() - own) <= 1e-6 * denom + 1e-30
    return wl, res, ref


@pytest.mark.parametrize("rd_mode", ["none", "mask", "weight", "mask_weight"])
@pytest.mark.parametrize("scale_mode", ["const", "token_mean"])
def test_tiny_fp32_all_modes(rd_mode, scale_mode):
    _run_case("tiny", rd_mode=rd_mode, scale_mode=scale_mode)


def test_tiny_fp32_token_scale_asymmetric_clip():
    _run_case("tiny", tscale=True, eps=(0.1, 0.3), scale_mode="const", loss_scale=0.5)


def test_tiny_stream_path_matches():
    _run_case("tiny", policy="stream")


@pytest.mark.parametrize("policy", ["auto", "stream"])
def test_small_vocab_bf16(policy):
    # 2 sequences of the 32000-vocabulary workload: spiked rows and +-1 lp_mu offsets
    _run_case("small_vocab", T=512, policy=policy)


def test_small_vocab_unit_scale_dlogits():
    # loss_scale = 1 makes dlogits O(1), so the relative bf16 bound is exercised
    _run_case("small_vocab", T=256, scale_mode="const", loss_scale=1.0)


@pytest.mark.parametrize("rd_mode", ["mask_weight", "weight"])
def test_large_vocab_full_rows(rd_mode):
    # full V = 151936: the 1024-thread x 19-chunk register-resident kernel
    _run_case("large_vocab", T=64, seq_len=8, rd_mode=rd_mode)


def test_large_vocab_unit_scale():
    _run_case("large_vocab", T=32, seq_len=4, scale_mode="const", loss_scale=1.0)


def test_large_vocab_paper_thresholds():
    # thresholds of the paper's threshold study (snap1003_1006) and Table 4's first row:
    # dense decisions near 1
    _run_case("large_vocab", T=64, seq_len=8, band=(1 / 1.003, 1.003), eps=(0.006, 0.006))
    _run_case("large_vocab", T=64, seq_len=8, band=(0.990, 1.010), eps=(0.003, 0.004))


def test_large_vocab_stream_path():
    _run_case("large_vocab", T=16, seq_len=2, policy="stream")


def test_long_agentic_masked_with_ewma_reference():
    # 40% observation tokens (mask 0), lp_ref = fixed-decay EWMA (beta = 0.9) of two
    # versions' log-probs; the GPU leg forms the proxy with ewma_proxy_update, the oracle
    # leg with its own recursion
    T = 512
    _say("long_agentic", T)
    wl = W.make_workload("long_agentic", device=DEV, T=T)
    anchor = oracle_anchor(wl.logits, wl.ids)
    lp_old, lp_prev, lp_mu = W.version_logprobs(anchor.to(DEV), wl)
    prox = lp_prev.clone()
    P.ewma_proxy_update(prox, lp_old, 0.9, normalized=False)
    ref_prox = oracle.ewma_fixed_step(lp_prev.cpu().double().numpy(),
                                      lp_old.cpu().double().numpy(), 0.9)
    np.testing.assert_allclose(prox.cpu().double().numpy(), ref_prox, rtol=1e-6, atol=1e-6)
    res = P.decoupled_ppo_loss_fwd_bwd(wl.logits, wl.ids, lp_mu, prox, wl.adv, wl.mask)
    torch.cuda.synchronize()
    params = oracle_params((0.5, 2.0), (0.2, 0.2), "mask_weight", "token_mean", 1.0)
    ref = oracle.decoupled_ppo_loss(bits_of(wl.logits), wl.ids.cpu().numpy(),
                                    lp_mu.cpu().double().numpy(), ref_prox,
                                    wl.adv.cpu().double().numpy(), wl.mask.cpu().numpy(),
                                    params=params)
    compare_loss(res, ref, params, wl.logits.dtype)
    m = wl.mask.cpu().numpy() == 0
    d = res.dlogits.cpu()
    assert torch.all(d[torch.from_numpy(m)] == 0)
    assert np.all(res.logp.cpu().numpy()[m] == 0) and np.all(res.flags.cpu().numpy()[m] == 0)
    assert res.stats[0].item() == int((~m).sum())


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("V", [1, 7, 8, 9, 1000, 1023, 1025, 4097, 32001, 77824, 77825,
                               151937, 155648, 155656])
def test_ragged_vocab_sizes(dtype, V):
    _say("ragged", dtype, V)
    T = 6
    g = torch.Generator(device=DEV).manual_seed(V)
    z = (torch.randn(T, V, generator=g, device=DEV) * 3).to(dtype)
    ids = torch.randint(0, V, (T,), generator=g, device=DEV)
    ids[0] = V - 1
    ids[1] = 0
    anchor = oracle_anchor(z, ids).to(DEV)
    lp_ref = (anchor + 0.1 * torch.randn(T, generator=g, device=DEV, dtype=torch.float64)).float()
    lp_mu = (lp_ref.double() + 0.05 * torch.randn(T, generator=g, device=DEV, dtype=torch.float64)).float()
    adv = torch.randn(T, generator=g, device=DEV)
    for policy in ("auto", "stream"):
        P.set_path_policy(policy)
        try:
            res = P.decoupled_ppo_loss_fwd_bwd(z, ids, lp_mu, lp_ref, adv, scale_mode="const")
            torch.cuda.synchronize()
        finally:
            P.set_path_policy("auto")
        params = oracle_params((0.5, 2.0), (0.2, 0.2), "mask_weight", "const", 1.0)
        ref = run_oracle(z, ids, lp_mu, lp_ref, adv, None, None, params)
        compare_loss(res, ref, params, dtype)


# One case per register-resident shape, with more rows than the grid has workgroups, so
# that a workgroup loops over at least three rows: both row buffers of the two-buffer
# kernels serve twice, and the persistent fp32 loop and the per-workgroup counters are
# exercised. Every 7th row is masked and a few valid rows carry bad ids, so rows that are
# not read (zero stores) alternate with rows that are.
RESIDENT_CASES = [
    (torch.bfloat16, 2000, 4600, "rows_bf16_resident<256, 1, true>"),
    (torch.bfloat16, 4000, 4600, "rows_bf16_resident<256, 2, true>"),
    (torch.bfloat16, 8192, 4600, "rows_bf16_resident<256, 4, true>"),
    (torch.bfloat16, 16000, 2000, "rows_bf16_resident_db<512, 4>"),
    (torch.bfloat16, 24000, 1400, "rows_bf16_resident_db<512, 6>"),
    (torch.bfloat16, 32000, 1400, "rows_bf16_resident_db<512, 8>"),
    (torch.bfloat16, 49000, 700, "rows_bf16_resident_db<1024, 6>"),
    (torch.bfloat16, 65536, 700, "rows_bf16_resident_db<1024, 8>"),
    (torch.bfloat16, 98000, 700, "rows_bf16_resident<1024, 12, true>"),
    (torch.float32, 1000, 4600, "rows_f32_resident<256, 1, true>"),
    (torch.float32, 4000, 4600, "rows_f32_resident<256, 4, true>"),
    (torch.float32, 8000, 2000, "rows_f32_resident<512, 4, true>"),
    (torch.float32, 16000, 1400, "rows_f32_resident<512, 8, true>"),
    (torch.float32, 24000, 700, "rows_f32_resident<1024, 6, true>"),
    (torch.float32, 76000, 700, "rows_f32_resident<1024, 19, true>"),
    # longer rows: resident prefix, streamed tail
    (torch.float32, 155656, 600, "rows_f32_prefix<1024, 19>"),
    (torch.bfloat16, 180000, 600, "rows_bf16_prefix<1024, 19>"),
]


@pytest.mark.parametrize("dtype,V,T,kernel", RESIDENT_CASES,
                         ids=[c[3].split("<")[0][5:] + f"_V{c[1]}" for c in RESIDENT_CASES])
def test_every_resident_shape_several_rows_per_workgroup(dtype, V, T, kernel):
    _say("resident shape", dtype, V, T, kernel)
    assert P.row_kernel_name(dtype, V) == "dppo::" + kernel
    g = torch.Generator(device=DEV).manual_seed(V + T)
    z = (torch.randn(T, V, generator=g, device=DEV) * 3).to(dtype)
    ids = torch.randint(0, V, (T,), generator=g, device=DEV)
    ids[5::97] = V + 1                                  # bad ids on valid rows
    mask = torch.ones(T, dtype=torch.uint8, device=DEV)
    mask[::7] = 0
    anchor = oracle_anchor(z, ids.clamp(0, V - 1)).to(DEV)
    lp_ref = (anchor + 0.2 * torch.randn(T, generator=g, device=DEV, dtype=torch.float64)).float()
    lp_mu = (lp_ref.double() + 0.3 * torch.randn(T, generator=g, device=DEV, dtype=torch.float64)).float()
    adv = torch.randn(T, generator=g, device=DEV)
    res = P.decoupled_ppo_loss_fwd_bwd(z, ids, lp_mu, lp_ref, adv, mask)
    torch.cuda.synchronize()
    params = oracle_params((0.5, 2.0), (0.2, 0.2), "mask_weight", "token_mean", 1.0)
    ref = run_oracle(z, ids, lp_mu, lp_ref, adv, mask, None, params)
    n_ties = compare_loss(res, ref, params, dtype)
    fl = res.flags.cpu().numpy()
    st = res.stats.cpu().numpy()
    np.testing.assert_array_equal(st, oracle.stats_of(fl, params))
    diff = np.abs(st.astype(np.int64) - np.asarray(ref["stats"], np.int64))
    assert diff[0] == 0 and diff[4] == 0 and np.all(diff <= n_ties), (st, ref["stats"], n_ties)
    assert st[4] == int(((ids.cpu().numpy() > V) & (mask.cpu().numpy() != 0)).sum()) > 0


@pytest.mark.parametrize("V,ld,T", [(77825, 77828, 500), (151937, 151940, 500),
                                    (151936, 151936, 7)])
def test_fp32_prefix_kernel_ragged_ends_and_strides(V, ld, T):
    """fp32 rows past the resident kernels with 16-byte-aligned strides: the resident-prefix
    kernel, with a ragged last chunk (V % 4 != 0) that one thread reads and writes element
    by element, a prefix that is the whole row but that end (V = 77825), in place and into a
    separate buffer, several rows per workgroup with masked rows and bad ids in between."""
    _say("fp32 prefix", V, ld, T)
    assert P.row_kernel_name(torch.float32, V, ld) == "dppo::rows_f32_prefix<1024, 19>"
    g = torch.Generator(device=DEV).manual_seed(V + T)
    zbuf = torch.full((T, ld), float("nan"), device=DEV)
    z = zbuf[:, :V]
    z.copy_(torch.randn(T, V, generator=g, device=DEV) * 3)
    ids = torch.randint(0, V, (T,), generator=g, device=DEV)
    ids[0] = V - 1                                      # in the ragged end
    ids[min(2, T - 1)] = 5
    if T > 40:
        ids[7::97] = V + 1                              # bad ids on valid rows
    mask = torch.ones(T, dtype=torch.uint8, device=DEV)
    mask[3::11] = 0
    anchor = oracle_anchor(z, ids.clamp(0, V - 1)).to(DEV)
    lp_ref = (anchor + 0.2 * torch.randn(T, generator=g, device=DEV, dtype=torch.float64)).float()
    lp_mu = (lp_ref.double() + 0.3 * torch.randn(T, generator=g, device=DEV, dtype=torch.float64)).float()
    adv = torch.randn(T, generator=g, device=DEV)
    params = oracle_params((0.5, 2.0), (0.2, 0.2), "mask_weight", "const", 1.0)
    ref = run_oracle(z, ids, lp_mu, lp_ref, adv, mask, None, params)
    dbuf = torch.full((T, ld), 7.0, device=DEV)
    res = P.decoupled_ppo_loss_fwd_bwd(z, ids, lp_mu, lp_ref, adv, mask, scale_mode="const",
                                       dlogits=dbuf[:, :V])
    torch.cuda.synchronize()
    compare_loss(res, ref, params, torch.float32)
    assert torch.all(dbuf[:, V:] == 7.0), "stores past the row"
    fl = res.flags.cpu().numpy()
    np.testing.assert_array_equal(res.stats.cpu().numpy(), oracle.stats_of(fl, params))
    inpl = P.decoupled_ppo_loss_fwd_bwd(z, ids, lp_mu, lp_ref, adv, mask, scale_mode="const",
                                        dlogits=z)
    torch.cuda.synchronize()
    assert torch.equal(z.view(torch.int32), res.dlogits.view(torch.int32)), "in place"
    assert torch.equal(inpl.logp.view(torch.int32), res.logp.view(torch.int32))
    assert torch.isnan(zbuf[:, V:]).all()


@pytest.mark.parametrize("V,ld,T", [(155649, 155656, 300), (262147, 262152, 300),
                                    (262144, 262144, 7)])
def test_bf16_prefix_kernel_ragged_ends_and_strides(V, ld, T):
    """bf16 rows past the resident kernels (more than 1024 x 19 x 8 = 155648 entries) with
    16-byte-aligned strides: the resident-prefix kernel, with a ragged last chunk (V % 8 != 0)
    that one thread reads and writes element by element, a prefix that is the whole row but
    one entry (V = 155649), the sampled id in the resident part, in the streamed tail and in
    the ragged end, in place and into a separate buffer, several rows per workgroup with
    masked rows and bad ids in between."""
    _say("bf16 prefix", V, ld, T)
    assert P.row_kernel_name(torch.bfloat16, V, ld) == "dppo::rows_bf16_prefix<1024, 19>"
    g = torch.Generator(device=DEV).manual_seed(V + T)
    zbuf = torch.full((T, ld), float("nan"), device=DEV, dtype=torch.bfloat16)
    z = zbuf[:, :V]
    z.copy_((torch.randn(T, V, generator=g, device=DEV) * 3).to(torch.bfloat16))
    ids = torch.randint(0, V, (T,), generator=g, device=DEV)
    ids[0] = V - 1                                      # in the ragged end (or the tail)
    ids[min(2, T - 1)] = 5                              # in the resident part
    ids[min(4, T - 1)] = 160000 if V > 160000 else V - 2   # in the streamed tail
    if T > 40:
        ids[7::97] = V + 1                              # bad ids on valid rows
    mask = torch.ones(T, dtype=torch.uint8, device=DEV)
    mask[3::11] = 0
    anchor = oracle_anchor(z, ids.clamp(0, V - 1)).to(DEV)
    lp_ref = (anchor + 0.2 * torch.randn(T, generator=g, device=DEV, dtype=torch.float64)).float()
    lp_mu = (lp_ref.double() + 0.3 * torch.randn(T, generator=g, device=DEV, dtype=torch.float64)).float()
    adv = torch.randn(T, generator=g, device=DEV)
    params = oracle_params((0.5, 2.0), (0.2, 0.2), "mask_weight", "const", 1.0)
    ref = run_oracle(z, ids, lp_mu, lp_ref, adv, mask, None, params)
    dbuf = torch.full((T, ld), 7.0, device=DEV, dtype=torch.bfloat16)
    res = P.decoupled_ppo_loss_fwd_bwd(z, ids, lp_mu, lp_ref, adv, mask, scale_mode="const",
                                       dlogits=dbuf[:, :V])
    torch.cuda.synchronize()
    compare_loss(res, ref, params, torch.bfloat16)
    assert torch.all(dbuf[:, V:] == 7.0), "stores past the row"
    fl = res.flags.cpu().numpy()
    np.testing.assert_array_equal(res.stats.cpu().numpy(), oracle.stats_of(fl, params))
    inpl = P.decoupled_ppo_loss_fwd_bwd(z, ids, lp_mu, lp_ref, adv, mask, scale_mode="const",
                                        dlogits=z)
    torch.cuda.synchronize()
    assert torch.equal(z.view(torch.int16), res.dlogits.view(torch.int16)), "in place"
    assert torch.equal(inpl.logp.view(torch.int32), res.logp.view(torch.int32))
    assert torch.isnan(zbuf[:, V:]).all()


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_unaligned_and_strided_rows(dtype):
    # base pointer off by one element and a row stride that is not a multiple of 16 bytes:
    # the element-wise streaming path
    T, V = 12, 5003
    _say("unaligned", dtype, T, V)
    ld = V + 3
    g = torch.Generator(device=DEV).manual_seed(5)
    buf = (torch.randn(T * ld + 1, generator=g, device=DEV) * 3).to(dtype)
    z = buf[1:1 + T * ld].view(T, ld)[:, :V]
    dbuf = torch.zeros(T * ld + 1, dtype=dtype, device=DEV)
    d = dbuf[1:1 + T * ld].view(T, ld)[:, :V]
    ids = torch.randint(0, V, (T,), generator=g, device=DEV)
    anchor = oracle_anchor(z, ids).to(DEV)
    lp_ref = (anchor + 0.1 * torch.randn(T, generator=g, device=DEV, dtype=torch.float64)).float()
    lp_mu = lp_ref.clone()
    adv = torch.randn(T, generator=g, device=DEV)
    res = P.decoupled_ppo_loss_fwd_bwd(z, ids, lp_mu, lp_ref, adv, dlogits=d, scale_mode="const")
    torch.cuda.synchronize()
    params = oracle_params((0.5, 2.0), (0.2, 0.2), "mask_weight", "const", 1.0)
    ref = run_oracle(z, ids, lp_mu, lp_ref, adv, None, None, params)
    compare_loss(res, ref, params, dtype)
    # the padding between rows and the element before the matrix are untouched
    pad = dbuf[1:1 + T * ld].view(T, ld)[:, V:]
    assert torch.all(pad == 0) and dbuf[0].item() == 0


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_in_place_dlogits(dtype):
    # 3000 rows: several per workgroup, so the bf16 two-buffer kernel swaps its buffers
    T, V = 3000, 32000
    _say("in_place", dtype, T, V)
    wl = W.make_workload("small_vocab", device=DEV, T=T, V=V, seed=7)
    z = wl.logits.to(dtype)
    anchor = oracle_anchor(z, wl.ids).to(DEV)
    lp_ref, lp_mu = W.reference_logprobs(anchor, wl)
    out_of_place = P.decoupled_ppo_loss_fwd_bwd(z, wl.ids, lp_mu, lp_ref, wl.adv)
    zz = z.clone()
    in_place = P.decoupled_ppo_loss_fwd_bwd(zz, wl.ids, lp_mu, lp_ref, wl.adv, dlogits=zz)
    torch.cuda.synchronize()
    assert torch.equal(in_place.dlogits, out_of_place.dlogits)
    assert in_place.dlogits.data_ptr() == zz.data_ptr()
    assert torch.equal(in_place.logp, out_of_place.logp)


# two-buffer rows, the flagship shape with several rows per workgroup, masked rows, rows
# with a phase
@pytest.mark.parametrize("name,T,V", [("small_vocab", 1024, None), ("large_vocab", 600, None),
                                      ("long_agentic", 600, None), ("small_vocab", 500, 151937)])
def test_deterministic_bitwise(name, T, V):
    """Three calls into dlogits buffers that start out as NaN and as zeros give the same bits:
    no entry is left unwritten or written from registers that were still being stored."""
    wl = W.make_workload(name, device=DEV, T=T, V=V, seed=11)
    _say("determinism", name, wl.T, wl.V)
    anchor = torch_anchor(wl.logits, wl.ids)
    lp_ref, lp_mu = W.reference_logprobs(anchor, wl)
    runs = []
    for fill in (float("nan"), 0.0, float("nan")):
        d = torch.full_like(wl.logits, fill)
        runs.append(P.decoupled_ppo_loss_fwd_bwd(wl.logits, wl.ids, lp_mu, lp_ref, wl.adv,
                                                 wl.mask, dlogits=d))
        torch.cuda.synchronize()
    a = runs[0]
    for b in runs[1:]:
        for x, y in ((a.loss, b.loss), (a.dlogits, b.dlogits), (a.logp, b.logp),
                     (a.stats, b.stats), (a.loss_tok, b.loss_tok), (a.flags, b.flags)):
            assert torch.equal(x.view(torch.uint8), y.view(torch.uint8))


# loss calls with the counters taken from the flags (count mode: the fp32 resident kernel)
# or counted by the kernels (every other family), against the same calls forced to count with
# the counting kernel and atomics
@pytest.mark.parametrize("name,T,V,rd_mode,scale_mode,bwd", [
    ("tiny", 256, None, "mask", "token_mean", True),
    ("small_vocab", 3000, None, "weight", "token_mean", True),
    ("large_vocab", 400, None, "mask_weight", "const", True),
    ("long_agentic", 700, 30000, "mask_weight", "token_mean", True),
    ("long_agentic", 700, 30000, "none", "token_mean", False),
    ("small_vocab", 500, 151937, "mask", "token_mean", True),
    ("long_agentic", 200, 262144, "mask_weight", "token_mean", True),
    ("tiny", 300, 151936, "mask_weight", "token_mean", True),
])
def test_counters_from_flags_equal_atomic_counters(name, T, V, rd_mode, scale_mode, bwd):
    wl = W.make_workload(name, device=DEV, T=T, V=V, seed=23)
    _say("count mode", name, wl.T, wl.V, rd_mode, scale_mode, bwd)
    anchor = torch_anchor(wl.logits, wl.ids)
    lp_ref, lp_mu = W.reference_logprobs(anchor, wl)
    ids = wl.ids.clone()
    ids[7] = wl.V + 3                                  # a bad id on a (probably) valid row
    res = {}
    for policy in ("auto", "auto+atomics"):
        P.set_path_policy(policy)
        try:
            out = None
            for _ in range(2):                         # stale outputs must not leak
                out = P.decoupled_ppo_loss_fwd_bwd(wl.logits, ids, lp_mu, lp_ref, wl.adv, wl.mask,
                                                   rd_mode=rd_mode, scale_mode=scale_mode,
                                                   loss_scale=0.5, want_dlogits=bwd, out=out)
            torch.cuda.synchronize()
        finally:
            P.set_path_policy("auto")
        res[policy] = out
    a, b = res["auto"], res["auto+atomics"]
    for x, y in ((a.stats, b.stats), (a.loss, b.loss), (a.logp, b.logp), (a.loss_tok, b.loss_tok),
                 (a.flags, b.flags)) + (((a.dlogits, b.dlogits),) if bwd else ()):
        assert torch.equal(x.view(torch.uint8), y.view(torch.uint8))
    st = a.stats.cpu().numpy()
    mask = wl.mask.cpu().numpy()
    assert st[P.STAT_N_VALID] == int((mask != 0).sum())
    params = oracle_params((0.5, 2.0), (0.2, 0.2), rd_mode, scale_mode, 0.5)
    np.testing.assert_array_equal(st, oracle.stats_of(a.flags.cpu().numpy(), params))


COUNT_KINDS = {  # logits dtype, V, row stride, the kernel expected (count mode)
    "f32": (torch.float32, 2000, 2000, "rows_f32_resident"),
    "bf16": (torch.bfloat16, 32000, 32000, "rows_bf16_resident_db"),
    "bf16_phase": (torch.bfloat16, 32000, 32001, "rows_bf16_phase_db"),
}


@pytest.mark.parametrize("kind", sorted(COUNT_KINDS))
@pytest.mark.parametrize("off", [0, 1, 3, 13])
def test_count_mode_mask_at_any_offset(kind, off):
    """The kernels that count the mask themselves (fp32 resident, bf16 with two row buffers)
    read it from the 16-byte boundary below it: a mask at any byte offset gives the counts,
    scale and outputs of the counting kernel, bit for bit."""
    dtype, V, ld, kname = COUNT_KINDS[kind]
    T = 3001
    _say("count mode mask offset", kind, off, T, V, ld)
    assert kname in P.row_kernel_name(dtype, V, ld)
    g = torch.Generator(device=DEV).manual_seed(41 + off)
    zbuf = (2.0 * torch.randn(T * ld + 8, generator=g, device=DEV)).to(dtype)
    z0 = 1 if ld != V else 0                         # the phase case starts off a 16-byte boundary
    z = zbuf[z0:z0 + T * ld].view(T, ld)[:, :V]
    dbuf = torch.zeros_like(zbuf)
    dl = dbuf[z0:z0 + T * ld].view(T, ld)[:, :V]     # dlogits in the logits' layout
    ids = torch.randint(0, V, (T,), generator=g, device=DEV)
    mbuf = (torch.rand(T + 16, generator=g, device=DEV) > 0.3).to(torch.uint8)
    mbuf[:off] = 7                                   # bytes before the mask must not count
    mbuf[off + T:] = 9                               # nor bytes after it
    mask = mbuf[off:off + T]
    lp_ref = torch.full((T,), -7.0, device=DEV) + 0.1 * torch.randn(T, generator=g, device=DEV)
    lp_mu = lp_ref + 0.05 * torch.randn(T, generator=g, device=DEV)
    adv = torch.randn(T, generator=g, device=DEV)
    res = {}
    for policy in ("auto", "auto+atomics"):
        P.set_path_policy(policy)
        try:
            r = P.decoupled_ppo_loss_fwd_bwd(z, ids, lp_mu, lp_ref, adv, mask, dlogits=dl)
            torch.cuda.synchronize()
            res[policy] = (r, dl.clone())
        finally:
            P.set_path_policy("auto")
    (a, da), (b, db) = res["auto"], res["auto+atomics"]
    for x, y in ((a.stats, b.stats), (a.loss, b.loss), (da, db), (a.logp, b.logp),
                 (a.loss_tok, b.loss_tok), (a.flags, b.flags)):
        assert torch.equal(x.view(torch.uint8), y.view(torch.uint8))
    assert a.stats[P.STAT_N_VALID].item() == int(mask.sum().item())


def test_masked_rows_bad_ids_and_nonfinite_rows():
    T, V = 10, 3000
    _say("edge rows", T, V)
    g = torch.Generator(device=DEV).manual_seed(3)
    for dtype in (torch.float32, torch.bfloat16):
        z = (torch.randn(T, V, generator=g, device=DEV) * 2).to(dtype)
        ids = torch.randint(0, V, (T,), generator=g, device=DEV)
        z[2, 17] = float("nan")            # NaN row
        z[3, 5] = float("inf")             # +inf row
        z[4, :] = float("-inf")            # all -inf row
        z[5, ::2] = float("-inf")          # some -inf entries
        ids[5] = 1
        z[6, :] = float("nan")             # masked: never read
        ids[7] = V                         # bad id on a valid row
        ids[8] = -5                        # bad id on a masked row
        mask = torch.ones(T, dtype=torch.uint8, device=DEV)
        mask[6] = 0
        mask[8] = 0
        lp_ref = torch.full((T,), -8.0, device=DEV)
        lp_mu = lp_ref.clone()
        adv = torch.linspace(-1, 1, T, device=DEV)
        for policy in ("auto", "stream"):
            P.set_path_policy(policy)
            try:
                res = P.decoupled_ppo_loss_fwd_bwd(z, ids, lp_mu, lp_ref, adv, mask,
                                                   scale_mode="const")
                torch.cuda.synchronize()
            finally:
                P.set_path_policy("auto")
            params = oracle_params((0.5, 2.0), (0.2, 0.2), "mask_weight", "const", 1.0)
            ref = run_oracle(z, ids, lp_mu, lp_ref, adv, mask, None, params)
            compare_loss(res, ref, params, dtype)
            st = res.stats.cpu().numpy()
            assert st[P.STAT_N_VALID] == 8 and st[P.STAT_N_BAD] == 1
            assert math.isnan(res.loss.item()) and math.isnan(ref["loss"])


# (dtype, V, T): the row kernel families, with T above the persistent grid where the row is
# short enough for the oracle to take it
NONFINITE_CASES = [
    (torch.bfloat16, 32000, 700),     # two-buffer 512 x 8
    (torch.bfloat16, 151936, 260),    # the flagship 1024 x 19, a second row per workgroup
    (torch.bfloat16, 50257, 300),     # rows with a phase (odd V)
    (torch.bfloat16, 262144, 40),     # resident prefix, streamed tail
    (torch.float32, 76000, 260),      # fp32 1024 x 19
    (torch.float32, 151936, 40),      # fp32 resident prefix
    (torch.float32, 32000, 40),       # fp32 one workgroup per row
]


@pytest.mark.parametrize("dtype,V,T", NONFINITE_CASES,
                         ids=[f"{str(c[0])[6:]}-{c[1]}-{c[2]}" for c in NONFINITE_CASES])
def test_nonfinite_rows_every_kernel_family(dtype, V, T):
    """NaN, +inf, all -inf and partly -inf rows, masked rows full of NaN and bad ids, at the
    start of the batch and again at its end (rows a persistent workgroup reaches after
    others), with and without dlogits: IEEE propagation as in the oracle."""
    _say("nonfinite rows", dtype, V, T)
    g = torch.Generator(device=DEV).manual_seed(V % 1000 + T)
    z = (torch.randn(T, V, generator=g, device=DEV) * 2).to(dtype)
    ids = torch.randint(0, V, (T,), generator=g, device=DEV)
    mask = torch.ones(T, dtype=torch.uint8, device=DEV)
    for b in (0, T - 9):
        z[b + 1, V // 3] = float("nan")    # NaN entry
        z[b + 2, V - 1] = float("inf")     # +inf entry at the row's end
        z[b + 3, :] = float("-inf")        # all -inf
        z[b + 4, 1::2] = float("-inf")     # every other entry -inf, the sampled one finite
        ids[b + 4] = 0
        z[b + 5, :] = float("nan")         # masked: never read
        mask[b + 5] = 0
        ids[b + 6] = V                     # bad id on a valid row
        ids[b + 7] = -1                    # bad id on a masked row
        mask[b + 7] = 0
        z[b + 8, 0] = float("inf")         # +inf at the row's start, sampled
        ids[b + 8] = 0
    lp_ref = torch.full((T,), -8.0, device=DEV)
    lp_mu = lp_ref.clone()
    adv = torch.linspace(-1, 1, T, device=DEV)
    params = oracle_params((0.5, 2.0), (0.2, 0.2), "mask_weight", "const", 1.0)
    ref = run_oracle(z, ids, lp_mu, lp_ref, adv, mask, None, params)
    for want in (True, False):
        res = P.decoupled_ppo_loss_fwd_bwd(z, ids, lp_mu, lp_ref, adv, mask, scale_mode="const",
                                           want_dlogits=want)
        torch.cuda.synchronize()
        compare_loss(res, ref, params, dtype)
        st = res.stats.cpu().numpy()
        assert st[P.STAT_N_VALID] == T - 4 and st[P.STAT_N_BAD] == 2
        assert math.isnan(res.loss.item()) and math.isnan(ref["loss"])
    # the log-prob call reads every row, masked ones included
    lp = P.logprob_fwd(z, ids)
    torch.cuda.synchronize()
    want_lp = oracle.logprob_fwd(_host_f64(z), ids.cpu().numpy())[0]
    got = lp.cpu().double().numpy()
    assert np.array_equal(np.isnan(got), np.isnan(want_lp))
    assert_close_rel(got, want_lp, TIGHT, "log-prob call")


def _host_f64(z):
    if z.dtype == torch.bfloat16:
        return oracle.bf16_bits_to_f64(z.cpu().view(torch.int16).numpy().view(np.uint16))
    return z.cpu().double().numpy()


def test_empty_batch():
    z = torch.zeros(0, 16, device=DEV)
    e = torch.zeros(0, device=DEV)
    res = P.decoupled_ppo_loss_fwd_bwd(z, torch.zeros(0, dtype=torch.int64, device=DEV), e, e, e)
    torch.cuda.synchronize()
    assert res.loss.item() == 0.0 and res.stats.tolist() == [0, 0, 0, 0, 0]


def test_worked_example_through_the_kernel():
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "loss_worked_example.json")))
    z_row = [math.log(v) for v in g["logits_row"]["log_terms"]]
    toks = g["tokens"]
    T = len(toks)
    z = torch.tensor([z_row] * T, dtype=torch.float32, device=DEV)
    ids = torch.tensor([t["y"] for t in toks], device=DEV)
    lpt = [math.log(g["lp_theta"][t["name"]][0]) for t in toks]
    lp_ref = torch.tensor([a - math.log(t["r_s"]) for a, t in zip(lpt, toks)], device=DEV)
    lp_mu = torch.tensor([a - math.log(t["r_s"]) - math.log(t["r_d"]) for a, t in zip(lpt, toks)],
                         device=DEV)
    adv = torch.tensor([t["adv"] for t in toks], device=DEV)
    for mode, exp in g["modes"].items():
        _say("worked example", mode)
        res = P.decoupled_ppo_loss_fwd_bwd(z, ids, lp_mu, lp_ref, adv, rd_mode=mode,
                                           scale_mode="const")
        torch.cuda.synchronize()
        np.testing.assert_allclose(res.loss_tok.cpu().numpy(), exp["loss_tok"], atol=2e-6)
        np.testing.assert_allclose(res.dlogits.cpu().numpy(), np.array(exp["dlogits"]), atol=2e-6)
        assert abs(res.loss.item() - exp["loss"]) < 1e-5
        assert res.stats.cpu().tolist() == exp["stats"]


def test_forward_only_and_autograd_wrapper():
    wl = W.make_workload("tiny", device=DEV)
    anchor = oracle_anchor(wl.logits, wl.ids).to(DEV)
    lp_ref, lp_mu = W.reference_logprobs(anchor, wl)
    fwd = P.decoupled_ppo_loss_fwd_bwd(wl.logits, wl.ids, lp_mu, lp_ref, wl.adv, want_dlogits=False)
    both = P.decoupled_ppo_loss_fwd_bwd(wl.logits, wl.ids, lp_mu, lp_ref, wl.adv)
    torch.cuda.synchronize()
    assert fwd.dlogits is None
    assert torch.equal(fwd.loss, both.loss) and torch.equal(fwd.logp, both.logp)
    z = wl.logits.clone().requires_grad_(True)
    loss, lp, st = P.DecoupledPPOLoss.apply(z, wl.ids, lp_mu, lp_ref, wl.adv, None, None, None)
    (2.0 * loss).backward()
    torch.cuda.synchronize()
    assert torch.allclose(z.grad, 2.0 * both.dlogits, rtol=0, atol=0)


@pytest.mark.parametrize("dtype,V", [(torch.bfloat16, 32000), (torch.bfloat16, 2000),
                                     (torch.float32, 4000), (torch.float32, 32000)])
def test_forward_only_matches_backward_on_many_short_rows(dtype, V):
    # the forward-only kernels sum their counters per workgroup like the backward ones:
    # per-token outputs, the loss and all five counters agree bit for bit
    T = 5000
    _say("fwd-only vs fwd+bwd", dtype, T, V)
    g = torch.Generator(device=DEV).manual_seed(V)
    z = (torch.randn(T, V, generator=g, device=DEV) * 3).to(dtype)
    ids = torch.randint(0, V, (T,), generator=g, device=DEV)
    ids[3::101] = -1
    mask = (torch.rand(T, generator=g, device=DEV) > 0.3).to(torch.uint8)
    lp_ref = torch.randn(T, generator=g, device=DEV) - 8.0
    lp_mu = lp_ref + 0.5 * torch.randn(T, generator=g, device=DEV)
    adv = torch.randn(T, generator=g, device=DEV)
    fwd = P.decoupled_ppo_loss_fwd_bwd(z, ids, lp_mu, lp_ref, adv, mask, want_dlogits=False)
    both = P.decoupled_ppo_loss_fwd_bwd(z, ids, lp_mu, lp_ref, adv, mask)
    torch.cuda.synchronize()
    assert torch.equal(fwd.logp.view(torch.int32), both.logp.view(torch.int32))
    assert torch.equal(fwd.loss_tok, both.loss_tok) and torch.equal(fwd.loss, both.loss)
    assert torch.equal(fwd.flags, both.flags) and torch.equal(fwd.stats, both.stats)
    st = both.stats.cpu().numpy()
    fl = both.flags.cpu().numpy()
    assert st[0] == int(mask.sum().item())
    assert st[4] == int(((ids.cpu().numpy() < 0) & (mask.cpu().numpy() != 0)).sum()) > 0
    params = oracle_params((0.5, 2.0), (0.2, 0.2), "mask_weight", "token_mean", 1.0)
    np.testing.assert_array_equal(st, oracle.stats_of(fl, params))


@pytest.mark.parametrize("kind", ["log_linear", "linear"])
@pytest.mark.parametrize("wl_name,T,n_gap,band,eps", [
    ("tiny", None, 1, (0.5, 2.0), (0.2, 0.2)),
    ("large_vocab", 64, 1, (0.99, 1.01), (0.003, 0.004)),      # Table 4, first block
    ("large_vocab", 64, 3, (1 / 1.003, 1.003), (0.006, 0.006)),
])
def test_interpolated_reference(kind, wl_name, T, n_gap, band, eps):
    """ref_mode log_linear / linear (App. A): the kernel builds pi_ref from mu_old and its own
    log-prob; the oracle takes the same proxy of its own float64 log-prob. Then Prop. 1 through
    the kernel: its kept tokens are those whose total ratio lies inside the effective bounds
    that the library's threshold helper reports."""
    alpha = 1.0 / (n_gap + 1)
    _say("interpolated ref", kind, wl_name, T, alpha, band, eps)
    wl = W.make_workload(wl_name, device=DEV, T=T, seq_len=8 if T else None)
    anchor = oracle_anchor(wl.logits, wl.ids)                 # oracle lp, float64
    _, lp_mu = W.reference_logprobs(anchor.to(DEV), wl)
    res = P.decoupled_ppo_loss_fwd_bwd(wl.logits, wl.ids, lp_mu, None, wl.adv, wl.mask,
                                       band=band, clip_eps=eps, ref_mode=kind, alpha=alpha)
    torch.cuda.synchronize()
    proxy = (oracle.log_linear_proxy_logprob if kind == "log_linear"
             else oracle.linear_proxy_logprob)(lp_mu.cpu().double().numpy(), anchor.numpy(), alpha)
    params = oracle_params(band, eps, "mask_weight", "token_mean", 1.0)
    ref = run_oracle(wl.logits, wl.ids, lp_mu, torch.from_numpy(proxy), wl.adv, wl.mask, None,
                     params)
    n_ties = compare_loss(res, ref, params, wl.logits.dtype)
    # Prop. 1: band and PPO decisions on the decoupled ratios = bounds on the total ratio
    m, c = P.effective_thresholds(band, (1 - eps[0], 1 + eps[1]), alpha, kind)
    r = np.exp(anchor.numpy() - lp_mu.cpu().double().numpy())
    adv = wl.adv.cpu().numpy()
    keep_eff = (r >= m[0]) & (r <= m[1]) & np.where(adv >= 0, r <= c[1], r >= c[0])
    fl = res.flags.cpu().numpy()
    keep = ((fl & P.FLAG_BAND) != 0) & ((fl & P.FLAG_PPO) != 0)
    bounds = np.log(np.array([b for b in (*m, *c) if np.isfinite(b) and b > 0]))
    edge = np.min(np.abs(np.log(r)[:, None] - bounds[None]), axis=1) < 1e-4
    assert np.array_equal(keep[~edge], keep_eff[~edge])
    _say("interpolated ref ok", kind, wl_name, "ties", n_ties, "kept", int(keep.sum()), "of", len(keep))


@pytest.mark.parametrize("V", [1000, 8192, 32000, 77824, 151936, 155648])
def test_forward_only_kernel_matches_gradient_call(V):
    """The forward-only call (its own row kernel for bf16) returns bit-for-bit the values of
    the call that also writes dlogits, on a batch with masked rows (40 %) and bad ids, and
    both match the oracle."""
    T = 96
    _say("forward-only", V, T)
    wl = W.make_workload("long_agentic", device=DEV, T=T, V=V, seq_len=48)
    wl.ids[5] = V + 2
    wl.ids[6] = -3
    anchor = oracle_anchor(wl.logits, wl.ids)
    lp_ref, lp_mu = W.reference_logprobs(anchor.to(DEV), wl)
    fwd = P.decoupled_ppo_loss_fwd_bwd(wl.logits, wl.ids, lp_mu, lp_ref, wl.adv, wl.mask,
                                       want_dlogits=False)
    both = P.decoupled_ppo_loss_fwd_bwd(wl.logits, wl.ids, lp_mu, lp_ref, wl.adv, wl.mask)
    torch.cuda.synchronize()
    for f in ("logp", "loss_tok", "flags", "stats", "loss"):
        a, b = getattr(fwd, f).cpu(), getattr(both, f).cpu()
        assert torch.equal(a.nan_to_num(7.0), b.nan_to_num(7.0)), f
    params = oracle_params((0.5, 2.0), (0.2, 0.2), "mask_weight", "token_mean", 1.0)
    ref = run_oracle(wl.logits, wl.ids, lp_mu, lp_ref, wl.adv, wl.mask, None, params)
    compare_loss(both, ref, params, wl.logits.dtype)


def test_short_form_matches_the_full_call():
    """decoupled_ppo_loss(...) -> (loss, lp, dlogits, stats) returns the full call's outputs."""
    wl = W.make_workload("small_vocab", device=DEV, T=300, seed=5)
    anchor = oracle_anchor(wl.logits, wl.ids).to(DEV)
    lp_ref, lp_mu = W.reference_logprobs(anchor, wl)
    loss, lp, d, st = P.decoupled_ppo_loss(wl.logits, wl.ids, lp_mu, lp_ref, wl.adv, wl.mask,
                                           band=(0.6, 1.8), eps=(0.1, 0.3), rd_mode="mask")
    full = P.decoupled_ppo_loss_fwd_bwd(wl.logits, wl.ids, lp_mu, lp_ref, wl.adv, wl.mask,
                                        band=(0.6, 1.8), clip_eps=(0.1, 0.3), rd_mode="mask")
    torch.cuda.synchronize()
    assert loss.dim() == 0 and torch.equal(loss.view(1), full.loss)
    assert torch.equal(lp, full.logp) and torch.equal(st, full.stats)
    assert torch.equal(d.view(torch.int16), full.dlogits.view(torch.int16))
