"""bf16 rows that do not start on a 16-byte boundary or are not a whole number of 16-byte
chunks long: the phase kernels read each row as the aligned chunks that cover it and write
only the row's own entries. Every case compares lp, loss_tok, flags and dlogits with the
oracle, and checks that every byte of the buffers outside the rows is left as it was
(the entries between rows, before the first row and after the last)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2605_12070_amd as P

from helpers import compare_loss, oracle_anchor, oracle_params, run_oracle

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
SENTINEL = 7.0                      # exactly representable in bf16


def _say(*a):
    print("[case]", *a, flush=True)


def _inputs(T, V, ld, off, seed):
    """Logits rows of length V at element offset `off` of a buffer, row stride ld; ids with
    the first and last entries of rows, a bad id, masked rows."""
    g = torch.Generator(device=DEV).manual_seed(seed)
    n = off + T * ld + 16
    buf = (torch.randn(n, generator=g, device=DEV) * 3).to(torch.bfloat16)
    z = buf[off:off + T * ld].view(T, ld)[:, :V]
    ids = torch.randint(0, V, (T,), generator=g, device=DEV)
    ids[0] = V - 1
    ids[1] = 0
    if T > 5:
        ids[5] = V + 3                   # bad id on a valid row
    mask = torch.ones(T, dtype=torch.uint8, device=DEV)
    mask[3::7] = 0
    anchor = oracle_anchor(z, ids.clamp(0, V - 1)).to(DEV)
    lp_ref = (anchor + 0.2 * torch.randn(T, generator=g, device=DEV, dtype=torch.float64)).float()
    lp_mu = (lp_ref.double() + 0.1 * torch.randn(T, generator=g, device=DEV,
                                                 dtype=torch.float64)).float()
    adv = torch.randn(T, generator=g, device=DEV)
    return buf, z, ids, mask, lp_mu, lp_ref, adv


def _outside(buf, off, T, ld, V):
    """Boolean mask of the buffer entries that belong to no row."""
    m = torch.ones(buf.numel(), dtype=torch.bool, device=buf.device)
    rows = off + torch.arange(T, device=buf.device)[:, None] * ld + torch.arange(V, device=buf.device)[None, :]
    m[rows.reshape(-1)] = False
    return m


CASES = [  # T, V, extra columns per row, element offset of row 0
    (40, 1, 0, 3), (40, 9, 0, 1), (300, 1003, 0, 0), (300, 1003, 5, 7), (200, 5003, 3, 1),
    (600, 8192, 1, 0), (120, 32001, 0, 5), (64, 50257, 0, 0), (64, 50257, 47, 2),
    (24, 151665, 271, 0), (24, 151937, 0, 6), (12, 155641, 0, 7),
]


@pytest.mark.parametrize("T,V,extra,off", CASES, ids=[f"T{c[0]}_V{c[1]}_x{c[2]}_o{c[3]}" for c in CASES])
def test_phase_rows_loss_and_untouched_neighbours(T, V, extra, off):
    ld = V + extra
    _say("phase rows", T, V, ld, off)
    buf, z, ids, mask, lp_mu, lp_ref, adv = _inputs(T, V, ld, off, seed=V + off)
    name = P.row_kernel_name(torch.bfloat16, V, ld)
    if (ld % 8 == 0) and (V % 8 == 0):
        assert "phase" not in name
    else:
        assert "phase" in name or "prefix" in name, name
    # dlogits into a second buffer with the same layout, filled with a sentinel
    dbuf = torch.full_like(buf, SENTINEL)
    d = dbuf[off:off + T * ld].view(T, ld)[:, :V]
    params = oracle_params((0.5, 2.0), (0.2, 0.2), "mask_weight", "const", 1.0)
    res = P.decoupled_ppo_loss_fwd_bwd(z, ids, lp_mu, lp_ref, adv, mask, dlogits=d,
                                       scale_mode="const")
    torch.cuda.synchronize()
    ref = run_oracle(z, ids, lp_mu, lp_ref, adv, mask, None, params)
    compare_loss(res, ref, params, torch.bfloat16)
    out = _outside(dbuf, off, T, ld, V)
    assert torch.all(dbuf[out] == SENTINEL), "entries outside the rows were written"
    # in place: the gradient overwrites the rows, and only the rows
    zin = buf.clone()
    zz = zin[off:off + T * ld].view(T, ld)[:, :V]
    res2 = P.decoupled_ppo_loss_fwd_bwd(zz, ids, lp_mu, lp_ref, adv, mask, dlogits=zz,
                                        scale_mode="const")
    torch.cuda.synchronize()
    assert torch.equal(zz.view(torch.int16), d.view(torch.int16)), "in place differs"
    assert torch.equal(zin[out].view(torch.int16), buf[out].view(torch.int16))
    assert torch.equal(res2.logp.view(torch.int32), res.logp.view(torch.int32))


@pytest.mark.parametrize("T,V,extra,off", CASES[:8], ids=[f"T{c[0]}_V{c[1]}_x{c[2]}_o{c[3]}" for c in CASES[:8]])
def test_phase_rows_forward_only(T, V, extra, off):
    ld = V + extra
    _say("phase rows forward", T, V, ld, off)
    buf, z, ids, mask, lp_mu, lp_ref, adv = _inputs(T, V, ld, off, seed=3 * V + off)
    lp = P.logprob_fwd(z, ids.clamp(0, V - 1))
    params = oracle_params((0.5, 2.0), (0.2, 0.2), "mask_weight", "const", 1.0)
    res = P.decoupled_ppo_loss_fwd_bwd(z, ids, lp_mu, lp_ref, adv, mask, want_dlogits=False,
                                       scale_mode="const")
    torch.cuda.synchronize()
    ref_lp, _ = oracle.logprob_fwd(oracle.bf16_bits_to_f64(
        z.cpu().view(torch.int16).numpy().view(np.uint16)), ids.clamp(0, V - 1).cpu().numpy())
    got = lp.cpu().double().numpy()
    assert np.all(np.abs(got - ref_lp) <= 2e-5 * np.maximum(np.abs(ref_lp), 1.0))
    ref = run_oracle(z, ids, lp_mu, lp_ref, adv, mask, None, params, want_dlogits=False)
    compare_loss(res, ref, params, torch.bfloat16, check_dlogits=False)


F32_CASES = [(300, 1003, 1), (200, 5003, 1), (120, 32001, 3), (40, 77821, 3)]


@pytest.mark.parametrize("T,V,extra", F32_CASES, ids=[f"T{c[0]}_V{c[1]}_x{c[2]}" for c in F32_CASES])
def test_fp32_ragged_rows_on_an_aligned_stride(T, V, extra):
    """fp32 rows whose length is not a multiple of 4 on a 16-byte stride: the resident kernel
    with its last entries loaded and stored one by one; the stride's padding is left alone."""
    ld = V + extra
    assert ld % 4 == 0
    _say("fp32 ragged rows", T, V, ld)
    assert P.row_kernel_name(torch.float32, V, ld).startswith("dppo::rows_f32_resident")
    g = torch.Generator(device=DEV).manual_seed(V)
    buf = torch.randn(T * ld, generator=g, device=DEV) * 3
    z = buf.view(T, ld)[:, :V]
    ids = torch.randint(0, V, (T,), generator=g, device=DEV)
    ids[0] = V - 1
    ids[2] = V - 2
    ids[5] = -1
    mask = torch.ones(T, dtype=torch.uint8, device=DEV)
    mask[3::7] = 0
    anchor = oracle_anchor(z, ids.clamp(0, V - 1)).to(DEV)
    lp_ref = (anchor + 0.2 * torch.randn(T, generator=g, device=DEV, dtype=torch.float64)).float()
    lp_mu = (lp_ref.double() + 0.1 * torch.randn(T, generator=g, device=DEV,
                                                 dtype=torch.float64)).float()
    adv = torch.randn(T, generator=g, device=DEV)
    dbuf = torch.full_like(buf, SENTINEL)
    d = dbuf.view(T, ld)[:, :V]
    params = oracle_params((0.5, 2.0), (0.2, 0.2), "mask_weight", "const", 1.0)
    res = P.decoupled_ppo_loss_fwd_bwd(z, ids, lp_mu, lp_ref, adv, mask, dlogits=d,
                                       scale_mode="const")
    lp = P.logprob_fwd(z, ids.clamp(0, V - 1))
    torch.cuda.synchronize()
    ref = run_oracle(z, ids, lp_mu, lp_ref, adv, mask, None, params)
    compare_loss(res, ref, params, torch.float32)
    assert torch.all(dbuf.view(T, ld)[:, V:] == SENTINEL)
    ref_lp, _ = oracle.logprob_fwd(z.cpu().double().numpy(), ids.clamp(0, V - 1).cpu().numpy())
    assert np.all(np.abs(lp.cpu().double().numpy() - ref_lp) <= 1e-5 * np.maximum(np.abs(ref_lp), 1.0))
    # in place
    zz = buf.clone().view(T, ld)
    P.decoupled_ppo_loss_fwd_bwd(zz[:, :V], ids, lp_mu, lp_ref, adv, mask, dlogits=zz[:, :V],
                                 scale_mode="const")
    torch.cuda.synchronize()
    assert torch.equal(zz[:, :V], d) and torch.equal(zz[:, V:], buf.view(T, ld)[:, V:])


def test_phase_rows_with_a_mismatched_gradient_layout_take_the_streaming_path():
    """dlogits at another offset within 16 bytes than the logits: the phase kernels cannot
    serve it, the streaming kernel does, with the same results."""
    T, V, ld, off = 50, 1003, 1003, 1
    buf, z, ids, mask, lp_mu, lp_ref, adv = _inputs(T, V, ld, off, seed=99)
    dbuf = torch.full((off + 1 + T * ld + 16,), SENTINEL, dtype=torch.bfloat16, device=DEV)
    d = dbuf[off + 1:off + 1 + T * ld].view(T, ld)[:, :V]
    params = oracle_params((0.5, 2.0), (0.2, 0.2), "mask_weight", "const", 1.0)
    res = P.decoupled_ppo_loss_fwd_bwd(z, ids, lp_mu, lp_ref, adv, mask, dlogits=d,
                                       scale_mode="const")
    torch.cuda.synchronize()
    ref = run_oracle(z, ids, lp_mu, lp_ref, adv, mask, None, params)
    compare_loss(res, ref, params, torch.bfloat16)
    out = _outside(dbuf, off + 1, T, ld, V)
    assert torch.all(dbuf[out] == SENTINEL)


def _random_cases(n=36, seed=2605):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        dtype = "bf16" if rng.random() < 0.7 else "f32"
        V = int(rng.choice([int(rng.integers(1, 64)), int(rng.integers(64, 4096)),
                            int(rng.integers(4096, 40000)), int(rng.integers(40000, 160000))]))
        extra = int(rng.choice([0, 0, int(rng.integers(1, 9)), 8 - V % 8]))
        off = int(rng.choice([0, 0, int(rng.integers(1, 8))]))
        T = int(max(2, min(400, 3_000_000 // max(V, 1))))
        out.append((i, dtype, T, V, extra, off, bool(rng.random() < 0.3), bool(rng.random() < 0.25)))
    return out


@pytest.mark.parametrize("i,dtype,T,V,extra,off,in_place,fwd_only", _random_cases(),
                         ids=[f"{c[0]}_{c[1]}_T{c[2]}_V{c[3]}_x{c[4]}_o{c[5]}" for c in _random_cases()])
def test_random_layouts_against_the_oracle(i, dtype, T, V, extra, off, in_place, fwd_only):
    """Seeded random layouts (dtype, V, stride, offset of the first row, T), with masked rows,
    bad ids, in place or into a second buffer, with or without dlogits: every output against
    the oracle, and no entry outside the rows written."""
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    ld = V + extra
    _say("random layout", i, dtype, T, V, ld, off, in_place, fwd_only)
    g = torch.Generator(device=DEV).manual_seed(1000 + i)
    n = off + T * ld + 16
    buf = (torch.randn(n, generator=g, device=DEV) * 3).to(tdt)
    ref_buf = buf.clone()
    z = buf[off:off + T * ld].view(T, ld)[:, :V]
    ids = torch.randint(0, V, (T,), generator=g, device=DEV)
    ids[torch.rand(T, generator=g, device=DEV) < 0.05] = V
    mask = (torch.rand(T, generator=g, device=DEV) >= 0.15).to(torch.uint8)
    anchor = oracle_anchor(z, ids.clamp(0, V - 1)).to(DEV)
    lp_ref = (anchor + 0.2 * torch.randn(T, generator=g, device=DEV, dtype=torch.float64)).float()
    lp_mu = (lp_ref.double() + 0.1 * torch.randn(T, generator=g, device=DEV,
                                                 dtype=torch.float64)).float()
    adv = torch.randn(T, generator=g, device=DEV)
    params = oracle_params((0.5, 2.0), (0.2, 0.2), "mask_weight", "const", 1.0)
    ref = run_oracle(z, ids, lp_mu, lp_ref, adv, mask, None, params, want_dlogits=not fwd_only)
    out = _outside(buf, off, T, ld, V)
    if fwd_only:
        res = P.decoupled_ppo_loss_fwd_bwd(z, ids, lp_mu, lp_ref, adv, mask, want_dlogits=False,
                                           scale_mode="const")
        torch.cuda.synchronize()
        compare_loss(res, ref, params, tdt, check_dlogits=False)
        assert torch.equal(buf.view(torch.int16) if dtype == "bf16" else buf, ref_buf.view(torch.int16) if dtype == "bf16" else ref_buf)
        return
    if in_place:
        res = P.decoupled_ppo_loss_fwd_bwd(z, ids, lp_mu, lp_ref, adv, mask, dlogits=z,
                                           scale_mode="const")
        torch.cuda.synchronize()
        compare_loss(res, ref, params, tdt)
        a, b = buf[out], ref_buf[out]
    else:
        dbuf = torch.full_like(buf, SENTINEL)
        d = dbuf[off:off + T * ld].view(T, ld)[:, :V]
        res = P.decoupled_ppo_loss_fwd_bwd(z, ids, lp_mu, lp_ref, adv, mask, dlogits=d,
                                           scale_mode="const")
        torch.cuda.synchronize()
        compare_loss(res, ref, params, tdt)
        a, b = dbuf[out], torch.full_like(dbuf[out], SENTINEL)
    if dtype == "bf16":
        a, b = a.view(torch.int16), b.view(torch.int16)
    assert torch.equal(a, b), "entries outside the rows were written"
