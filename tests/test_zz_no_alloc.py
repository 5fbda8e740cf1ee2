"""GPU test of fused_lm_head_loss_fwd_bwd_noalloc, the entry point that allocates nothing
(its workspace is the library's static per-device scratch), called through the C ABI.

Two calls in a row on one device, the second with a smaller input: a chunked call (T = 4096,
V = 151936, whose one-pass workspace does not fit the 64 MiB scratch) and then a one-pass
call. Each is compared bit for bit with fused_lm_head_loss_fwd_bwd run with a workspace
of its own and the vocab_chunk the no-allocation call reports (same kernels, same order).
"""
import ctypes as C

import numpy as np
import pytest
import torch

import paper_2605_12070_amd as P
from paper_2605_12070_amd import _lib
from paper_2605_12070_amd import workloads as W

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _inputs(T, d, V, seed):
    wl = W.make_lm_head_workload(DEV, T=T, d=d, V=V, seed=seed, seq_len=8, mask_frac=0.2,
                                 weight_std=0.1)
    wl.ids[5] = V + 2                                   # a bad id
    g = torch.Generator(device=DEV).manual_seed(seed)
    lp_ref = -5.0 + 0.5 * torch.randn(T, generator=g, device=DEV)
    lp_mu = lp_ref + 0.2 * torch.randn(T, generator=g, device=DEV)
    return wl, lp_mu, lp_ref


def _fields(res):
    return dict(logp=res.logp, loss_tok=res.loss_tok, loss=res.loss, flags=res.flags,
                stats=res.stats, dhidden=res.dhidden, dweight=res.dweight)


def _case(T, d, V, seed, expect_chunked):
    print(f"[case] noalloc T={T} d={d} V={V} seed={seed}", flush=True)
    wl, lp_mu, lp_ref = _inputs(T, d, V, seed)
    got, used = P.fused_lm_head_loss_fwd_bwd_noalloc(wl.hidden, wl.weight, wl.ids, lp_mu,
                                                     lp_ref, wl.adv, wl.mask)
    torch.cuda.synchronize()
    assert (used > 0) == expect_chunked, used
    ref = P.fused_lm_head_loss_fwd_bwd(wl.hidden, wl.weight, wl.ids, lp_mu, lp_ref, wl.adv,
                                       wl.mask, vocab_chunk=used)
    torch.cuda.synchronize()
    for name, a in _fields(got).items():
        b = _fields(ref)[name]
        assert torch.equal(a.view(torch.uint8) if a.dtype == torch.uint8 else a.view(torch.int32),
                           b.view(torch.uint8) if b.dtype == torch.uint8 else b.view(torch.int32)), name
    st = got.stats.cpu().numpy()
    assert st[0] == int(wl.mask.sum().item()) and st[4] == int(wl.mask[5].item())
    assert torch.isfinite(got.dweight).all() and torch.isfinite(got.dhidden).all()
    return used


def test_noalloc_matches_workspace_entry_point_twice():
    scratch = _lib.lib().fused_lm_head_noalloc_scratch_bytes()
    assert scratch == 64 << 20
    c1 = _case(4096, 256, 151936, seed=31, expect_chunked=True)
    assert P.lm_head_workspace_bytes(4096, 256, 151936, c1) <= scratch
    assert P.lm_head_workspace_bytes(4096, 256, 151936, c1 + 256) > scratch
    c2 = _case(300, 128, 5000, seed=32, expect_chunked=False)
    assert c2 == 0
