"""GPU parity of logprob_fwd and ewma_proxy_update (through the C ABI) against the oracle."""
import numpy as np
import pytest
import torch

import oracle
import paper_2605_12070_amd as P
from paper_2605_12070_amd import workloads as W

from helpers import TIGHT, assert_close_rel, bits_of, rtol_for

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _say(*a):
    print("[case]", *a, flush=True)


@pytest.mark.parametrize("name,T,V", [("tiny", None, None), ("small_vocab", 512, None),
                                      ("large_vocab", 48, None)])
@pytest.mark.parametrize("policy", ["auto", "stream"])
def test_logprob_workloads(name, T, V, policy):
    _say("logprob", name, T, V, policy)
    wl = W.make_workload(name, device=DEV, T=T, V=V, seq_len=8 if name == "large_vocab" else None)
    P.set_path_policy(policy)
    try:
        lp, lse = P.logprob_fwd(wl.logits, wl.ids, with_lse=True)
        torch.cuda.synchronize()
    finally:
        P.set_path_policy("auto")
    ref_lp, ref_lse = oracle.logprob_fwd(bits_of(wl.logits), wl.ids.cpu().numpy())
    rt = rtol_for(wl.logits.dtype)
    for got, ref, what in ((lp, ref_lp, "lp"), (lse, ref_lse, "lse")):
        g = got.cpu().double().numpy()
        assert_close_rel(g, ref, rt, what)
        assert_close_rel(g, ref, TIGHT, what + " (tight)")


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_logprob_bad_ids_and_shapes(dtype):
    for V in (1, 3, 1025, 151936):
        _say("logprob shapes", dtype, V)
        T = 5
        g = torch.Generator(device=DEV).manual_seed(V)
        z = (torch.randn(T, V, generator=g, device=DEV) * 4).to(dtype)
        ids = torch.tensor([0, V - 1, V, -1, V // 2], device=DEV)
        lp, lse = P.logprob_fwd(z, ids, with_lse=True)
        torch.cuda.synchronize()
        ref_lp, ref_lse = oracle.logprob_fwd(bits_of(z), ids.cpu().numpy())
        assert_close_rel(lp.cpu().double().numpy(), ref_lp, TIGHT, "lp")
        assert_close_rel(lse.cpu().double().numpy(), ref_lse, TIGHT, "lse")
        assert np.isnan(lp[2].item()) and np.isnan(lp[3].item())


def test_logprob_one_hot_rows():
    # a single dominant logit: log pi = -log(1 + (V-1) e^-40) ~ 0, well conditioned
    V = 151936
    z = torch.zeros(4, V, device=DEV, dtype=torch.bfloat16)
    z[:, 1234] = 40.0
    ids = torch.full((4,), 1234, device=DEV)
    lp = P.logprob_fwd(z, ids)
    torch.cuda.synchronize()
    ref, _ = oracle.logprob_fwd(bits_of(z), ids.cpu().numpy())
    assert np.all(np.abs(lp.cpu().double().numpy() - ref) < 1e-6)


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("n", [1, 5, 8, 1000, (1 << 20) + 3])
def test_ewma_normalized_recursion(dtype, n):
    _say("ewma normalized", dtype, n)
    g = torch.Generator(device=DEV).manual_seed(n)
    hist = [torch.randn(n, generator=g, device=DEV).to(dtype) for _ in range(6)]
    beta = 0.75
    x = torch.full((n,), float("nan"), device=DEV, dtype=dtype)   # first step must not read it
    w = 0.0
    x_ref, w_ref = np.full(n, np.nan), 0.0
    for t, th in enumerate(hist):
        reset = t == 4
        w = P.ewma_proxy_update(x, th, beta, w, reset=reset)
        if reset:
            x_ref, w_ref = bits_of(th), oracle.ewma_reset()
        else:
            x_ref, w_ref = oracle.ewma_normalized_step(x_ref, bits_of(th), beta, w_ref)
        # the stored value is the float32 result rounded to the buffer's dtype
        tol = 2.0 ** -8 if dtype == torch.bfloat16 else 2e-6
        got = bits_of(x)
        np.testing.assert_allclose(got, x_ref, rtol=tol * (t + 1), atol=tol * (t + 1))
        assert abs(w - w_ref) < 1e-12
    # the closed form of Eq. 5 from the reset point on (fp32 only: no rounding per step)
    if dtype == torch.float32:
        cf = oracle.ewma_closed_form([bits_of(h) for h in hist[4:]], beta)
        np.testing.assert_allclose(bits_of(x), cf, rtol=1e-5, atol=1e-5)


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_ewma_fixed_and_unaligned(dtype):
    n = 4099
    _say("ewma fixed unaligned", dtype, n)
    g = torch.Generator(device=DEV).manual_seed(1)
    xb = torch.randn(n + 1, generator=g, device=DEV).to(dtype)
    nb = torch.randn(n + 1, generator=g, device=DEV).to(dtype)
    x, xn = xb[1:], nb[1:]                    # misaligned base pointers
    x0 = bits_of(x)
    P.ewma_proxy_update(x, xn, 0.9, normalized=False)
    torch.cuda.synchronize()
    ref = oracle.ewma_fixed_step(x0, bits_of(xn), 0.9)
    tol = 2.0 ** -8 if dtype == torch.bfloat16 else 2e-6
    np.testing.assert_allclose(bits_of(x), ref, rtol=tol, atol=tol)
    assert bits_of(xb[:1]).tolist() == bits_of(torch.randn(n + 1, generator=torch.Generator(
        device=DEV).manual_seed(1), device=DEV).to(dtype)[:1]).tolist()


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("n", [1, 7, 9, 4099, 65536 * 8 + 5])
def test_ewma_leaves_the_rest_of_the_allocation_alone(dtype, n):
    """Vector threads and tail threads write exactly [0, n): guards after the end keep
    their bits (the buffers are slices of larger allocations with 16-byte-aligned bases)."""
    _say("ewma guards", dtype, n)
    g = torch.Generator(device=DEV).manual_seed(7)
    xb = torch.randn(n + 40, generator=g, device=DEV).to(dtype)
    nb = torch.randn(n + 40, generator=g, device=DEV).to(dtype)
    before = bits_of(xb)
    P.ewma_proxy_update(xb[:n], nb[:n], 0.5, w=1.0)
    torch.cuda.synchronize()
    after = bits_of(xb)
    assert np.array_equal(after[n:], before[n:])
    ref, _ = oracle.ewma_normalized_step(before[:n], bits_of(nb[:n]), 0.5, 1.0)
    tol = 2.0 ** -8 if dtype == torch.bfloat16 else 2e-6
    np.testing.assert_allclose(after[:n], ref, rtol=tol, atol=tol)


def test_ewma_controller_resets_on_low_rho():
    n = 64
    x0 = torch.zeros(n, device=DEV)
    ctl = P.EwmaProxy(x0, beta=0.75, tau=0.9, patience=2)
    hist = [torch.full((n,), float(k + 1), device=DEV) for k in range(6)]
    healthy = [100, 99, 99, 95, 0]        # rho = 0.95
    collapsed = [100, 80, 90, 70, 0]      # rho = 0.70
    fired = [ctl.step(hist[0], healthy), ctl.step(hist[1], collapsed),
             ctl.step(hist[2], collapsed), ctl.step(hist[3], healthy)]
    torch.cuda.synchronize()
    assert fired == [False, False, True, False]
    assert oracle.reset_schedule([0.95, 0.7, 0.7, 0.95], 0.9, 2) == fired
    # after the reset at step 3 (value 3) and one more step (value 4): closed form
    cf = oracle.ewma_closed_form([np.full(n, 3.0), np.full(n, 4.0)], 0.75)
    np.testing.assert_allclose(ctl.x.cpu().numpy(), cf, rtol=1e-6)
    assert ctl.resets == 1 and abs(ctl.w - 1.75) < 1e-12


@pytest.mark.parametrize("dtype,V,K,policy", [
    (torch.bfloat16, 1000, 3, "auto"),          # ragged V: streaming kernel
    (torch.bfloat16, 151936, 2, "auto"),        # register-resident persistent kernel
    (torch.bfloat16, 32000, 4, "stream"),
    (torch.float32, 4096, 4, "auto"),           # fp32 resident kernel
])
def test_logprob_versioned(dtype, V, K, policy):
    """Each token reads the logits of its own policy version; unknown versions give NaN."""
    T = 150
    _say("logprob versioned", dtype, V, K, policy)
    g = torch.Generator(device=DEV).manual_seed(V + K)
    zs = [(3.0 * torch.randn(T, V, generator=g, device=DEV)).to(dtype) for _ in range(K)]
    ids = torch.randint(0, V, (T,), generator=g, device=DEV)
    ver = torch.randint(0, K, (T,), generator=g, device=DEV, dtype=torch.int32)
    ver[:4] = torch.tensor([-1, K, 99, -7], dtype=torch.int32, device=DEV)
    ids[5] = V + 1                               # bad id on a good version
    P.set_path_policy(policy)
    try:
        lp, lse = P.logprob_fwd_versioned(zs, ver, ids, with_lse=True)
        torch.cuda.synchronize()
    finally:
        P.set_path_policy("auto")
    ref = oracle.versioned_logprob([bits_of(z) for z in zs], ver.cpu().numpy(), ids.cpu().numpy())
    got = lp.cpu().double().numpy()
    bad = np.array([0, 1, 2, 3, 5])
    assert np.isnan(got[bad]).all() and np.isnan(ref[bad]).all()
    assert np.isfinite(got[4]) and np.isfinite(ref[4])
    ok = ~np.isnan(ref)
    err = np.abs(got[ok] - ref[ok]) / np.maximum(np.abs(ref[ok]), 1.0)
    assert err.max() < 2e-5, err.max()


def test_ewma_parameter_sized_buffer():
    """The PPO-EWMA update at the benchmark's parameter-sized shape (n = 2^30 fp32, normalised
    form): the first step copies, the second and third follow the recursion of App. B.
    Sampled elements (2^20 random ones plus both ends) are compared with the oracle's
    recursion; on every element, the result lies between the old value and the new one
    (a convex combination), which any misplaced read or write would break."""
    n = 1 << 30
    print(f"[case] ewma parameter-sized n={n}", flush=True)
    g = torch.Generator(device=DEV).manual_seed(30)
    hist = [torch.randn(n, generator=g, device=DEV) for _ in range(3)]
    x = torch.empty(n, device=DEV)
    beta = P.beta_from_window(6)
    rng = np.random.default_rng(30)
    idx = np.unique(np.concatenate([rng.integers(0, n, 1 << 20), [0, 1, n - 2, n - 1]]))
    it = torch.as_tensor(idx, device=DEV)
    w, w_ref, x_ref = 0.0, 0.0, None
    for t, th in enumerate(hist):
        prev = x.clone() if t > 0 else None
        w = P.ewma_proxy_update(x, th, beta, w)
        x_ref, w_ref = oracle.ewma_normalized_step(x_ref, th[it].cpu().double().numpy(), beta,
                                                   w_ref)
        torch.cuda.synchronize()
        assert abs(w - w_ref) < 1e-12
        np.testing.assert_allclose(x[it].cpu().double().numpy(), x_ref, rtol=2e-6 * (t + 1),
                                   atol=2e-6 * (t + 1))
        if prev is None:
            assert torch.equal(x, th)
        else:
            for a in range(0, n, 1 << 28):
                lo = torch.minimum(prev[a:a + (1 << 28)], th[a:a + (1 << 28)])
                hi = torch.maximum(prev[a:a + (1 << 28)], th[a:a + (1 << 28)])
                xs = x[a:a + (1 << 28)]
                slack = 1e-6 * torch.maximum(lo.abs(), hi.abs())
                assert torch.all((xs >= lo - slack) & (xs <= hi + slack))
            del prev
