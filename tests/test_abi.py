"""Host-side checks of the C ABI: the library loads, exports every function that
include/dppo.h declares, and rejects bad arguments before touching the GPU."""
import ctypes as C
import os
import re

import pytest

from paper_2605_12070_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dppo.h")

pytestmark = pytest.mark.skipif(not os.path.exists(_lib.LIB_PATH),
                                reason="libdppo.so not built")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    src = re.sub(r"//[^\n]*", "", src)
    src = re.sub(r"#[^\n]*", "", src)
    names = []
    for stmt in src.split(";"):
        stmt = " ".join(stmt.split())
        if "(" not in stmt or stmt.startswith("typedef") or "{" in stmt:
            continue
        m = re.search(r"(\w+)\s*\(", stmt)
        if m:
            names.append(m.group(1))
    return names


def test_header_declares_the_boundary():
    names = declared_functions()
    for required in ("logprob_fwd", "decoupled_ppo_loss_fwd_bwd", "ewma_proxy_update",
                     "dppo_strerror"):
        assert required in names
    assert set(names) == set(_lib.SIGNATURES), "binding signatures out of sync with the header"


def test_library_exports_every_declared_symbol():
    h = C.CDLL(_lib.LIB_PATH)
    for name in declared_functions():
        assert hasattr(h, name), name
    assert _lib.lib().dppo_abi_version() == _lib.ABI_VERSION


def test_strerror():
    L = _lib.lib()
    assert L.dppo_strerror(0) == b"success"
    assert b"invalid" in L.dppo_strerror(1)
    assert L.dppo_strerror(99) == b"unknown status"


FAKE = 0x10000  # never dereferenced: every case below fails its host-side check first


def _params(**kw):
    d = dict(band_lo=0.5, band_hi=2.0, clip_eps_lo=0.2, clip_eps_hi=0.2, rd_mode=3,
             scale_mode=1, loss_scale=1.0)
    d.update(kw)
    return _lib.DppoParams(**d)


def _loss(T=4, V=8, ld=8, dtype=1, p=None, dl=None, ldd=8, ids=FAKE, logits=FAKE, stats=FAKE,
          loss=FAKE, ref=FAKE):
    p = p or _params()
    L = _lib.lib()
    return L.decoupled_ppo_loss_fwd_bwd(logits, dtype, T, V, ld, ids, FAKE, ref, FAKE, None,
                                        None, C.byref(p), FAKE, FAKE, loss, None, dl, ldd,
                                        stats, None)


@pytest.mark.parametrize("kw,frag", [
    (dict(dtype=7), "dtype"),
    (dict(T=-1), "T ="),
    (dict(V=0), "V ="),
    (dict(ld=4), "stride"),
    (dict(ids=None), "required"),
    (dict(logits=None), "NULL"),
    (dict(stats=None), "required"),
    (dict(loss=None), "required"),
    (dict(p=_params(band_lo=3.0)), "band"),
    (dict(p=_params(band_lo=float("nan"))), "band"),
    (dict(p=_params(band_lo=-0.5)), "band"),
    (dict(p=_params(clip_eps_lo=-0.1)), "clip"),
    (dict(p=_params(clip_eps_hi=float("inf"))), "clip"),
    (dict(p=_params(loss_scale=float("nan"))), "loss_scale"),
    (dict(p=_params(rd_mode=9)), "rd_mode"),
    (dict(p=_params(scale_mode=5)), "scale_mode"),
    (dict(p=_params(ref_mode=3, alpha=0.5)), "ref_mode"),
    (dict(p=_params(ref_mode=1, alpha=0.0)), "alpha"),
    (dict(p=_params(ref_mode=2, alpha=1.0)), "alpha"),
    (dict(p=_params(ref_mode=1, alpha=float("nan"))), "alpha"),
    (dict(ref=None), "logp_ref is required"),
    (dict(dl=FAKE + 2 * 8, ldd=8), "overlaps"),        # dlogits overlaps logits, not equal
    (dict(dl=FAKE, ldd=16, ld=8), "overlaps"),          # same base, different stride
    (dict(dl=FAKE + 64, ldd=4), "stride"),
])
def test_loss_rejects_bad_arguments(kw, frag):
    st = _loss(**kw)
    assert st == _lib.DPPO_ERR_INVALID_ARG
    assert frag in _lib.lib().dppo_last_error().decode()


def test_loss_null_params():
    L = _lib.lib()
    st = L.decoupled_ppo_loss_fwd_bwd(FAKE, 1, 4, 8, 8, FAKE, FAKE, FAKE, FAKE, None, None,
                                      None, FAKE, FAKE, FAKE, None, None, 0, FAKE, None)
    assert st == _lib.DPPO_ERR_INVALID_ARG


@pytest.mark.parametrize("args,frag", [
    ((FAKE, 5, 4, 8, 8, FAKE, FAKE, None, None), "dtype"),
    ((FAKE, 1, 4, 8, 7, FAKE, FAKE, None, None), "stride"),
    ((FAKE, 1, 4, 8, 8, None, FAKE, None, None), "required"),
    ((FAKE, 1, 4, 8, 8, FAKE, None, None, None), "required"),
    ((FAKE, 1, 1 << 31, 8, 8, FAKE, FAKE, None, None), "T ="),
])
def test_logprob_rejects_bad_arguments(args, frag):
    st = _lib.lib().logprob_fwd(*args)
    assert st == _lib.DPPO_ERR_INVALID_ARG
    assert frag in _lib.lib().dppo_last_error().decode()


def test_logprob_empty_batch_is_a_no_op():
    # T = 0 enqueues nothing, so it is safe without a GPU
    assert _lib.lib().logprob_fwd(None, 1, 0, 8, 8, None, None, None, None) == _lib.DPPO_OK


@pytest.mark.parametrize("kw,frag", [
    (dict(dtype=3), "dtype"),
    (dict(n=-1), "n ="),
    (dict(beta=1.0), "beta"),
    (dict(beta=-0.1), "beta"),
    (dict(beta=float("nan")), "beta"),
    (dict(xp=None), "required"),
    (dict(w=None), "w is required"),
    (dict(w=-1.0), "w_{t-1}"),
    (dict(xn=FAKE + 8), "overlaps"),
])
def test_ewma_rejects_bad_arguments(kw, frag):
    d = dict(xp=FAKE, xn=FAKE + 4096, dtype=0, n=16, beta=0.5, w=0.0, reset=0, normalized=1)
    d.update(kw)
    wref = None if d["w"] is None else C.byref(C.c_double(d["w"]))
    st = _lib.lib().ewma_proxy_update(d["xp"], d["xn"], d["dtype"], d["n"], d["beta"], wref,
                                      d["reset"], d["normalized"], None)
    assert st == _lib.DPPO_ERR_INVALID_ARG
    assert frag in _lib.lib().dppo_last_error().decode()


@pytest.mark.parametrize("kw,frag", [
    (dict(dtype=3), "dtype"),
    (dict(n=-1), "n ="),
    (dict(beta=1.0), "beta"),
    (dict(beta=float("nan")), "beta"),
    (dict(tau=float("inf")), "tau"),
    (dict(tau=float("nan")), "tau"),
    (dict(patience=0), "patience"),
    (dict(state=None), "state is required"),
    (dict(state=FAKE + 65536 + 4), "8-byte aligned"),
    (dict(xp=None), "required"),
    (dict(xn=FAKE + 8), "overlaps"),
    (dict(state=FAKE + 32), "state overlaps"),
])
def test_ewma_step_rejects_bad_arguments(kw, frag):
    """The device-side step checks its host arguments before any launch (the normaliser
    itself lives on the device and is checked there)."""
    d = dict(xp=FAKE, xn=FAKE + 4096, dtype=0, n=16, beta=0.5, tau=0.9, patience=1,
             normalized=1, stats=None, state=FAKE + 65536)
    d.update(kw)
    st = _lib.lib().ewma_proxy_step(d["xp"], d["xn"], d["dtype"], d["n"], d["beta"], d["tau"],
                                    d["patience"], d["normalized"], d["stats"], d["state"], None)
    assert st == _lib.DPPO_ERR_INVALID_ARG
    assert frag in _lib.lib().dppo_last_error().decode()


def test_ewma_state_layout():
    """dppo_ewma_state is 40 bytes with the normaliser first (the binding writes it)."""
    assert C.sizeof(_lib.DppoEwmaState) == 40
    assert _lib.DppoEwmaState.w.offset == 0 and _lib.DppoEwmaState.last_rho.offset == 24
    assert _lib.DppoEwmaState.cb.offset == 32


def test_ewma_empty_buffer_updates_w_only():
    w = C.c_double(0.0)
    L = _lib.lib()
    assert L.ewma_proxy_update(None, None, 0, 0, 0.5, C.byref(w), 0, 1, None) == _lib.DPPO_OK
    assert w.value == 1.0
    assert L.ewma_proxy_update(None, None, 0, 0, 0.5, C.byref(w), 0, 1, None) == _lib.DPPO_OK
    assert w.value == 1.5
    assert L.ewma_proxy_update(None, None, 0, 0, 0.5, C.byref(w), 1, 1, None) == _lib.DPPO_OK
    assert w.value == 1.0


def test_path_policy_validation():
    L = _lib.lib()
    for bad in (-1, 4, 7):
        assert L.dppo_set_path_policy(bad) == _lib.DPPO_ERR_INVALID_ARG
    for ok in (3, 2, 1, 0):
        assert L.dppo_set_path_policy(ok) == _lib.DPPO_OK


def test_timer_read_requires_outputs():
    assert _lib.lib().dppo_timer_read(None, None) == _lib.DPPO_ERR_INVALID_ARG


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(_lib, "_lib", None)
    monkeypatch.setattr(_lib, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(RuntimeError, match="no CPU fallback"):
        _lib.lib()


def test_host_controller_logic():
    import paper_2605_12070_amd as P
    assert P.beta_from_window(6) == 0.75 and P.beta_from_window(2) == 0.5
    assert P.train_infer_mask_value([10, 9, 9, 8, 0]) == 0.8
    assert P.train_infer_mask_value([0, 0, 0, 0, 0]) == 1.0
    assert abs(P.ppo_clip_ratio([10, 9, 7, 6, 0]) - 0.3) < 1e-12
    assert P.ppo_clip_ratio([0, 0, 0, 0, 0]) == 0.0


def test_host_controller_exports_match_the_oracle():
    """The a9 arithmetic lives in the library (dppo_beta_from_window, dppo_*_value,
    dppo_reset_decision), called here through ctypes on the CPU, against the oracle's
    definitions: beta = W / (W + 2) with centre of mass W / 2 (App. B), rho_t and the clip
    ratio from the counters, and the reset schedule over seeded rho sequences (Sec. 5.2;
    App. E) for several patiences and thresholds."""
    import numpy as np
    from oracle import dppo_oracle as oracle
    L = _lib.lib()
    out = C.c_double(0.0)
    for W in (0.0, 0.5, 1, 2, 3, 6, 10, 1e6):
        assert L.dppo_beta_from_window(float(W), C.byref(out)) == _lib.DPPO_OK
        assert out.value == oracle.beta_from_window(W)
        if W > 0:
            assert abs(oracle.ewma_center_of_mass(out.value) - W / 2) <= 1e-9 * max(1.0, W)
    for bad in (-1.0, float("inf"), float("nan")):
        assert L.dppo_beta_from_window(bad, C.byref(out)) == _lib.DPPO_ERR_INVALID_ARG
    assert L.dppo_beta_from_window(1.0, None) == _lib.DPPO_ERR_INVALID_ARG

    rng = np.random.default_rng(11)
    for _ in range(200):
        nv = int(rng.integers(0, 5000))
        nb, np_ = (int(rng.integers(0, nv + 1)) for _ in range(2))
        na = int(rng.integers(0, min(nb, np_) + 1))
        st = [nv, nb, np_, na, int(rng.integers(0, 3))]
        arr = (C.c_int32 * 5)(*st)
        assert L.dppo_train_infer_mask_value(arr, C.byref(out)) == _lib.DPPO_OK
        assert out.value == oracle.train_infer_mask_value(st)
        assert L.dppo_ppo_clip_ratio(arr, C.byref(out)) == _lib.DPPO_OK
        assert out.value == oracle.ppo_clip_ratio(st)

    for tau, patience, seed in ((0.9, 1, 0), (0.9, 2, 1), (0.8, 3, 2), (0.95, 1, 3)):
        r = np.random.default_rng(seed)
        n_valid = 1000
        actives = r.integers(700, 1001, size=60)
        stats = [[n_valid, n_valid, n_valid, int(a), 0] for a in actives]
        stats[7] = [0, 0, 0, 0, 0]                       # no valid token: rho = 1
        rhos = [oracle.train_infer_mask_value(s) for s in stats]
        want = oracle.reset_schedule(rhos, tau=tau, patience=patience)
        streak = C.c_int32(0)
        rho = C.c_double(0.0)
        fire = C.c_int32(0)
        got = []
        for s_, rho_want in zip(stats, rhos):
            arr = (C.c_int32 * 5)(*s_)
            assert L.dppo_reset_decision(arr, tau, patience, C.byref(streak), C.byref(rho),
                                         C.byref(fire)) == _lib.DPPO_OK
            assert rho.value == rho_want
            got.append(bool(fire.value))
        assert got == list(want), (tau, patience)
        assert any(want) and not all(want)
    # stats = NULL: no decision input, as in ewma_proxy_step: no reset, streak unchanged
    streak = C.c_int32(3)
    assert L.dppo_reset_decision(None, 0.9, 5, C.byref(streak), None, C.byref(fire)) == _lib.DPPO_OK
    assert fire.value == 0 and streak.value == 3
    arr = (C.c_int32 * 5)(10, 10, 10, 1, 0)
    for kw in (dict(tau=float("nan")), dict(patience=0), dict(streak=-1)):
        a = dict(tau=0.9, patience=1, streak=0)
        a.update(kw)
        sk = C.c_int32(a["streak"])
        assert L.dppo_reset_decision(arr, a["tau"], a["patience"], C.byref(sk), None,
                                     C.byref(fire)) == _lib.DPPO_ERR_INVALID_ARG


def test_host_ewma_proxy_decisions_follow_the_library(monkeypatch):
    """EwmaProxy.decide_reset keeps only the streak and passes the counters through: its
    decisions equal the oracle's schedule (no GPU: the buffer update is not called)."""
    import paper_2605_12070_amd as P
    from oracle import dppo_oracle as oracle

    class _NoBuf:
        def clone(self):
            return self

    px = P.EwmaProxy(_NoBuf(), beta=0.75, tau=0.9, patience=2)
    stats = [[100, 100, 100, a, 0] for a in (95, 85, 80, 99, 70, 60, 50, 91, 89, 88)]
    want = oracle.reset_schedule([oracle.train_infer_mask_value(s) for s in stats], 0.9, 2)
    got = [px.decide_reset(s) for s in stats]
    assert got == list(want)
    assert px.last_rho == 0.88


def test_row_kernel_name_follows_the_selection_rule():
    """Host-only query: the resident kernel while a row fits NT x NC 16-byte chunks (at most
    1024 x 19 x 8 = 155648 bf16 elements) with whole chunks; bf16 rows that are unaligned or
    ragged use the phase kernels while the chunks they touch (ceil((V + 7) / 8), or ceil(V / 8)
    on an aligned stride) fit; beyond, the resident-prefix kernel for aligned rows with
    dlogits, the streaming kernel otherwise."""
    import torch
    from paper_2605_12070_amd import row_kernel_name
    bf, f32 = torch.bfloat16, torch.float32
    assert row_kernel_name(bf, 151936) == "dppo::rows_bf16_resident<1024, 19, true>"
    assert row_kernel_name(bf, 155648) == "dppo::rows_bf16_resident<1024, 19, true>"
    # longer bf16 rows with dlogits: a resident prefix and a streamed tail
    assert row_kernel_name(bf, 155656) == "dppo::rows_bf16_prefix<1024, 19>"
    assert row_kernel_name(bf, 155649, ld=155656) == "dppo::rows_bf16_prefix<1024, 19>"
    assert row_kernel_name(bf, 262144) == "dppo::rows_bf16_prefix<1024, 19>"
    assert row_kernel_name(bf, 155649).endswith("true, false>")             # unaligned stride
    assert row_kernel_name(bf, 262144, with_dlogits=False).startswith("dppo::rows_stream<unsigned short, 1024, false")
    assert row_kernel_name(bf, 151936, with_dlogits=False) == "dppo::rows_bf16_fwd<1024, 19>"
    assert row_kernel_name(f32, 32000, with_dlogits=False) == "dppo::rows_f32_resident<1024, 8, false>"
    assert row_kernel_name(bf, 2048) == "dppo::rows_bf16_resident<256, 1, true>"
    assert row_kernel_name(bf, 77825) == "dppo::rows_bf16_phase<1024, 12, true>"  # ragged
    assert row_kernel_name(bf, 64, ld=68) == "dppo::rows_bf16_phase<256, 1, true>"  # unaligned
    assert row_kernel_name(bf, 50257) == "dppo::rows_bf16_phase_db<1024, 8>"
    assert row_kernel_name(bf, 50257, with_dlogits=False) == "dppo::rows_bf16_fwd_phase<1024, 8>"
    assert row_kernel_name(bf, 151665, ld=151936) == "dppo::rows_bf16_phase<1024, 19, true>"
    assert row_kernel_name(bf, 155647, ld=155648) == "dppo::rows_bf16_phase<1024, 19, true>"
    assert row_kernel_name(bf, 155641) == "dppo::rows_bf16_phase<1024, 19, true>"
    assert row_kernel_name(bf, 155642).startswith("dppo::rows_stream")     # up to 7 more chunks
    assert row_kernel_name(f32, 32000) == "dppo::rows_f32_resident<1024, 8, true>"
    # fp32 rows past the resident kernels: a resident prefix and a streamed tail when the
    # row holds at least the prefix's 1024 x 19 whole chunks; otherwise the streaming kernel
    assert row_kernel_name(f32, 151936) == "dppo::rows_f32_prefix<1024, 19>"
    assert row_kernel_name(f32, 77825, ld=77828) == "dppo::rows_f32_prefix<1024, 19>"
    assert row_kernel_name(f32, 77825).endswith("true, false>")            # unaligned stride
    assert row_kernel_name(f32, 77823).startswith("dppo::rows_stream<float")
    assert row_kernel_name(f32, 151936, with_dlogits=False).startswith("dppo::rows_stream<float")
    # two row buffers for the bf16 backward shapes 512 x 4 .. 1024 x 8 only
    assert row_kernel_name(bf, 32000) == "dppo::rows_bf16_resident_db<512, 8>"
    assert row_kernel_name(bf, 65536) == "dppo::rows_bf16_resident_db<1024, 8>"
    assert row_kernel_name(bf, 98000) == "dppo::rows_bf16_resident<1024, 12, true>"
    assert row_kernel_name(bf, 8192) == "dppo::rows_bf16_resident<256, 4, true>"
    assert row_kernel_name(bf, 32000, with_dlogits=False) == "dppo::rows_bf16_fwd<512, 8>"
    L = _lib.lib()
    assert L.dppo_row_kernel_name(7, 100, 100, 1) is None
    assert L.dppo_row_kernel_name(1, 0, 0, 1) is None
    assert L.dppo_row_kernel_name(1, 100, 99, 1) is None


# ---------------------------------------------------------------------- effective thresholds
GOLDEN4 = os.path.join(ROOT, "tests", "golden", "table4_effective_thresholds.csv")


def _table4():
    import csv
    with open(GOLDEN4) as f:
        return list(csv.DictReader(l for l in f if not l.startswith("#")))


@pytest.mark.parametrize("row", _table4(), ids=lambda r: f"{r['mask_lo']}-{r['clip_hi']}-n{r['n']}-{r['kind']}")
def test_effective_thresholds_match_table4(row):
    """The library's host helper reproduces every printed entry of Table 4 (App. A)."""
    from paper_2605_12070_amd import effective_thresholds
    alpha = 1.0 / (int(row["n"]) + 1)
    m, c = effective_thresholds((float(row["mask_lo"]), float(row["mask_hi"])),
                                (float(row["clip_lo"]), float(row["clip_hi"])), alpha, row["kind"])
    want = [float(row[k]) for k in ("eff_mask_lo", "eff_mask_hi", "eff_clip_lo", "eff_clip_hi")]
    for g, w in zip([*m, *c], want):
        assert abs(g - w) <= 0.5e-4 + 1e-12, (g, w)


@pytest.mark.parametrize("kind", ["log_linear", "linear"])
def test_effective_thresholds_match_the_oracle(kind):
    import numpy as np
    import oracle
    from paper_2605_12070_amd import effective_thresholds
    rng = np.random.default_rng(3)
    for _ in range(200):
        alpha = rng.uniform(0.05, 0.95)
        m_lo, m_hi = np.sort(rng.uniform(0.3, 2.0, size=2))
        c_lo, c_hi = rng.uniform(0.5, 1.0), rng.uniform(1.0, 1.0 / (1.0 - alpha) - 1e-3)
        got = effective_thresholds((m_lo, m_hi), (c_lo, c_hi), alpha, kind)
        ref = oracle.effective_thresholds(m_lo, m_hi, c_lo, c_hi, alpha, kind)
        np.testing.assert_allclose(np.array(got).ravel(), np.array(ref).ravel(), rtol=1e-12)


def test_linear_clip_bound_beyond_reach_is_infinite():
    """With pi_ref = alpha mu + (1 - alpha) pi_theta, r_s = r / (alpha + (1 - alpha) r) never
    exceeds 1 / (1 - alpha): a clip bound at or above that never binds."""
    import numpy as np
    from paper_2605_12070_amd import effective_thresholds
    alpha = 0.25
    (_, _), (lo, hi) = effective_thresholds((0.5, 2.0), (0.9, 1.0 / (1 - alpha)), alpha, "linear")
    assert hi == float("inf") and np.isfinite(lo)
    r = np.logspace(-6, 6, 1001)
    assert np.all(r / (alpha + (1 - alpha) * r) <= 1.0 / (1 - alpha))


@pytest.mark.parametrize("args,frag", [
    ((0.9, 1.1, 0.8, 1.2, 0.5, 0), "not an interpolated"),
    ((0.9, 1.1, 0.8, 1.2, 0.5, 7), "not an interpolated"),
    ((0.9, 1.1, 0.8, 1.2, 0.0, 1), "alpha"),
    ((0.9, 1.1, 0.8, 1.2, 1.0, 2), "alpha"),
    ((1.2, 1.1, 0.8, 1.2, 0.5, 1), "bounds"),
    ((0.9, 1.1, -0.1, 1.2, 0.5, 2), "bounds"),
])
def test_effective_thresholds_reject_bad_arguments(args, frag):
    out = (C.c_double * 4)()
    assert _lib.lib().dppo_effective_thresholds(*args, out) == _lib.DPPO_ERR_INVALID_ARG
    assert frag in _lib.lib().dppo_last_error().decode()
    assert _lib.lib().dppo_effective_thresholds(0.9, 1.1, 0.8, 1.2, 0.5, 1, None) == \
        _lib.DPPO_ERR_INVALID_ARG


# ---------------------------------------------------------------------- fused LM head
def _lmh(T=4, d=64, V=300, dtype=1, hidden=FAKE, weight=FAKE, ws=FAKE, wsb=1 << 40, p=None,
         loss=FAKE, stats=FAKE):
    p = p or _params()
    return _lib.lib().fused_lm_head_loss_fwd_bwd(
        hidden, weight, dtype, T, d, V, FAKE, FAKE, FAKE, FAKE, None, None, C.byref(p), FAKE,
        FAKE, loss, None, stats, None, None, 0, ws, wsb, None)


@pytest.mark.parametrize("kw,frag,code", [
    (dict(dtype=0), "bf16", 2),
    (dict(dtype=5), "dtype", 1),
    (dict(d=60), "multiple of 8", 1),
    (dict(d=0), "multiple of 8", 1),
    (dict(V=0), "V =", 1),
    (dict(T=-1), "T =", 1),
    (dict(hidden=None), "aligned", 1),
    (dict(weight=FAKE + 8), "aligned", 1),
    (dict(wsb=100), "workspace", 1),
    (dict(ws=FAKE + 16), "256-byte", 1),
    (dict(loss=None), "required", 1),
    (dict(p=_params(rd_mode=8)), "rd_mode", 1),
])
def test_lm_head_rejects_bad_arguments(kw, frag, code):
    assert _lmh(**kw) == code
    assert frag in _lib.lib().dppo_last_error().decode()


def test_lm_head_workspace_size():
    L = _lib.lib()
    T, d, V = 8192, 4096, 151936
    n = L.fused_lm_head_workspace_bytes(T, d, V, 0)
    # partial sums of at least ceil(V / 256) tiles per token, four per-token vectors, and a
    # bf16 gradient chunk covering all of V
    assert n >= -(-V // 256) * T * 8 + T * 13 + T * V * 2
    assert L.fused_lm_head_workspace_bytes(T, d, V, 16384) < n
    assert L.fused_lm_head_workspace_bytes(T, 4, V, 0) == -1
    assert L.fused_lm_head_workspace_bytes(-1, d, V, 0) == -1


@pytest.mark.parametrize("K,frag", [(0, "versions"), (9, "versions")])
def test_versioned_logprob_rejects_bad_k(K, frag):
    arr = (C.c_void_p * 9)(*([FAKE] * 9))
    st = _lib.lib().logprob_fwd_versioned(arr, K, 1, 4, 8, 8, FAKE, FAKE, FAKE, None, None)
    assert st == _lib.DPPO_ERR_INVALID_ARG
    assert frag in _lib.lib().dppo_last_error().decode()


def test_versioned_logprob_rejects_null_pointers():
    L = _lib.lib()
    arr = (C.c_void_p * 2)(FAKE, None)
    assert L.logprob_fwd_versioned(arr, 2, 1, 4, 8, 8, FAKE, FAKE, FAKE, None, None) == _lib.DPPO_ERR_INVALID_ARG
    arr = (C.c_void_p * 2)(FAKE, FAKE)
    assert L.logprob_fwd_versioned(arr, 2, 1, 4, 8, 8, None, FAKE, FAKE, None, None) == _lib.DPPO_ERR_INVALID_ARG
    assert L.logprob_fwd_versioned(None, 2, 1, 4, 8, 8, FAKE, FAKE, FAKE, None, None) == _lib.DPPO_ERR_INVALID_ARG
    # T = 0 is a no-op that touches nothing
    assert L.logprob_fwd_versioned(None, 1, 1, 0, 8, 8, None, None, None, None, None) == _lib.DPPO_OK


def test_bench_refuses_more_than_one_gpu():
    """bench.py measures one GPU: asked for more it exits with status 2 and says so, before it
    touches a device."""
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    p = subprocess.run([sys.executable, os.path.join(root, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=300, cwd=root)
    assert p.returncode == 2, (p.returncode, p.stderr[-500:])
    assert "one GPU only" in p.stderr and p.stdout == ""


def test_noalloc_rejects_sizes_beyond_its_scratch():
    """Host-side checks of the no-allocation LM head: sizes whose 256-row chunked workspace
    exceeds the static scratch are UNSUPPORTED, bad sizes INVALID_ARG, before any HIP call."""
    L = _lib.lib()
    p = _params()
    used = C.c_int64(-7)
    args = lambda T, V: (FAKE, FAKE, 1, T, 64, V, FAKE, FAKE, FAKE, FAKE, None, None, C.byref(p),
                         FAKE, FAKE, FAKE, None, FAKE, None, None, C.byref(used), None)
    assert L.fused_lm_head_loss_fwd_bwd_noalloc(*args(65536, 151936)) == _lib.DPPO_ERR_UNSUPPORTED
    assert b"scratch" in L.dppo_last_error()
    assert L.fused_lm_head_loss_fwd_bwd_noalloc(*args(-1, 100)) == _lib.DPPO_ERR_INVALID_ARG
    assert L.fused_lm_head_loss_fwd_bwd_noalloc(*args(16, (1 << 21) + 1)) == _lib.DPPO_ERR_INVALID_ARG
    assert used.value == -7

