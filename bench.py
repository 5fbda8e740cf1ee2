"""Benchmark of the fused log-prob + decoupled PPO loss stage on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload large_vocab] [--no-cpu-baseline]

A step is one pass of the whole loss stage over one batch: the fused kernel (valid-token
count, per-row log-sum-exp / ratios / decisions / loss / dlogits, loss sum), then the reset
controller reading the five stats and the PPO-EWMA update of the per-token proxy buffer,
both on the device (no device-to-host copy inside the step). Inputs are synthetic, seeded, and resident in HBM
before the timed region. Prints one JSON line.
"""
from __future__ import annotations

import argparse
import concurrent.futures as cf
import hashlib
import json
import os
import platform
import re
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import paper_2605_12070_amd as P  # noqa: E402
from paper_2605_12070_amd import workloads as W  # noqa: E402

METRIC = "tokens/sec for fused logprob+decoupled PPO loss fwd+bwd; % of peak HBM GB/s"
HBM_PEAK_GBPS = 8000.0          # MI355X HBM3E, AMD specification
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")
CSRC = os.path.join(ROOT, "paper_2605_12070_amd", "csrc")


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


KERNEL_SOURCES = ("dppo_device.h", "loss_stage.h", "token_math.h", "loss_stage.hip")
SHARD_SOURCES = ("dppo_device.h", "loss_stage.h", "token_math.h", "vocab_shard.h",
                 "vocab_shard.hip")
EWMA_SOURCES = ("dppo_device.h", "ewma.h", "ewma.hip")


def kernel_source_hash(names=KERNEL_SOURCES) -> str:
    """Hash of a kernel's device sources, comments and spacing aside: a stored HBM-traffic
    figure is reported only while it still describes the kernel being timed."""
    h = hashlib.sha256()
    for name in names:
        with open(os.path.join(CSRC, name)) as f:
            code = re.sub(r"/\*.*?\*/|//[^\n]*", "", f.read(), flags=re.S)   # comments
        h.update(name.encode() + " ".join(code.split()).encode())
    return h.hexdigest()[:16]


def recorded_traffic(key, names=KERNEL_SOURCES):
    """HBM bytes per launch from the committed FETCH_SIZE / WRITE_SIZE summary, or None when
    the kernel's sources (names) have changed since the counters were taken."""
    try:
        tr = json.load(open(TRAFFIC_FILE)).get(key)
    except (OSError, ValueError):
        return None
    if tr and tr.get("source_hash") == kernel_source_hash(names):
        return tr["bytes_per_launch"]
    return None


def anchor_logprob(logits, ids, chunk=1024):
    """Sampled-token log-probs from PyTorch (float32), only to synthesise lp_ref / lp_mu."""
    T = logits.shape[0]
    out = torch.empty(T, dtype=torch.float64, device=logits.device)
    for a in range(0, T, chunk):
        z = logits[a:a + chunk].float()
        out[a:a + chunk] = (z.gather(1, ids[a:a + chunk, None])[:, 0]
                            - torch.logsumexp(z, dim=1)).double()
    return out


def algorithmic_bytes(T, V, n_valid, esize, per_token):
    """Logits read once (valid rows), dlogits written once (all rows), per-token vectors."""
    return n_valid * V * esize + T * V * esize + T * per_token


def cpu_baseline(wl, lp_mu, lp_ref, rows, threads):
    """The float64 oracle on a fixed sample of rows, in a thread pool over row chunks."""
    import oracle
    mask = wl.mask.cpu().numpy()
    params = oracle.Params(0.5, 2.0, 0.2, 0.2, "mask_weight", "token_mean", 1.0)
    scale = oracle.batch_scale(mask, params)
    idx = torch.as_tensor(rows, device=wl.logits.device)
    z16 = (wl.logits if len(rows) == wl.T else wl.logits[idx]).cpu()
    if z16.dtype == torch.bfloat16:
        zb = z16.view(torch.int16).numpy().view(np.uint16)
        decode = oracle.bf16_bits_to_f64
    else:
        zb = z16.numpy()
        decode = oracle.as_f64
    ids = wl.ids[idx].cpu().numpy()
    mu = lp_mu[idx].cpu().double().numpy()
    ref = lp_ref[idx].cpu().double().numpy()
    adv = wl.adv[idx].cpu().double().numpy()
    m = mask[rows]
    chunk = 32
    jobs = [(a, min(len(rows), a + chunk)) for a in range(0, len(rows), chunk)]

    def work(ab):
        a, b = ab
        oracle.per_token(decode(zb[a:b]), ids[a:b], mu[a:b], ref[a:b], adv[a:b], m[a:b], None,
                         params, scale, want_dlogits=True)
        return b - a

    t0 = time.perf_counter()
    with cf.ThreadPoolExecutor(max_workers=threads) as ex:
        done = sum(ex.map(work, jobs))
    dt = time.perf_counter() - t0
    return done / dt, dt


def copy_bandwidth(dev, nbytes=2 << 30, reps=10):
    """Device-to-device copy rate (read + write bytes per second), a practical ceiling."""
    a = torch.empty(nbytes // 2, dtype=torch.bfloat16, device=dev)
    b = torch.empty_like(a)
    b.copy_(a)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        b.copy_(a)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    del a, b
    return 2 * nbytes / (ms * 1e-3) / 1e9


def ewma_bandwidth(dev, n, reps=20):
    """PPO-EWMA update of a parameter-sized fp32 buffer (normalised form: x_prox and x_new
    are read, x_prox written, 12 bytes per element), timed with events on the stream the
    library launches on (torch's current stream)."""
    x_prox = torch.zeros(n, dtype=torch.float32, device=dev)
    x_new = torch.ones(n, dtype=torch.float32, device=dev)
    w = P.ewma_proxy_update(x_prox, x_new, 0.75, w=0.0)      # first step (copy)
    w = P.ewma_proxy_update(x_prox, x_new, 0.75, w=w)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream(dev)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        w = P.ewma_proxy_update(x_prox, x_new, 0.75, w=w)
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    del x_prox, x_new
    gbps = 12 * n / (ms * 1e-3) / 1e9
    return {"bound": "hbm", "achieved": round(gbps, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
            "frac": round(gbps / HBM_PEAK_GBPS, 4), "kernel": "dppo::ewma_kernel<false, true>",
            "n": n, "dtype": "f32", "alg_bytes_per_launch": 12 * n, "kernel_ms": round(ms, 4),
            "traffic": recorded_traffic("ewma_f32_1Gi", EWMA_SOURCES) if n == 1 << 30 else None}


def versioned_logprob_measure(dev, wl, K=4, reps=20):
    """Exact old log-probs of a partial-rollout batch: K per-version logits matrices of the
    batch's shape (version 0 is the batch's own logits, the others fresh N(0, 3^2) draws) and
    a per-token version id (1..4 segments per sequence); each token's row is read from its
    version only. Algorithmic bytes: T V esize + 16 B per token (id, version, log-prob)."""
    T, V = wl.T, wl.V
    g = torch.Generator(device=dev).manual_seed(11)
    mats = [wl.logits]
    for _ in range(K - 1):
        z = torch.empty(T, V, dtype=wl.logits.dtype, device=dev)
        for a in range(0, T, 2048):
            z[a:a + 2048] = (3.0 * torch.randn(min(2048, T - a), V, generator=g, device=dev)).to(z.dtype)
        mats.append(z)
    ver = torch.as_tensor(W.version_ids(T, wl.seq_len, seed=12) % K, device=dev)
    lp = P.logprob_fwd_versioned(mats, ver, wl.ids)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream(dev)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    with P.KernelTimer() as kt:
        e0.record(stream)
        for _ in range(reps):
            lp = P.logprob_fwd_versioned(mats, ver, wl.ids)
        e1.record(stream)
        torch.cuda.synchronize()
        k_ms, k_n = kt.read()
    call_ms = e0.elapsed_time(e1) / reps
    ms = k_ms / max(1, k_n)
    b_alg = T * V * wl.logits.element_size() + 16 * T
    gbps = b_alg / (ms * 1e-3) / 1e9
    counts = np.bincount(ver.cpu().numpy(), minlength=K).tolist()
    del mats, lp
    return {"bound": "hbm", "achieved": round(gbps, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
            "frac": round(gbps / HBM_PEAK_GBPS, 4),
            "kernel": P.row_kernel_name(wl.logits.dtype, V, with_dlogits=False),
            "kernel_ms": round(ms, 4), "alg_bytes_per_launch": b_alg, "versions": K,
            "tokens_per_version": counts, "call_ms": round(call_ms, 4),
            "tokens_per_s": round(T / (call_ms * 1e-3), 1)}


def vocab_shard_measure(dev, wl, lp_mu, lp_ref, n_shards=8, reps=20):
    """One GPU's share of an n_shards-way vocabulary-parallel loss stage on the large_vocab batch:
    a contiguous [T, V / n_shards] bf16 shard. Times the shard-statistics kernel (reads the shard) and
    the shard loss kernel (reads it again, writes its dlogits); the exchange between shards
    is not part of a one-GPU run. The global lse and z[y] come from the unsharded log-prob
    call (input preparation, not timed)."""
    T, V = wl.T, wl.V
    Vs = V // n_shards
    shard = wl.logits[:, :Vs].contiguous()
    dl = torch.empty_like(shard)
    lp, lse = P.logprob_fwd(wl.logits, wl.ids, with_lse=True)
    zy = lp + lse
    kw = dict(scale_mode="const", loss_scale=1.0)

    def stats():
        return P.vocab_shard_stats(shard, wl.ids, 0, V, wl.mask)

    def loss():
        return P.decoupled_ppo_loss_shard_fwd_bwd(shard, 0, V, lse, zy, wl.ids, lp_mu, lp_ref,
                                                   wl.adv, wl.mask, dlogits=dl, **kw)

    res = {}
    for name, fn in (("stats", stats), ("loss", loss)):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        stream = torch.cuda.current_stream(dev)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        with P.KernelTimer() as kt:
            e0.record(stream)
            for _ in range(reps):
                fn()
            e1.record(stream)
            torch.cuda.synchronize()
            k_ms, k_n = kt.read()
        res[name] = (k_ms / max(1, k_n), e0.elapsed_time(e1) / reps)
    n_valid = int(wl.mask.sum().item())
    b_stats = n_valid * Vs * 2 + T * (8 + 1 + 4 + 4)
    b_loss = n_valid * Vs * 2 + T * Vs * 2 + T * (30 + 8)
    k_stats, c_stats = res["stats"]
    k_loss, c_loss = res["loss"]
    ach = b_loss / (k_loss * 1e-3) / 1e9
    del shard, dl
    return {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
            "frac": round(ach / HBM_PEAK_GBPS, 4),
            "kernel": "dppo::shard_token + dppo::shard_grad<true> (the shard loss call)",
            "kernel_ms": round(k_loss, 4), "alg_bytes_per_launch": b_loss,
            "traffic": recorded_traffic("vocab_shard_loss", SHARD_SOURCES),
            "shard": f"T={T} x Vs={Vs} (V/{n_shards}) bf16, contiguous",
            "stats_kernel": {"kernel": "dppo::shard_stats<true, true>",
                             "kernel_ms": round(k_stats, 4), "alg_bytes_per_launch": b_stats,
                             "achieved": round(b_stats / (k_stats * 1e-3) / 1e9, 1),
                             "frac": round(b_stats / (k_stats * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
                             "traffic": recorded_traffic("vocab_shard_stats", SHARD_SOURCES)},
            "step_ms": round(c_stats + c_loss, 4),
            "tokens_per_s": round(T / ((c_stats + c_loss) * 1e-3), 1)}


def interpolated_reference_measure(dev, wl, lp_mu, dlogits, b_alg, reps=20):
    """The fused call with the reference interpolated between mu_old and the current policy
    (App. A: log-linear and arithmetic proxies, alpha = 0.5) on the large_vocab batch, the
    reference formed per token inside the row kernel. Same algorithmic bytes as the main call
    less the reference log-prob it no longer reads (4 B per token)."""
    res = {}
    for mode in ("log_linear", "linear"):
        def call():
            return P.decoupled_ppo_loss_fwd_bwd(wl.logits, wl.ids, lp_mu, None, wl.adv, wl.mask,
                                                dlogits=dlogits, ref_mode=mode, alpha=0.5)
        for _ in range(3):
            call()
        torch.cuda.synchronize()
        stream = torch.cuda.current_stream(dev)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        with P.KernelTimer() as kt:
            e0.record(stream)
            for _ in range(reps):
                call()
            e1.record(stream)
            torch.cuda.synchronize()
            k_ms, k_n = kt.read()
        ms = k_ms / max(1, k_n)
        b = b_alg - 4 * wl.T
        gbps = b / (ms * 1e-3) / 1e9
        res[mode] = {"kernel_ms": round(ms, 4), "achieved": round(gbps, 1),
                     "frac": round(gbps / HBM_PEAK_GBPS, 4), "alg_bytes_per_launch": b,
                     "call_ms": round(e0.elapsed_time(e1) / reps, 4)}
    return {"bound": "hbm", "peak": HBM_PEAK_GBPS, "unit": "GB/s", "alpha": 0.5,
            "kernel": P.row_kernel_name(wl.logits.dtype, wl.V), **res}


def long_rows_measure(dev, dtype=torch.float32, T=8192, V=151936, reps=10, key="fp32_rows"):
    """Rows longer than the register-resident kernels hold (fp32 past 77824 entries, bf16 past
    155648): N(0, 3^2) logits of `dtype`, uniform token ids, every token valid, the fused
    forward and backward. Timed by the library's events around the per-row kernel (the
    resident-prefix kernel); algorithmic bytes as for the flagship rows (logits read once,
    dlogits written once, 29 B of per-token vectors)."""
    g = torch.Generator(device=dev).manual_seed(7)
    z = torch.empty(T, V, dtype=dtype, device=dev)
    for a in range(0, T, 1024):
        z[a:a + 1024] = (3.0 * torch.randn(min(1024, T - a), V, generator=g, device=dev)).to(dtype)
    ids = torch.randint(0, V, (T,), generator=g, device=dev)
    anchor = anchor_logprob(z, ids)
    lp_ref = (anchor + 0.2 * torch.randn(T, generator=g, device=dev, dtype=torch.float64)).float()
    lp_mu = (lp_ref.double() + 0.05 * torch.randn(T, generator=g, device=dev,
                                                  dtype=torch.float64)).float()
    adv = torch.randn(T, generator=g, device=dev)
    dl = torch.empty_like(z)
    out = None
    for _ in range(3):
        out = P.decoupled_ppo_loss_fwd_bwd(z, ids, lp_mu, lp_ref, adv, dlogits=dl, out=out)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream(dev)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    with P.KernelTimer() as kt:
        e0.record(stream)
        for _ in range(reps):
            out = P.decoupled_ppo_loss_fwd_bwd(z, ids, lp_mu, lp_ref, adv, dlogits=dl, out=out)
        e1.record(stream)
        torch.cuda.synchronize()
        k_ms, k_n = kt.read()
    call_ms = e0.elapsed_time(e1) / reps
    ms = k_ms / max(1, k_n)
    esize = torch.finfo(dtype).bits // 8
    b_alg = algorithmic_bytes(T, V, T, esize, 29)
    gbps = b_alg / (ms * 1e-3) / 1e9
    del z, dl, out
    name = "fp32" if dtype == torch.float32 else "bf16"
    return {"bound": "hbm", "achieved": round(gbps, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
            "frac": round(gbps / HBM_PEAK_GBPS, 4),
            "kernel": P.row_kernel_name(dtype, V), "kernel_ms": round(ms, 4),
            "alg_bytes_per_launch": b_alg, "workload": f"{name} rows T={T} V={V}",
            "call_ms": round(call_ms, 4), "tokens_per_s": round(T / (call_ms * 1e-3), 1),
            "traffic": recorded_traffic(key)}


MFMA_BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 matrix-core peak, AMD specification


def lm_head_measure(dev, reps=5):
    """Fused LM-head loss stage (hidden [8192, 4096] x weight [151936, 4096]^T, bf16, logits
    never materialised) with both gradients, one-pass backward: per-call time, and the
    matrix-core rate of the library's three product kernels (forward logit tiles, dhidden =
    G W, dW = G^T hidden; 2 T d V flops each, timed by the library's events on the call's
    stream). The method needs those three products: 6 T d V flops per call."""
    wl = W.make_lm_head_workload(dev)
    T, V, d = wl.T, wl.V, wl.hidden.shape[1]
    anchor = torch.empty(T, dtype=torch.float64, device=dev)
    for a in range(0, T, 512):           # input synthesis only (reference log-probs)
        z = wl.hidden[a:a + 512].float() @ wl.weight.float().T
        anchor[a:a + 512] = (z.gather(1, wl.ids[a:a + 512, None])[:, 0]
                             - torch.logsumexp(z, dim=1)).double()
        del z
    lp_ref, lp_mu = W.reference_logprobs(anchor, wl)
    out = None
    for _ in range(2):
        out = P.fused_lm_head_loss_fwd_bwd(wl.hidden, wl.weight, wl.ids, lp_mu, lp_ref, wl.adv,
                                           wl.mask, out=out)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream(dev)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    with P.KernelTimer() as kt:
        e0.record(stream)
        for _ in range(reps):
            out = P.fused_lm_head_loss_fwd_bwd(wl.hidden, wl.weight, wl.ids, lp_mu, lp_ref,
                                               wl.adv, wl.mask, out=out)
        e1.record(stream)
        torch.cuda.synchronize()
        k_ms, k_n = kt.read()
    call_ms = e0.elapsed_time(e1) / reps
    assert k_n == 3 * reps, k_n
    prod_ms = k_ms / k_n                 # mean over the three product kernels
    prod_flops = 2.0 * T * d * V
    achieved = prod_flops / (prod_ms * 1e-3) / 1e12
    method_flops = 3 * prod_flops
    del out, wl
    return {"bound": "mfma", "achieved": round(achieved, 1), "peak": MFMA_BF16_PEAK_TFLOPS,
            "unit": "TFLOP/s", "frac": round(achieved / MFMA_BF16_PEAK_TFLOPS, 4),
            "kernel": "dppo::lmh_fwd_tiles / dppo::lmh_grad_gemm<false, true> (dhidden) / "
                      "dppo::lmh_grad_gemm<true, true> (dW), mean per launch",
            "kernel_ms": round(prod_ms, 3), "alg_flops_per_launch": prod_flops,
            "workload": f"lm_head T={T} d={d} V={V} bf16, both gradients, one-pass backward",
            "call_ms": round(call_ms, 3), "tokens_per_s": round(T / (call_ms * 1e-3), 1),
            "call_tflops": round(method_flops / (call_ms * 1e-3) / 1e12, 1),
            "call_frac": round(method_flops / (call_ms * 1e-3) / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4),
            "call_flops": method_flops}


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or platform.machine()


def timed_steps(step, steps, dev, flush_bytes):
    """Time `steps` steps. Without a flush: back to back between two events, mean per step,
    and the library's events around the per-row kernel (mean per launch). With a flush: a
    flush_bytes buffer is read before every step (outside its events), which evicts the
    previous step's data from the 256 MB Infinity Cache without leaving dirty lines to write
    back during the step, and the medians of the per-step and per-launch times are
    returned."""
    stream = torch.cuda.current_stream(dev)
    if flush_bytes <= 0:
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        with P.KernelTimer() as kt:
            torch.cuda.synchronize()
            e0.record(stream)
            for _ in range(steps):
                step()
            e1.record(stream)
            torch.cuda.synchronize()
            k_ms_total, k_launches = kt.read()
        return e0.elapsed_time(e1) / steps, k_ms_total / max(1, k_launches), "mean"
    buf = torch.ones(flush_bytes // 4, dtype=torch.float32, device=dev)
    per_step, per_kernel = [], []
    for _ in range(steps):
        buf.sum()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        with P.KernelTimer() as kt:
            e0.record(stream)
            step()
            e1.record(stream)
            torch.cuda.synchronize()
            k_ms, k_n = kt.read()
        per_step.append(e0.elapsed_time(e1))
        per_kernel.append(k_ms / max(1, k_n))
    del buf
    return float(np.median(per_step)), float(np.median(per_kernel)), "median, cache flushed"


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="large_vocab", choices=sorted(W.WORKLOADS))
    ap.add_argument("--cpu-rows", type=int, default=0,
                    help="rows of the batch the oracle baseline runs on (0: the whole batch)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-copy", action="store_true")
    ap.add_argument("--ewma-elems", type=int, default=1 << 30,
                    help="size of the parameter-sized EWMA measurement (0 to skip)")
    ap.add_argument("--no-lm-head", action="store_true",
                    help="skip the fused LM-head measurement")
    ap.add_argument("--no-shard", action="store_true",
                    help="skip the vocabulary-shard measurement")
    ap.add_argument("--no-interp", action="store_true",
                    help="skip the fused call with interpolated references (large_vocab only)")
    ap.add_argument("--no-versioned", action="store_true",
                    help="skip the versioned log-prob measurement")
    ap.add_argument("--no-fp32", action="store_true",
                    help="skip the fp32 long-row measurement")
    ap.add_argument("--no-bf16-long", action="store_true",
                    help="skip the bf16 long-row measurement (V = 262144)")
    ap.add_argument("--flush-mb", type=int, default=-1,
                    help="read this many MB before every timed step and report medians "
                         "(default: 512 for tiny and small_vocab, whose working set fits the "
                         "256 MB Infinity Cache; 0 otherwise)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path (the loss "
              "stage would shard by token rows, with an all-reduce of five counters). "
              "Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    log(f"workload {args.workload}: drawing inputs")
    wl = W.make_workload(args.workload, device=dev)
    T, V = wl.T, wl.V
    anchor = anchor_logprob(wl.logits, wl.ids)
    if wl.e_prev is not None:                      # long_agentic: EWMA proxy reference
        lp_old, lp_prev, lp_mu = W.version_logprobs(anchor, wl)
        lp_ref = lp_prev.clone()
        P.ewma_proxy_update(lp_ref, lp_old, 0.9, normalized=False)
        x_new = lp_old
    else:
        lp_ref, lp_mu = W.reference_logprobs(anchor, wl)
        x_new = lp_ref
    del anchor
    mask = wl.mask
    n_valid = int(mask.sum().item())
    esize = wl.logits.element_size()
    dlogits = torch.empty_like(wl.logits)
    out = None
    proxy = P.EwmaProxyDevice(x_new, beta=P.beta_from_window(6), tau=0.9, patience=1)
    torch.cuda.synchronize()

    def step():
        nonlocal out
        out = P.decoupled_ppo_loss_fwd_bwd(wl.logits, wl.ids, lp_mu, lp_ref, wl.adv, mask,
                                           dlogits=dlogits, out=out)
        proxy.step(x_new, out.stats)               # reset rule + EWMA on the device, no sync

    log(f"warmup {args.warmup}")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    flush_mb = args.flush_mb
    if flush_mb < 0:
        flush_mb = 512 if args.workload in ("tiny", "small_vocab") else 0
    log(f"timing {args.steps} steps" + (f", {flush_mb} MB flush before each" if flush_mb else ""))
    ms_per_step, k_ms, timing = timed_steps(step, args.steps, dev, flush_mb << 20)
    tokens_per_s = T / (ms_per_step * 1e-3)

    # per-token vectors: ids 8, lp_mu 4, lp_ref 4, adv 4, mask 1, lp out 4, loss out 4, flags 1
    per_token = 8 + 4 + 4 + 4 + 1 + 4 + 4 + 1
    b_alg = algorithmic_bytes(T, V, n_valid, esize, per_token)
    achieved = b_alg / (k_ms * 1e-3) / 1e9
    roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS,
                "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4), "traffic": None,
                "kernel": P.row_kernel_name(wl.logits.dtype, V),
                "kernel_ms": round(k_ms, 4), "alg_bytes_per_launch": b_alg}
    roofline["traffic"] = recorded_traffic(args.workload)

    result = {
        "metric": METRIC, "value": round(tokens_per_s, 1), "unit": "tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32",
        "data": "synthetic (seeded; stands in for the paper's agentic corpus)",
        "config": {"workload": args.workload, "T": T, "V": V,
                   "logits_dtype": "bf16" if esize == 2 else "f32",
                   "sequences": f"{-(-T // wl.seq_len)}x{wl.seq_len}",
                   "masked_fraction": round(1 - n_valid / T, 4),
                   "rd_mode": "mask_weight", "band": [0.5, 2.0], "clip_eps": [0.2, 0.2],
                   "parallelism": "none (1 GPU)",
                   "timing": f"{timing} of {args.steps} steps (HIP events)"},
        "hbm_pct_of_peak": round(100 * achieved / HBM_PEAK_GBPS, 2),
        "roofline": roofline,
    }
    if not args.no_shard and args.workload == "large_vocab":
        log("vocabulary shard")
        result["vocab_shard_roofline"] = vocab_shard_measure(dev, wl, lp_mu, lp_ref)
    if not args.no_interp and args.workload == "large_vocab":
        log("interpolated references")
        result["interp_reference_roofline"] = interpolated_reference_measure(
            dev, wl, lp_mu, dlogits, b_alg)
    if not args.no_versioned:
        log("versioned log-prob")
        del dlogits
        vr = versioned_logprob_measure(dev, wl)
        if args.workload == "large_vocab":
            vr["traffic"] = recorded_traffic("versioned_logprob")
        result["versioned_logprob_roofline"] = vr
    if not args.no_fp32 and args.workload == "large_vocab":
        log("fp32 long rows")
        result["fp32_rows_roofline"] = long_rows_measure(dev)
    if not args.no_bf16_long and args.workload == "large_vocab":
        log("bf16 long rows")
        result["bf16_long_rows_roofline"] = long_rows_measure(
            dev, torch.bfloat16, T=8192, V=262144, key="bf16_long_rows")
    if args.ewma_elems > 0:
        result["ewma_roofline"] = ewma_bandwidth(dev, args.ewma_elems)
    if not args.no_lm_head:
        log("fused LM head")
        result["lm_head_roofline"] = lm_head_measure(dev)
    if not args.no_copy:
        result["context"] = {"d2d_copy_GBps": round(copy_bandwidth(dev), 1)}
    if not args.no_cpu_baseline:
        threads = min(16, len(os.sched_getaffinity(0)))
        if 0 < args.cpu_rows < T:
            rows = np.sort(np.random.default_rng(0).choice(T, size=args.cpu_rows, replace=False))
        else:
            rows = np.arange(T)
        log(f"cpu baseline: oracle on {len(rows)} rows, {threads} threads")
        rate, dt = cpu_baseline(wl, lp_mu, lp_ref, rows, threads)
        result["cpu_baseline"] = {
            "value": round(rate, 1), "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": (f"the whole {args.workload} batch" if len(rows) == T else
                       f"{len(rows)} seeded rows of the {args.workload} batch") + f" (T={T}, V={V}), "
                      f"float64 numpy oracle incl. dlogits, {dt:.1f} s wall",
            "cpu": cpu_model()}
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
