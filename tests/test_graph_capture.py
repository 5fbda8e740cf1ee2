"""The loss stage under HIP graph capture: the fused call and the device-side PPO-EWMA step
enqueue only kernels (no memset or copy nodes, no host synchronisation), so a caller can
capture them with its model step. Each replay must equal an eager run of the same step,
with eager work and synchronisations between the replays."""
import pytest
import torch

import paper_2605_12070_amd as P
from paper_2605_12070_amd import workloads as W

from helpers import torch_anchor

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


# tiny and small_vocab take count mode (the row kernel counts the mask), large_vocab the
# counting kernel and atomics
@pytest.mark.parametrize("name,T", [("tiny", 256), ("small_vocab", 1024), ("large_vocab", 512)])
def test_captured_step_replays_match_eager(name, T):
    print(f"[case] graph capture {name} T={T}", flush=True)
    wl = W.make_workload(name, device=DEV, T=T)
    anchor = torch_anchor(wl.logits, wl.ids)
    lp_ref, lp_mu = W.reference_logprobs(anchor, wl)
    dl = torch.empty_like(wl.logits)
    out = P.decoupled_ppo_loss_fwd_bwd(wl.logits, wl.ids, lp_mu, lp_ref, wl.adv, wl.mask,
                                       dlogits=dl)
    proxy = P.EwmaProxyDevice(lp_ref, beta=P.beta_from_window(6), tau=0.9, patience=1)
    x_new = lp_ref + 0.01

    def step():
        P.decoupled_ppo_loss_fwd_bwd(wl.logits, wl.ids, lp_mu, lp_ref, wl.adv, wl.mask,
                                     dlogits=dl, out=out)
        proxy.step(x_new, out.stats)

    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()

    def snapshot():
        return [t.clone() for t in (out.loss, out.stats, out.logp, out.loss_tok, out.flags, dl,
                                    proxy.x, proxy.state)]

    for r in range(3):
        before = (proxy.x.clone(), proxy.state.clone())
        step()                                   # eager reference from this state
        torch.cuda.synchronize()
        want = snapshot()
        proxy.x.copy_(before[0])
        proxy.state.copy_(before[1])
        dl.fill_(float("nan"))
        out.loss.fill_(float("nan"))
        out.stats.fill_(-1)                      # every counter must be rewritten
        g.replay()
        torch.cuda.synchronize()
        got = snapshot()
        for a, b in zip(got, want):
            assert torch.equal(a.view(torch.uint8), b.view(torch.uint8)), f"replay {r}"
        step()                                   # eager work between replays
        torch.cuda.synchronize()
