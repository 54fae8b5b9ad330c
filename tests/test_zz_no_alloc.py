"""hero_routed_layer_noalloc (the entry point for callers that cannot allocate: its scratch is the
library's fixed device area) against hero_routed_layer with a caller workspace, through the C ABI:
two calls in a row on the same device, the second with fewer tokens and another layer index, each
compared bit for bit (outputs, router state, statistics)."""
import numpy as np
import pytest

from paper_2609_08189_amd import hero as H
from paper_2609_08189_amd import synth

pytestmark = pytest.mark.gpu

# decode-sized bf16 layers: the FFN products split K into fp32 partials (the part of the scratch
# that the adapter's partial sums share), with ragged row counts
W = synth.Workload("noalloc", "bf16", d=1024, d_ff=2688, d_r=64, L_R=8, d_m=128, T=256,
                   mode="budget", budget=0.27)


def _host(dp, stats):
    import torch
    torch.cuda.synchronize()
    out = {"h": dp.h_out.view(torch.int16).cpu().numpy().copy(), "S": dp.S.cpu().numpy().copy(),
           "zeta": dp.zeta.cpu().numpy().copy(), "p": dp.p_hist.cpu().numpy().copy(),
           "m": dp.m_hist.cpu().numpy().copy()}
    st = stats.host()
    # the index lists are defined up to their counts only
    st["idx_ffn"] = st["idx_ffn"][:st["n_ffn"]]
    st["idx_ad"] = st["idx_ad"][:st["n_ad"]]
    for k, v in st.items():
        out["stats_" + k] = v
    return out


def _case(w, j, seed, tiled=False):
    import torch
    from paper_2609_08189_amd.device import DeviceProblem, LayerStats
    print(f"case noalloc d={w.d} d_ff={w.d_ff} T={w.T} j={j} seed={seed} tiled={tiled}", flush=True)
    prob = synth.make_problem(w, seed=seed, layer_j=j)
    dp = DeviceProblem(prob, tiled=tiled)
    state0 = [x.clone() for x in (dp.S, dp.zeta, dp.p_hist, dp.m_hist)]
    # the workspace entry point
    dp.h_out.fill_(7)
    H.check(H.hero_routed_layer(dp.dims, j, dp.T, dp.hbar, dp.prev1, dp.prev2, dp.h_out, dp.state_s,
                                dp.ffn_s[0], dp.router_s, dp.adapter_s[0], dp.eta[j - 1], dp.routing_s,
                                dp.stats[0].struct, dp.ws, dp.ws_bytes, dp.stream()), "hero_routed_layer")
    ref = _host(dp, dp.stats[0])
    # the same call on the fixed scratch: state restored, outputs and stats poisoned
    for x, x0 in zip((dp.S, dp.zeta, dp.p_hist, dp.m_hist), state0):
        x.copy_(x0)
    dp.h_out.fill_(-3)
    st2 = LayerStats(dp.T, dp.device)
    for t in (st2.mask, st2.idx_ffn, st2.idx_ad, st2.counts):
        t.fill_(0x55)
    st2.logit.fill_(float("nan"))
    st2.gate.fill_(float("nan"))
    st2.lam.fill_(float("nan"))
    H.check(H.hero_routed_layer_noalloc(dp.dims, j, dp.T, dp.hbar, dp.prev1, dp.prev2, dp.h_out, dp.state_s,
                                        dp.ffn_s[0], dp.router_s, dp.adapter_s[0], dp.eta[j - 1], dp.routing_s,
                                        st2.struct, dp.stream()), "hero_routed_layer_noalloc")
    got = _host(dp, st2)
    for k in ref:
        np.testing.assert_array_equal(np.asarray(got[k]), np.asarray(ref[k]), err_msg=k)
    print(f"  bit-identical: n_ffn {ref['stats_n_ffn']}, n_ad {ref['stats_n_ad']}", flush=True)
    del dp
    torch.cuda.empty_cache()


def test_noalloc_equals_workspace_call_twice():
    _case(W, 3, seed=11)
    _case(W.replace(T=97, budget=0.39), 2, seed=12)


def test_noalloc_with_tiled_decode_weights():
    """The same comparison with the FFN weights' tiled copies (hero_ffn_decode_weights_make), which
    the decode-sized products of both entry points read."""
    _case(W.replace(T=200), 4, seed=13, tiled=True)
