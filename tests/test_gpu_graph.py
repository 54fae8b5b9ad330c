"""Replays of a call captured as a HIP graph (torch.cuda.graph around the library's launches) give
the eager call's results bit for bit.  Every replay is checked, with eager work and host
synchronisation between replays, and the outputs are poisoned before each replay so that a replay
that did not run is caught."""
import numpy as np
import pytest

from paper_2609_08189_amd import synth

pytestmark = pytest.mark.gpu


def _stack_case(w, seed):
    import torch
    from paper_2609_08189_amd.device import DeviceProblem
    print(f"case graph {w.name} T={w.T} d={w.d} d_ff={w.d_ff} L_R={w.L_R}", flush=True)
    prob = synth.make_problem(w, seed=seed)
    dp = DeviceProblem(prob, stats=True)
    dp.run_stack()
    torch.cuda.synchronize()
    ref = {k: v.clone() for k, v in dict(h=dp.h_out, S=dp.S, zeta=dp.zeta, p=dp.p_hist, m=dp.m_hist,
                                         gate=dp.stats[-1].gate, idx=dp.stats[-1].idx_ffn).items()}
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        dp.run_stack()
    torch.cuda.synchronize()
    junk = torch.randn(1 << 20, device="cuda")
    for rep in range(3):
        for t in (dp.h_out, dp.S, dp.zeta, dp.p_hist, dp.m_hist, dp.stats[-1].gate):
            t.view(torch.uint8).fill_(0xFF)
        junk.mul_(1.0001)                     # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = dict(h=dp.h_out, S=dp.S, zeta=dp.zeta, p=dp.p_hist, m=dp.m_hist, gate=dp.stats[-1].gate,
                   idx=dp.stats[-1].idx_ffn)
        for k in ref:
            assert torch.equal(got[k].view(torch.uint8), ref[k].view(torch.uint8)), f"replay {rep}: {k}"
    del g, dp
    torch.cuda.empty_cache()


def test_graph_replay_of_a_stack():
    _stack_case(synth.Workload("graph_bf16", "bf16", d=512, d_ff=1408, d_r=64, L_R=4, d_m=64, T=300,
                               mode="budget", budget=0.27), 1)


def test_graph_replay_of_a_decode_sized_stack():
    """Few rows per layer: the FFN products take the K-split path with its reduce passes."""
    _stack_case(synth.Workload("graph_dec", "bf16", d=1024, d_ff=2816, d_r=64, L_R=3, d_m=128, T=96,
                               mode="budget", budget=0.27), 2)


def test_graph_replay_of_the_block_backward():
    import torch
    from paper_2609_08189_amd.device import DeviceBackward
    from oracle import hero_oracle as O
    w = synth.Workload("graph_bwd", "bf16", d=512, d_ff=1408, d_r=64, L_R=4, d_m=64, T=333, mode="budget",
                       budget=0.27)
    print(f"case graph backward T={w.T}", flush=True)
    hbar = synth.hidden(w, 3)
    ffn, ad = synth.ffn_layer(w, 0, 3), synth.adapter_layer(w, 0, 3)
    dh, gate, use_ffn = synth.backward_inputs(w, 3, n_adapter=O.n_skip_for(w.budget, w.T))
    db = DeviceBackward(w, hbar, ffn, ad, dh, gate, use_ffn, budget=w.budget)
    db.run()
    torch.cuda.synchronize()
    outs = (db.dhbar, db.dgate, db.dlogit, db.dw1, db.dw2)
    ref = [t.clone() for t in outs]
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        db.run()
    torch.cuda.synchronize()
    for rep in range(3):
        for t in outs:
            t.view(torch.uint8).fill_(0xFF)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for name, a, b in zip(("dhbar", "dgate", "dlogit", "dw1", "dw2"), outs, ref):
            assert torch.equal(a.view(torch.uint8), b.view(torch.uint8)), f"replay {rep}: {name}"
    del g, db
    torch.cuda.empty_cache()
