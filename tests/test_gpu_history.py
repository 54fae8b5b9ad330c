"""GPU parity of the depth-history form of the router memory (hero_routed_layer_hist,
hero_routed_stack_hist, hero_history_state) against the CPU oracle's matrix form.

The incoming state of a mid-stack layer call is given to the GPU as the pairs of the earlier
layers and to the oracle as the matrix-form state the oracle builds from the same pairs
(memory_from_pairs, pinned against the recurrence).  History entries the call must not read
hold NaN, so any stray read shows up in the outputs."""
import dataclasses

import numpy as np
import pytest

from oracle import hero_oracle as O
from paper_2609_08189_amd import synth
from tests.parity import check_layer, check_stack, check_stack_layerwise

pytestmark = pytest.mark.gpu

BF16_SMALL = synth.Workload("bf16_small", "bf16", d=512, d_ff=1408, d_r=64, L_R=8, d_m=128, T=777,
                            mode="budget", budget=0.27)
F32_SMALL = synth.Workload("f32_small", "f32", d=256, d_ff=688, d_r=16, L_R=4, d_m=32, T=130,
                           mode="budget", budget=0.27)
BF16_STACK = synth.Workload("bf16_stack", "bf16", d=512, d_ff=1408, d_r=64, L_R=6, d_m=64, T=513,
                            mode="budget", budget=0.3882)


def _fmt(report):
    return {k: (f"{v:.2e}" if isinstance(v, float) else v) for k, v in report.items()}


def _oracle_problem(prob, j):
    """The problem with its incoming matrix-form state rebuilt in float64 from the memory pairs,
    with the decays of layers 1..j-1."""
    if prob.mem_k is None:
        return prob
    rho = O.sigmoid(prob.eta[:j - 1].astype(np.float64))
    S, zeta = O.memory_from_pairs(prob.mem_k.astype(np.float64), prob.mem_v.astype(np.float64), rho)
    return dataclasses.replace(prob, S=S, zeta=zeta)


def _run_layer(w, j, seed=0, rows=None, prob=None):
    import torch
    from paper_2609_08189_amd.device import DeviceProblem
    print(f"case history {w.name} dtype={w.dtype} j={j} T={w.T} d={w.d} d_m={w.d_m} mode={w.mode} "
          f"seed={seed}", flush=True)
    prob = prob or synth.make_problem(w, seed=seed, layer_j=j)
    dp = DeviceProblem(prob, history=True)
    dp.run_layer(j)
    res = dp.results()
    report = {}
    check_layer(_oracle_problem(prob, j), res, j, rows=rows, report=report)
    print("  errors:", _fmt(report), flush=True)
    del dp
    torch.cuda.empty_cache()
    return res


@pytest.mark.parametrize("j", [1, 2, 3, 6])
def test_bf16_layer_history(j):
    _run_layer(BF16_SMALL, j)


@pytest.mark.parametrize("d_m", [32, 64, 256])
def test_history_memory_widths(d_m):
    _run_layer(BF16_SMALL.replace(d_m=d_m, T=300), 5)


def test_f32_layer_history():
    _run_layer(F32_SMALL, 3)


def test_history_state_matches_oracle():
    """hero_history_state against the oracle's memory_from_pairs for every prefix n."""
    import torch
    from paper_2609_08189_amd import hero as H
    from paper_2609_08189_amd.device import dims_struct
    w = BF16_SMALL.replace(L_R=7, d_m=64, T=37)
    dims = dims_struct(w)
    rng = np.random.default_rng(5)
    k = np.exp(0.5 * rng.standard_normal((w.T, w.L_R, w.d_m))).astype(np.float32)
    v = rng.standard_normal((w.T, w.L_R, w.d_m)).astype(np.float32)
    eta = np.linspace(-1.0, 3.0, w.L_R).astype(np.float32)
    kv = torch.from_numpy(np.stack([k, v], axis=2)).to("cuda:0")
    for n in range(0, w.L_R + 1):
        S = torch.empty((w.T, w.d_m, w.d_m), dtype=torch.float32, device="cuda:0")
        zeta = torch.empty((w.T, w.d_m), dtype=torch.float32, device="cuda:0")
        H.check(H.hero_history_state(dims, n, w.T, kv, list(eta[:n]), S, zeta), "hero_history_state")
        torch.cuda.synchronize()
        S_ref, z_ref = O.memory_from_pairs(k[:, :n].astype(np.float64), v[:, :n].astype(np.float64),
                                           O.sigmoid(eta[:n].astype(np.float64)))
        scale = max(float(np.abs(S_ref).max()), 1.0)
        assert float(np.abs(S.cpu().numpy() - S_ref).max()) <= 1e-5 * scale, n
        assert float(np.abs(zeta.cpu().numpy() - z_ref).max()) <= 1e-5 * max(float(np.abs(z_ref).max()), 1.0), n


def test_history_stack_and_chained():
    """The history-form stack against the oracle, and equal bit for bit to chained
    hero_routed_layer_hist calls (output, pairs, p, m)."""
    import torch
    from paper_2609_08189_amd.device import DeviceProblem
    w = BF16_STACK
    print(f"case history stack {w.name} L_R={w.L_R} T={w.T}", flush=True)
    prob = synth.make_problem(w, seed=0)
    dp = DeviceProblem(prob, history=True)
    dp.run_stack()
    res = dp.results()
    report = {}
    check_stack(prob, res, report=report)
    print("  errors:", _fmt(report), flush=True)
    ref = [t.clone() for t in (dp.h_out, dp.kv, dp.p_hist, dp.m_hist)]
    dp.run_chained()
    torch.cuda.synchronize()
    assert torch.equal(dp.h_out.view(torch.int16), ref[0].view(torch.int16))
    for a, b in zip((dp.kv, dp.p_hist, dp.m_hist), ref[1:]):
        assert torch.equal(a, b)
    del dp
    torch.cuda.empty_cache()


def test_llama31_8b_layer_history_full_shape():
    """Llama-3.1-8B shape, j = 17 of 32, T = 4096, budget 26.87 %, 16 stored pairs per token;
    router, memory and decisions for every token, branch outputs on sampled rows."""
    import torch
    from paper_2609_08189_amd.device import DeviceProblem
    w = synth.WORKLOADS["llama31_8b_layer"]
    print(f"case history {w.name} T={w.T} j={w.layer_j}", flush=True)
    prob = synth.make_problem(w, seed=0)
    dp = DeviceProblem(prob, history=True)
    dp.run_layer(w.layer_j)
    res = dp.results()
    mask = res["layers"][0]["mask"]
    rng = np.random.default_rng(0)
    rows = np.zeros(w.T, bool)
    rows[rng.choice(np.nonzero(mask)[0], 48, replace=False)] = True
    rows[rng.choice(np.nonzero(~mask)[0], 24, replace=False)] = True
    report = {}
    check_layer(_oracle_problem(prob, w.layer_j), res, w.layer_j, rows=rows, report=report)
    print("  errors:", _fmt(report), flush=True)
    del dp
    torch.cuda.empty_cache()


def test_llama31_8b_stack_history_full_shape():
    """The 32-layer, 16 x 2048-token stack in history form: stack == chained calls bit for
    bit, then every layer on sampled rows against the oracle on the GPU's own inputs."""
    import torch
    from paper_2609_08189_amd.device import DeviceProblem
    w = synth.WORKLOADS["llama31_8b_stack"]
    print(f"case history {w.name} L_R={w.L_R} T={w.T}", flush=True)
    prob = synth.make_problem(w, seed=0)
    dp = DeviceProblem(prob, history=True)
    dp.run_stack()
    torch.cuda.synchronize()
    ref = [t.clone() for t in (dp.h_out, dp.kv, dp.p_hist, dp.m_hist)]
    rows = np.sort(np.random.default_rng(99).choice(w.T, size=48, replace=False))
    io = dp.run_chained(rows=rows)
    torch.cuda.synchronize()
    assert torch.equal(dp.h_out.view(torch.int16), ref[0].view(torch.int16))
    for a, b in zip((dp.kv, dp.p_hist, dp.m_hist), ref[1:]):
        assert torch.equal(a, b)
    print("  stack == chained layer calls (bit-exact)", flush=True)
    del ref
    report = {}
    check_stack_layerwise(prob, io, rows=rows, report=report, verbose=True)
    print("  per-layer errors:", _fmt(report), flush=True)
    del dp
    torch.cuda.empty_cache()
