"""GPU parity of hero_routed_stack against the CPU oracle (through the C ABI)."""
import numpy as np
import pytest

from paper_2609_08189_amd import synth
from tests.parity import check_stack

pytestmark = pytest.mark.gpu

BF16_STACK = synth.Workload("bf16_stack", "bf16", d=512, d_ff=1408, d_r=64, L_R=6, d_m=64, T=513,
                            mode="budget", budget=0.3882)


def _run_stack(w, seed=0, rows=None):
    import torch
    from paper_2609_08189_amd.device import DeviceProblem
    print(f"case {w.name} dtype={w.dtype} L_R={w.L_R} T={w.T} d={w.d} d_ff={w.d_ff} d_m={w.d_m} "
          f"mode={w.mode} seed={seed}", flush=True)
    prob = synth.make_problem(w, seed=seed)
    dp = DeviceProblem(prob)
    dp.run_stack()
    res = dp.results()
    report = {}
    check_stack(prob, res, rows=rows, report=report)
    print("  errors:", {k: (f"{v:.2e}" if isinstance(v, float) else v) for k, v in report.items()}, flush=True)
    del dp
    torch.cuda.empty_cache()
    return prob, res


def test_bf16_stack_bf16_state():
    """A 6-layer bf16 stack with S stored in bf16 across depth."""
    _run_stack(BF16_STACK.replace(state_dtype="bf16"), seed=4)


def test_tiny_f32_stack():
    """4 routed layers, d=256, d_ff=688 (ragged for any 64-wide tile), r=16, d_m=32, T=64, 27 % skip."""
    prob, res = _run_stack(synth.WORKLOADS["tiny_f32_stack"], seed=0)
    assert all(L["n_ad"] == 17 for L in res["layers"])


def test_bf16_stack_budget():
    _run_stack(BF16_STACK, seed=1)


def test_bf16_stack_threshold_bimodal():
    _run_stack(BF16_STACK.replace(mode="threshold", bias="bimodal_runs", T=700, d_m=128), seed=2)


@pytest.mark.parametrize("L_R", [1, 2])
def test_short_stacks(L_R):
    _run_stack(BF16_STACK.replace(L_R=L_R, T=200), seed=3)


def test_stack_equals_chained_layer_calls():
    """The stack is L_R chained layer calls, bit for bit (same kernels, same rounding points)."""
    import torch
    from paper_2609_08189_amd import hero as H
    from paper_2609_08189_amd.device import DeviceProblem, LayerStats
    w = BF16_STACK.replace(T=300)
    prob = synth.make_problem(w, seed=4)
    dp = DeviceProblem(prob)
    dp.run_stack()
    ref = dp.results()
    # chained: hbar_1 = h_in, hbar_{j+1} = h_j
    hs = [dp.hbar]
    ws_bytes = H.hero_workspace_size(dp.dims, w.T, False)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dp.device)
    S = torch.full_like(dp.S, float("nan"))      # layer 1 must not read the incoming state
    zeta = torch.full_like(dp.zeta, float("nan"))
    p = torch.full_like(dp.p_hist, float("nan"))
    m = torch.full_like(dp.m_hist, float("nan"))
    state = H.hero_state(S.data_ptr(), zeta.data_ptr(), p.data_ptr(), m.data_ptr())
    stats = [LayerStats(w.T, dp.device) for _ in range(w.L_R)]
    for j in range(1, w.L_R + 1):
        out = torch.empty_like(dp.hbar)
        H.check(H.hero_routed_layer(dp.dims, j, w.T, hs[-1], hs[-2] if j >= 2 else None,
                                    hs[-3] if j >= 3 else None, out, state, dp.ffn_s[j - 1], dp.router_s,
                                    dp.adapter_s[j - 1], dp.eta[j - 1], dp.routing_s, stats[j - 1].struct,
                                    ws, ws_bytes, dp.stream()), "hero_routed_layer")
        hs.append(out)
    torch.cuda.synchronize()
    assert torch.equal(hs[-1].view(torch.int16), dp.h_out.view(torch.int16))
    assert torch.equal(S, dp.S) and torch.equal(zeta, dp.zeta)
    assert torch.equal(p, dp.p_hist) and torch.equal(m, dp.m_hist)
    for a, b in zip(stats, ref["layers"]):
        h = a.host()
        for k in ("mask", "logit", "gate"):
            np.testing.assert_array_equal(h[k], b[k])
        assert h["lam"] == b["lam"] and h["n_ffn"] == b["n_ffn"]


@pytest.mark.parametrize("budget", [0.0, 0.27, 0.39])
def test_llama2_7b_decode_stack_full_shape(budget):
    """Llama-2-7B shape, 32 routed layers, 256 sequences x 1 token, skip swept over 0, 27 and
    39 %; every token.  The stack is rerun as chained layer calls (bit-identical to it,
    captured per layer) and each layer is checked on the GPU's own inputs, so bf16 rounding
    cannot compound."""
    import torch
    from paper_2609_08189_amd.device import DeviceProblem
    from tests.parity import check_stack_layerwise
    w = synth.WORKLOADS["llama2_7b_decode"].replace(budget=budget)
    print(f"case {w.name} L_R={w.L_R} T={w.T} budget={budget}", flush=True)
    prob = synth.make_problem(w, seed=0)
    dp = DeviceProblem(prob)
    dp.run_stack()
    res = dp.results()
    io = dp.run_chained()
    final = dp.results()
    np.testing.assert_array_equal(final["h"], res["h"])
    np.testing.assert_array_equal(final["S"], res["S"])
    report = {}
    check_stack_layerwise(prob, io, report=report)
    print("  per-layer errors:", {k: (f"{v:.2e}" if isinstance(v, float) else v) for k, v in report.items()},
          flush=True)
    del dp
    torch.cuda.empty_cache()


def _full_stack_sampled(name, n_rows=48, seed=0):
    """A full-size stack workload: the stack is run once, then rerun as chained layer calls,
    which must reproduce it bit for bit (output and final state, compared on the device);
    the chained run captures a seeded sample of token rows per layer, and every layer is
    checked on those rows against the oracle on the GPU's own inputs."""
    import torch
    from paper_2609_08189_amd.device import DeviceProblem
    from tests.parity import check_stack_layerwise
    w = synth.WORKLOADS[name]
    print(f"case {w.name} L_R={w.L_R} T={w.T} d={w.d} d_ff={w.d_ff} d_m={w.d_m} mode={w.mode} "
          f"sampled rows={n_rows}", flush=True)
    prob = synth.make_problem(w, seed=seed)
    dp = DeviceProblem(prob)
    print("  inputs on the device", flush=True)
    dp.run_stack()
    torch.cuda.synchronize()
    ref = [t.clone() for t in (dp.h_out, dp.S, dp.zeta, dp.p_hist, dp.m_hist)]
    rows = np.sort(np.random.default_rng(1234 + seed).choice(w.T, size=n_rows, replace=False))
    io = dp.run_chained(rows=rows)
    torch.cuda.synchronize()
    for a, b in zip((dp.h_out, dp.S, dp.zeta, dp.p_hist, dp.m_hist), ref):
        assert torch.equal(a.view(torch.int16) if a.dtype == torch.bfloat16 else a,
                           b.view(torch.int16) if b.dtype == torch.bfloat16 else b)
    print("  stack == chained layer calls (bit-exact)", flush=True)
    del ref
    report = {}
    check_stack_layerwise(prob, io, rows=rows, report=report, verbose=True)
    print("  per-layer errors:", {k: (f"{v:.2e}" if isinstance(v, float) else v) for k, v in report.items()},
          flush=True)
    del dp
    torch.cuda.empty_cache()


def test_llama31_8b_stack_full_shape():
    """Llama-3.1-8B shape, 32 routed layers, 16 x 2048 tokens, skip budget 38.82 %."""
    _full_stack_sampled("llama31_8b_stack")


def test_llama2_13b_prefill_full_shape():
    """Llama-2-13B shape, 40 routed layers, 8 x 4096 tokens, threshold rule with the
    position-clustered bimodal logit bias."""
    _full_stack_sampled("llama2_13b_prefill")
