"""The FFN weights in the decode products' streaming order (hero_ffn_decode_weights_make).

A branch of at most 256 rows reads the tiled copies instead of W_g, W_u, W_d.  The same rows land
in the same LDS slots either way, so a call with the tiled weights must equal the call without them
bit for bit; each case also checks the tiled call against the oracle.
"""
import numpy as np
import pytest

from paper_2609_08189_amd import synth
from tests.parity import check_layer

pytestmark = pytest.mark.gpu

BF16_DECODE = synth.Workload("bf16_decode", "bf16", d=512, d_ff=1408, d_r=64, L_R=8, d_m=128, T=256,
                             mode="budget", budget=0.27)


def _bits(t):
    import torch
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t


def test_tiled_layout_is_the_documented_permutation():
    """w_gate_up_tiled[t][b][0|1][r][c] = W_g|W_u[16 b + r][64 t + c]; w_down_tiled[t][b][r][c] = W_d[16 b + r][64 t + c]."""
    import torch
    from paper_2609_08189_amd.device import DeviceProblem
    w = BF16_DECODE.replace(T=16)
    prob = synth.make_problem(w, seed=3, layer_j=2)
    dp = DeviceProblem(prob, tiled=True)
    torch.cuda.synchronize()
    f = dp.ffn[0]
    d, d_ff = w.d, w.d_ff
    tile = lambda m, n, k: m.view(n // 16, 16, k // 64, 64).permute(2, 0, 1, 3)
    want_gu = torch.stack([tile(f["w_gate"], d_ff, d), tile(f["w_up"], d_ff, d)], dim=2).reshape(-1)
    want_d = tile(f["w_down"], d, d_ff).reshape(-1)
    assert torch.equal(_bits(f["w_gate_up_tiled"]), _bits(want_gu))
    assert torch.equal(_bits(f["w_down_tiled"]), _bits(want_d))


@pytest.mark.parametrize("T,budget", [(1, 0.0), (37, 0.27), (200, 0.39), (256, 0.27), (256, 0.0)])
def test_decode_layer_tiled_equals_untiled(T, budget):
    """Ragged decode batches (1 to 256 rows, every row tile count of the skinny products): the layer
    call with the tiled weights equals the call without them bit for bit, and matches the oracle."""
    import torch
    from paper_2609_08189_amd.device import DeviceProblem
    w = BF16_DECODE.replace(T=T, budget=budget)
    print(f"case {w.name} T={T} budget={budget} j=3", flush=True)
    prob = synth.make_problem(w, seed=11 + T, layer_j=3)
    out = []
    for tiled in (False, True):
        dp = DeviceProblem(prob, tiled=tiled)
        dp.run_layer(3)
        torch.cuda.synchronize()
        out.append((dp, [t.clone() for t in (dp.h_out, dp.S, dp.zeta, dp.p_hist, dp.m_hist)]))
    for a, b in zip(out[0][1], out[1][1]):
        assert torch.equal(_bits(a), _bits(b))
    res = out[1][0].results()
    report = {}
    check_layer(prob, res, 3, report=report)
    print("  errors:", {k: (f"{v:.2e}" if isinstance(v, float) else v) for k, v in report.items()}, flush=True)
    del out
    torch.cuda.empty_cache()


@pytest.mark.parametrize("budget", [0.0, 0.27, 0.39])
def test_llama2_7b_decode_stack_tiled(budget):
    """The Llama-2-7B decode stack (32 layers, 256 sequences x 1 token) as bench.py times it, with the
    tiled weights: bit-identical to the stack on the row-major weights; at 27 % skip every layer is
    also checked against the oracle on the GPU's own inputs (chained layer calls, every token)."""
    import torch
    from paper_2609_08189_amd.device import DeviceProblem, make_tiled
    from tests.parity import check_stack_layerwise
    w = synth.WORKLOADS["llama2_7b_decode"].replace(budget=budget)
    print(f"case {w.name} L_R={w.L_R} T={w.T} budget={budget} tiled", flush=True)
    prob = synth.make_problem(w, seed=0)
    dp = DeviceProblem(prob)
    dp.run_stack()
    torch.cuda.synchronize()
    ref = [t.clone() for t in (dp.h_out, dp.S, dp.zeta, dp.p_hist, dp.m_hist)]
    ref_stats = [s.host() for s in dp.stats]
    make_tiled(dp.dims, dp.ffn, dp.ffn_s, dp.device)
    dp.run_stack()
    torch.cuda.synchronize()
    for a, b in zip((dp.h_out, dp.S, dp.zeta, dp.p_hist, dp.m_hist), ref):
        assert torch.equal(_bits(a), _bits(b))
    for a, b in zip(dp.stats, ref_stats):
        h = a.host()
        for k in ("mask", "logit", "gate"):
            np.testing.assert_array_equal(h[k], b[k])
    print("  tiled stack == row-major stack (bit-exact)", flush=True)
    if budget == 0.27:
        io = dp.run_chained()
        report = {}
        check_stack_layerwise(prob, io, report=report)
        print("  per-layer errors:", {k: (f"{v:.2e}" if isinstance(v, float) else v) for k, v in report.items()},
              flush=True)
    del dp, ref
    torch.cuda.empty_cache()
