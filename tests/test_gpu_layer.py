"""GPU parity of hero_routed_layer against the CPU oracle (through the C ABI)."""
import sys

import numpy as np
import pytest

from paper_2609_08189_amd import synth
from tests.parity import check_layer

pytestmark = pytest.mark.gpu

# bf16 shapes that span several GEMM tiles in every dimension with ragged token counts
BF16_SMALL = synth.Workload("bf16_small", "bf16", d=512, d_ff=1408, d_r=64, L_R=8, d_m=128, T=777,
                            mode="budget", budget=0.27)
F32_SMALL = synth.Workload("f32_small", "f32", d=256, d_ff=688, d_r=16, L_R=4, d_m=32, T=130,
                           mode="budget", budget=0.27)


def _run(w, j, seed=0, rows=None):
    import torch
    from paper_2609_08189_amd.device import DeviceProblem
    print(f"case {w.name} dtype={w.dtype} j={j} T={w.T} d={w.d} d_ff={w.d_ff} d_m={w.d_m} "
          f"mode={w.mode} seed={seed}", flush=True)
    prob = synth.make_problem(w, seed=seed, layer_j=j)
    dp = DeviceProblem(prob)
    dp.run_layer(j)
    res = dp.results()
    report = {}
    check_layer(prob, res, j, rows=rows, report=report)
    print("  errors:", {k: (f"{v:.2e}" if isinstance(v, float) else v) for k, v in report.items()},
          flush=True)
    del dp
    torch.cuda.empty_cache()
    return report


@pytest.mark.parametrize("j", [1, 2, 3, 6])
def test_bf16_layer_budget(j):
    _run(BF16_SMALL, j, seed=1)


@pytest.mark.parametrize("j", [1, 4])
def test_bf16_layer_threshold_bimodal(j):
    _run(BF16_SMALL.replace(mode="threshold", bias="bimodal_runs", T=1029), j, seed=2)


@pytest.mark.parametrize("j", [1, 2, 3])
def test_f32_layer(j):
    _run(F32_SMALL, j, seed=4)


@pytest.mark.parametrize("d_m", [32, 64, 256])
def test_bf16_memory_widths(d_m):
    _run(BF16_SMALL.replace(d_m=d_m, T=300), 3, seed=5)


@pytest.mark.parametrize("budget", [0.0, 1.0])
def test_budget_extremes(budget):
    _run(BF16_SMALL.replace(budget=budget, T=333), 2, seed=6)


@pytest.mark.parametrize("T", [1, 2, 65])
def test_tiny_token_counts(T):
    _run(BF16_SMALL.replace(T=T), 3, seed=7)
    _run(BF16_SMALL.replace(T=T, mode="threshold"), 1, seed=7)


@pytest.mark.parametrize("state_dtype", ["f32", "bf16"])
def test_llama31_8b_layer_full_shape(state_dtype):
    """Llama-3.1-8B shape, j = 17 of 32, T = 4096, budget 26.87 %, in the launch configuration the
    benchmark times (S stored in fp32, or in bf16).  Router, memory, decisions and index lists
    are checked for every token; the branch outputs on a sample of 48 FFN and 24 adapter rows
    (the oracle's FFN is costly)."""
    import torch
    from paper_2609_08189_amd.device import DeviceProblem
    w = synth.WORKLOADS["llama31_8b_layer"].replace(state_dtype=state_dtype)
    print(f"case {w.name} T={w.T} j={w.layer_j} state={state_dtype}", flush=True)
    prob = synth.make_problem(w, seed=0)
    dp = DeviceProblem(prob)
    dp.run_layer(w.layer_j)
    res = dp.results()
    mask = res["layers"][0]["mask"]
    rng = np.random.default_rng(0)
    rows = np.zeros(w.T, bool)
    rows[rng.choice(np.nonzero(mask)[0], 48, replace=False)] = True
    rows[rng.choice(np.nonzero(~mask)[0], 24, replace=False)] = True
    report = {}
    check_layer(prob, res, w.layer_j, rows=rows, report=report)
    print("  errors:", report, flush=True)
    assert res["layers"][0]["n_ad"] == 1101
    del dp
    torch.cuda.empty_cache()


@pytest.mark.parametrize("d_r,mode", [(256, "budget"), (896, "budget"), (896, "threshold")])
def test_wide_adapter(d_r, mode):
    """Adapter ranks above 128 (the paper's 896) on the GEMM path, with ragged token counts."""
    w = BF16_SMALL.replace(d_r=d_r, mode=mode, T=613, bias="bimodal_runs" if mode == "threshold" else "none")
    _run(w, 3)


def test_llama31_8b_paper_operating_point_full_shape():
    """Llama-3.1-8B shape at the paper's operating point: adapter rank 896, memory dim 64, j = 17,
    T = 4096, 25 % skip; branch outputs on 48 FFN and 48 adapter rows, the rest for every token."""
    import torch
    from paper_2609_08189_amd.device import DeviceProblem
    w = synth.WORKLOADS["llama31_8b_paper"]
    print(f"case {w.name} T={w.T} j={w.layer_j} d_r={w.d_r} d_m={w.d_m}", flush=True)
    prob = synth.make_problem(w, seed=0)
    dp = DeviceProblem(prob)
    dp.run_layer(w.layer_j)
    res = dp.results()
    mask = res["layers"][0]["mask"]
    rng = np.random.default_rng(1)
    rows = np.zeros(w.T, bool)
    rows[rng.choice(np.nonzero(mask)[0], 48, replace=False)] = True
    rows[rng.choice(np.nonzero(~mask)[0], 48, replace=False)] = True
    report = {}
    check_layer(prob, res, w.layer_j, rows=rows, report=report)
    print("  errors:", report, flush=True)
    assert res["layers"][0]["n_ad"] == 1024
    del dp
    torch.cuda.empty_cache()


def test_persistent_gate_up_ragged():
    """More FFN tiles than CUs (the persistent gate/up kernel: each tile's results leave during
    the next tile) with a row count that is not a multiple of the tile height."""
    w = BF16_SMALL.replace(d_ff=5120, T=2001, budget=0.27)
    _run(w, 3)


def test_ffn_single_pass_tiles_ragged():
    """Enough FFN rows that both products run K in one pass (more than half the CUs' worth of
    output tiles), with a ragged row count; smaller cases split K and reduce partial sums."""
    w = BF16_SMALL.replace(d=2048, d_ff=2816, T=2201, budget=0.27)
    _run(w, 2, seed=7)


def test_ffn_split_k_decode_rows():
    """A decode-sized batch (one row tile): both FFN products split K into fp32 slices; the
    row count is ragged and K splits unevenly (d_ff / 64 = 42 k-tiles over 16 slices)."""
    w = BF16_SMALL.replace(d=1024, d_ff=2688, T=256, budget=0.27)
    _run(w, 5, seed=8)


@pytest.mark.parametrize("j", [1, 3])
def test_bf16_state(j):
    """S stored in bf16 between layers (every element written is rounded to nearest even)."""
    _run(BF16_SMALL.replace(state_dtype="bf16"), j, seed=9)


@pytest.mark.parametrize("d_m", [64, 256])
def test_bf16_state_widths_f32_weights(d_m):
    _run(F32_SMALL.replace(d_m=d_m, state_dtype="bf16"), 2, seed=10)
