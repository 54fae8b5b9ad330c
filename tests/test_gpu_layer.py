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
