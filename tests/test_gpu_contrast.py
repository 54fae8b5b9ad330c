"""High-contrast GPU parity in the benchmark's launch configurations (bf16, budget mode, fp32 state):
branch outputs several times larger than hbar and gates spread over (0.05, 0.95), so that a wrong
branch scale, a dropped part of the adapter's contraction or swapped gate factors would exceed the
2e-2 tolerance by at least five times (shown per case from the oracle).  The router's fp32 outputs
(logit, gate, p, m, S, zeta) are held to 1e-4."""
import numpy as np
import pytest

from paper_2609_08189_amd import synth
from tests.contrast import CONTRAST, mutant_errors, sample_rows
from tests.parity import TOL, check_layer, oracle_layer

pytestmark = pytest.mark.gpu


def _run(w, seed):
    import torch
    from paper_2609_08189_amd.device import DeviceProblem
    print(f"case contrast d={w.d} d_ff={w.d_ff} d_r={w.d_r} d_m={w.d_m} T={w.T} j={w.layer_j} "
          f"budget={w.budget} seed={seed}", flush=True)
    prob = synth.make_problem(w, seed=seed)
    dp = DeviceProblem(prob)
    dp.run_layer(w.layer_j)
    res = dp.results()
    mask = res["layers"][0]["mask"]
    rows = sample_rows(mask, 48, seed=seed)
    report = {}
    check_layer(prob, res, w.layer_j, rows=rows, report=report)
    ref = oracle_layer(prob, w.layer_j, forced_ffn=mask, rows=rows)
    margins = mutant_errors(prob, ref, rows)
    print("  errors:", {k: (f"{v:.2e}" if isinstance(v, float) else v) for k, v in report.items()}, flush=True)
    print("  planted-mistake errors (x tolerance):",
          {k: f"{v:.3f} ({v / TOL['bf16']:.0f}x)" for k, v in margins.items()}, flush=True)
    for k in ("logit", "gate", "p", "m", "S", "zeta"):
        assert report[k] <= 1e-4, (k, report[k])
    assert report["h"] <= TOL["bf16"]
    assert min(margins.values()) >= 5 * TOL["bf16"], margins
    g = res["layers"][0]["gate"]
    assert g.min() < 0.1 and g.max() > 0.9
    del dp
    torch.cuda.empty_cache()


@pytest.mark.parametrize("d_r", [32, 64, 96, 128])
def test_contrast_stack_tiles(d_r):
    """8192 tokens: the FFN products run 256-row tiles, as at the 8B stack's ~20k FFN rows."""
    _run(CONTRAST.replace(d_r=d_r), seed=d_r)


def test_contrast_layer_tiles_wide_adapter():
    """4096 tokens: the persistent 192-row gate/up kernel, as at the 8B layer; adapter rank 256
    on the matrix-core adapter path."""
    _run(CONTRAST.replace(d_r=256, T=4096, batch=2), seed=7)
