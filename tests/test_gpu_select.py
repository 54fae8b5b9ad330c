"""GPU branch decision and compaction at large token counts (the run-per-thread select kernel,
above 8192 tokens) and at most 1024 tokens (one chunk of the radix-select kernel): exact budget selection on the GPU's own logits (the n_skip smallest
(logit, index) pairs, lambda), exact compaction against the GPU's mask, threshold mode, the budget
extremes, and logits tied exactly in large groups (a per-token bias of +-1e10 absorbs the router's
logit in fp32, so only the token index orders each group)."""
import numpy as np
import pytest

from oracle import hero_oracle as O
from paper_2609_08189_amd import synth
from tests.parity import check_budget_selection, check_compaction

pytestmark = pytest.mark.gpu

W = synth.Workload("select_large", "bf16", d=256, d_ff=512, d_r=32, L_R=4, d_m=32, T=9000,
                   mode="budget", budget=0.27, d_e=64, d_head=64)


def _layer(w, seed, beta=None):
    import torch
    from paper_2609_08189_amd.device import DeviceProblem
    print(f"case select T={w.T} mode={w.mode} budget={w.budget} ties={beta is not None} seed={seed}", flush=True)
    prob = synth.make_problem(w, seed=seed, layer_j=2)
    if beta is not None:
        prob.beta = beta
    dp = DeviceProblem(prob)
    dp.run_layer(2)
    L = dp.stats[0].host()
    del dp
    torch.cuda.empty_cache()
    return L


@pytest.mark.parametrize("T", [8193, 9000, 16384, 16385, 24577, 32768])
@pytest.mark.parametrize("budget", [0.0, 0.27, 0.3882, 1.0])
def test_budget_select_large(T, budget):
    w = W.replace(T=T, budget=budget)
    L = _layer(w, seed=T % 97)
    check_compaction(L, T)
    check_budget_selection(L, budget, T)


@pytest.mark.parametrize("T", [9000, 32768])
def test_budget_select_exact_ties(T):
    rng = np.random.default_rng(T)
    beta = np.where(rng.uniform(size=T) < 0.5, -1e10, 1e10).astype(np.float32)
    w = W.replace(T=T, budget=0.3882, bias="none")
    L = _layer(w, seed=5, beta=beta)
    # the router's logit vanishes into the bias: two groups of exactly equal logits
    assert set(np.unique(L["logit"])) == {np.float32(-1e10), np.float32(1e10)}
    check_compaction(L, T)
    check_budget_selection(L, w.budget, T)
    n_skip = O.n_skip_for(w.budget, T)
    low = np.nonzero(beta < 0)[0]
    # the skipped tokens are the lowest group taken in index order (and, past it, the next group's)
    if n_skip <= low.size:
        np.testing.assert_array_equal(np.nonzero(~L["mask"])[0], low[:n_skip])


@pytest.mark.parametrize("T", [9000, 32768])
def test_threshold_select_large(T):
    w = W.replace(T=T, mode="threshold", bias="bimodal_runs")
    L = _layer(w, seed=3)
    check_compaction(L, T)
    np.testing.assert_array_equal(L["mask"], L["logit"] >= np.float32(0.0))
    assert L["lam"] == 0.0


# At most 1024 tokens (a decode step): one chunk of the radix-select kernel, from a single token
# to a full chunk, ragged last waves.
@pytest.mark.parametrize("T", [1, 2, 63, 64, 65, 255, 256, 700, 1024])
@pytest.mark.parametrize("budget", [0.0, 0.27, 0.3882, 1.0])
def test_budget_select_small(T, budget):
    w = W.replace(T=T, budget=budget)
    L = _layer(w, seed=T % 89)
    check_compaction(L, T)
    check_budget_selection(L, budget, T)


@pytest.mark.parametrize("T", [256, 1024])
def test_budget_select_small_exact_ties(T):
    rng = np.random.default_rng(T + 1)
    beta = np.where(rng.uniform(size=T) < 0.5, -1e10, 1e10).astype(np.float32)
    w = W.replace(T=T, budget=0.3882, bias="none")
    L = _layer(w, seed=7, beta=beta)
    assert set(np.unique(L["logit"])) == {np.float32(-1e10), np.float32(1e10)}
    check_compaction(L, T)
    check_budget_selection(L, w.budget, T)
    n_skip = O.n_skip_for(w.budget, T)
    low = np.nonzero(beta < 0)[0]
    if n_skip <= low.size:
        np.testing.assert_array_equal(np.nonzero(~L["mask"])[0], low[:n_skip])


@pytest.mark.parametrize("T", [1, 200, 1024])
def test_threshold_select_small(T):
    w = W.replace(T=T, mode="threshold", bias="bimodal_runs")
    L = _layer(w, seed=3)
    check_compaction(L, T)
    np.testing.assert_array_equal(L["mask"], L["logit"] >= np.float32(0.0))
    assert L["n_ffn"] == int(L["mask"].sum())
    assert L["lam"] == 0.0
