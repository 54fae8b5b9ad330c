"""GPU parity of the router ablations (Table 3, Sec. 4.3) against the CPU oracle, through the
C ABI: every ablation bit alone and combined, in both kernel families (bf16 matrix cores,
fp32), for single layers, a stack and the depth-history memory form.  The ablations without
memory access must leave the memory buffers bit-for-bit as they were."""
import dataclasses

import numpy as np
import pytest

from oracle import hero_oracle as O
from paper_2609_08189_amd import synth
from tests.parity import TOL, check_layer, check_stack, oracle_layer, row_rel_err, scalar_err

pytestmark = pytest.mark.gpu

BF16 = synth.Workload("bf16_abl", "bf16", d=512, d_ff=1408, d_r=64, L_R=8, d_m=128, T=333,
                      mode="budget", budget=0.27)
F32 = synth.Workload("f32_abl", "f32", d=256, d_ff=688, d_r=16, L_R=4, d_m=32, T=130,
                     mode="budget", budget=0.27)


def _run(w, j, seed):
    import torch
    from paper_2609_08189_amd.device import DeviceProblem
    print(f"case {w.name} dtype={w.dtype} j={j} T={w.T} d_m={w.d_m} ablation={w.ablation} "
          f"seed={seed}", flush=True)
    prob = synth.make_problem(w, seed=seed, layer_j=j)
    dp = DeviceProblem(prob)
    dp.run_layer(j)
    res = dp.results()
    report = {}
    check_layer(prob, res, j, report=report)
    print("  errors:", {k: (f"{v:.2e}" if isinstance(v, float) else v) for k, v in report.items()},
          flush=True)
    del dp
    torch.cuda.empty_cache()
    return res


@pytest.mark.parametrize("ablation,j", [(O.NO_POS_STATE, 3), (O.NO_AUX_STATE, 3), (O.NO_MEMREAD, 3),
                                        (O.NO_HISTORY, 3), (O.NO_MEMREAD, 1), (O.NO_HISTORY, 1),
                                        (15, 4), (O.NO_POS_STATE | O.NO_MEMREAD, 2)])
def test_bf16_layer_ablation(ablation, j):
    res = _run(BF16.replace(ablation=ablation), j, seed=20 + ablation)
    if ablation & O.NO_HISTORY:
        assert np.all(res["p_hist"] == 1.0) and np.all(res["m_hist"] == 1.0)


@pytest.mark.parametrize("ablation,j", [(O.NO_MEMREAD, 2), (O.NO_HISTORY, 3),
                                        (O.NO_POS_STATE | O.NO_AUX_STATE, 3)])
def test_f32_layer_ablation(ablation, j):
    _run(F32.replace(ablation=ablation), j, seed=40 + ablation)


@pytest.mark.parametrize("ablation", [O.NO_POS_STATE | O.NO_MEMREAD, O.NO_AUX_STATE | O.NO_HISTORY])
def test_f32_stack_ablation(ablation):
    import torch
    from paper_2609_08189_amd.device import DeviceProblem
    w = synth.WORKLOADS["tiny_f32_stack"].replace(ablation=ablation)
    print(f"case {w.name} ablation={ablation}", flush=True)
    prob = synth.make_problem(w, seed=3)
    dp = DeviceProblem(prob)
    dp.run_stack()
    report = {}
    check_stack(prob, dp.results(), report=report)
    print("  errors:", report, flush=True)
    del dp
    torch.cuda.empty_cache()


def test_history_form_without_memread_leaves_the_pairs():
    """Depth-history memory form, mid-stack layer, w/o MemRead: the stored pairs (NaN past the
    earlier layers' entries) come back bit-for-bit, and the routed outputs match the oracle."""
    import torch
    from paper_2609_08189_amd.device import DeviceProblem
    j = 4
    w = BF16.replace(ablation=O.NO_MEMREAD)
    print(f"case {w.name} history form j={j} ablation={w.ablation}", flush=True)
    prob = synth.make_problem(w, seed=61, layer_j=j)
    dp = DeviceProblem(prob, history=True)
    kv0 = dp.kv.clone()
    dp.run_layer(j)
    torch.cuda.synchronize()
    assert torch.equal(dp.kv.view(torch.int32), kv0.view(torch.int32)), "stored pairs were written"
    L = dp.stats[0].host()
    h = dp.results()["h"]
    p = dp.p_hist.cpu().numpy().astype(np.float64)
    m = dp.m_hist.cpu().numpy().astype(np.float64)
    # the oracle ignores the memory under this ablation, so any incoming state serves
    ref = oracle_layer(dataclasses.replace(prob, S=np.zeros_like(prob.S), zeta=np.zeros_like(prob.zeta)),
                       j, forced_ffn=L["mask"])
    tol = TOL[w.dtype]
    errs = dict(logit=scalar_err(L["logit"], ref.logit), gate=scalar_err(L["gate"], ref.gate),
                h=row_rel_err(h, ref.h), p=scalar_err(p, ref.state.p_hist),
                m=scalar_err(m, ref.state.m_hist))
    print("  errors:", errs, flush=True)
    for k, v in errs.items():
        assert v <= tol, f"{k}: {v:.3e} > {tol:.0e}"
    del dp
    torch.cuda.empty_cache()
