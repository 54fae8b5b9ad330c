"""GPU parity of the router's backward at one routed layer (hero_router_backward, Sec. 3.2 in
reverse order) against the oracle's router_layer_backward on the same inputs: the layer's
post-attention states, the router weights, the state entering the layer, dL/dlogit and a carried
state gradient, all seeded.  Every output is compared as one tensor, relative to its largest
reference entry: the three post-attention states' shares of dL/dhbar, all 13 router weight
gradients, dL/deta, and the carried gradient over the state the layer received (over S and zeta
only from j = 2: at j = 1 the state is a constant).  The kernels compute in fp32 from the stored
inputs (bf16 values are exact in fp32), so the bar is fp32's, 1e-4, for both storage dtypes."""
import numpy as np
import pytest

from oracle import hero_oracle as O
from paper_2609_08189_amd import synth
from tests.oracle_inputs import adapter_of, dims_of, ffn_of, router_of, state_of

TOL = 1e-4

pytestmark = pytest.mark.gpu

BF16 = synth.Workload("rbwd_bf16", "bf16", d=512, d_ff=1408, d_r=64, L_R=6, d_m=64, T=300,
                      mode="budget", budget=0.3)
F32 = synth.Workload("rbwd_f32", "f32", d=256, d_ff=688, d_r=16, L_R=4, d_m=32, T=97,
                     mode="budget", budget=0.3)


def _err(x, ref):
    return float(np.max(np.abs(x - ref)) / max(np.max(np.abs(ref)), 1e-30))


def _run(w, j, seed, c_from_forward=False):
    import torch
    from paper_2609_08189_amd.device import DeviceProblem, DeviceRouterBackward
    print(f"case {w.name} dtype={w.dtype} j={j} T={w.T} d={w.d} d_m={w.d_m} d_s={w.d_s} seed={seed} "
          f"c_from_forward={c_from_forward}", flush=True)
    prob = synth.make_problem(w, seed=seed, layer_j=j)
    T, dm = w.T, w.d_m
    rng = np.random.default_rng(seed + 1000)
    dl = rng.standard_normal(T).astype(np.float32)
    dS = (0.05 * rng.standard_normal((T, dm, dm))).astype(np.float32)
    dz = (0.1 * rng.standard_normal((T, dm))).astype(np.float32)
    dph = rng.standard_normal(T).astype(np.float32)
    dmh = rng.standard_normal(T).astype(np.float32)
    dp = DeviceProblem(prob, stats=False)
    rb = DeviceRouterBackward(dp, j, dl, dS, dz, dph, dmh, c_from_forward=c_from_forward)
    c_gpu = rb.c_read.cpu().numpy().astype(np.float64) if rb.c_read is not None else None
    rb.run()
    res = rb.results()
    del rb, dp
    torch.cuda.empty_cache()

    dims, R = dims_of(w), router_of(prob)
    state = state_of(prob) if j > 1 else O.State.initial(T, dm)
    hb = prob.hbar.f64
    h1 = prob.hbar_prev1.f64 if j >= 2 else None
    h2 = prob.hbar_prev2.f64 if j >= 3 else None
    eta = float(prob.eta[j - 1])
    fwd = O.routed_layer(j, dims, hb, h1, h2, state, ffn_of(prob.ffn[0]), R, adapter_of(prob.adapter[0]), eta,
                         mode=w.mode, budget=w.budget, tau=w.tau, round_output=False,
                         compute_rows=np.zeros(T, dtype=bool))    # the router's backward needs no branch
    G = O._zero_router(R)
    dhb, dh1, dh2, drho, dS_p, dz_p, dp_p, dm_p = O.router_layer_backward(
        j, dims, hb, h1, h2, state, fwd, R, dl.astype(np.float64), dS.astype(np.float64),
        dz.astype(np.float64), dph.astype(np.float64), dmh.astype(np.float64), G)
    rho = fwd.debug["rho"]
    if c_from_forward and j >= 2:
        errs_c = _err(c_gpu, fwd.debug["c"])
        print(f"  forward memory read c: {errs_c:.2e}", flush=True)
        assert errs_c <= TOL, f"c_read: {errs_c:.3e}"
    errs = {"dhbar": _err(res["dhbar"], dhb), "deta": abs(res["deta"] - drho * rho * (1 - rho)) /
            max(abs(drho * rho * (1 - rho)), 1e-30), "dp": _err(res["dp"], dp_p), "dm": _err(res["dm"], dm_p)}
    if j >= 2:
        errs["dhbar1"] = _err(res["dhbar1"], dh1)
        errs["dS"] = _err(res["dS"], dS_p)
        errs["dzeta"] = _err(res["dzeta"], dz_p)
    if j >= 3:
        errs["dhbar2"] = _err(res["dhbar2"], dh2)
    for name in O.RouterParams.__dataclass_fields__:
        ref = getattr(G, name)
        if name == "w_q" and j == 2:
            # entering layer 2 the memory holds one layer's pair, so the read c = v_1 (phi(q).phi(k_1)) /
            # (phi(q).phi(k_1) + eps) does not depend on q up to eps: dL/dq is the rounding residue of two
            # cancelling terms, measured against the companion projection's gradient scale
            x = res["grads"][name]
            print(f"  w_q at j = 2: max|ref| {np.max(np.abs(ref)):.2e}, max|gpu| {np.max(np.abs(x)):.2e}, "
                  f"max|dW_k| {np.max(np.abs(G.w_k)):.2e}", flush=True)
            errs["dw_q"] = float(np.max(np.abs(x - ref)) / np.max(np.abs(G.w_k)))
        elif np.any(ref):
            errs["d" + name] = _err(res["grads"][name], ref)
        else:   # structural zeros (one-layer memory terms at j = 1) stay exactly zero
            assert not np.any(res["grads"][name]), name
    print("  errors:", {k: f"{v:.2e}" for k, v in errs.items()}, flush=True)
    tol = TOL
    for k, v in errs.items():
        assert v <= tol, f"{k}: {v:.3e} > {tol:.0e}"
    return errs


@pytest.mark.parametrize("j", [1, 2, 3, 6])
def test_router_backward_bf16(j):
    _run(BF16, j, seed=j)


@pytest.mark.parametrize("j", [1, 2, 4])
def test_router_backward_f32(j):
    _run(F32, j, seed=10 + j)


@pytest.mark.parametrize("d_m", [128, 256])
def test_router_backward_memory_widths(d_m):
    _run(BF16.replace(d_m=d_m, T=129), 3, seed=20 + d_m)


def test_router_backward_odd_router_widths():
    """Router sub-widths that are not multiples of the wave or the tile (fp32 accepts any)."""
    _run(F32.replace(d_s=19, d_h=11, d_a=8, d_e=86, d_p=53, d_head=149, T=61), 3, seed=31)


def test_router_backward_one_token():
    _run(BF16.replace(T=1), 4, seed=41)


@pytest.mark.parametrize("c_from_forward", [False, True])
def test_router_backward_1500_tokens(c_from_forward):
    """94 batches of 16 tokens, the last one ragged (12 tokens)."""
    _run(BF16.replace(T=1500), 3, seed=61, c_from_forward=c_from_forward)


def test_router_backward_llama31_8b_layer_full_shape():
    """The Llama-3.1-8B routed layer's router (d = 4096, d_m = 128, 4096 tokens, routed layer 17):
    every token, every weight gradient."""
    w = synth.WORKLOADS["llama31_8b_layer"]
    _run(w, w.layer_j, seed=3)


@pytest.mark.parametrize("w,j", [(BF16, 2), (BF16, 3), (BF16, 6), (F32, 4), (BF16.replace(T=1), 4),
                                 (BF16.replace(d_m=256, T=129), 3)],
                         ids=["bf16-j2", "bf16-j3", "bf16-j6", "f32-j4", "one-token", "d_m256"])
def test_router_backward_with_the_forwards_memory_read(w, j):
    """The layer's forward writes its memory read c to hero_state.c_read and the backward takes it
    instead of reading S_{j-1} for it a second time: c itself and every gradient to the same bar."""
    _run(w, j, seed=50 + j, c_from_forward=True)


def test_router_backward_llama31_8b_layer_with_the_forwards_memory_read():
    w = synth.WORKLOADS["llama31_8b_layer"]
    _run(w, w.layer_j, seed=4, c_from_forward=True)


def test_router_backward_first_layer_without_state():
    """At j = 1 the received state is the initial one and need not be passed: the same results with
    and without it, bit for bit."""
    import torch
    from paper_2609_08189_amd import hero as H
    from paper_2609_08189_amd.device import DeviceProblem, DeviceRouterBackward
    w = BF16.replace(T=77)
    prob = synth.make_problem(w, seed=51, layer_j=1)
    rng = np.random.default_rng(52)
    T, dm = w.T, w.d_m
    args = (rng.standard_normal(T).astype(np.float32), (0.05 * rng.standard_normal((T, dm, dm))).astype(np.float32),
            (0.1 * rng.standard_normal((T, dm))).astype(np.float32), rng.standard_normal(T).astype(np.float32),
            rng.standard_normal(T).astype(np.float32))
    dp = DeviceProblem(prob, stats=False)
    outs = []
    for with_state in (True, False):
        rb = DeviceRouterBackward(dp, 1, *args)
        if not with_state:
            dp.state_s, saved = None, dp.state_s
        rb.run()
        if not with_state:
            dp.state_s = saved
        outs.append(rb.results())
    a, b = outs
    for k in ("dhbar", "dS", "dzeta", "dp", "dm"):
        np.testing.assert_array_equal(a[k], b[k])
    for k in a["grads"]:
        np.testing.assert_array_equal(a["grads"][k], b["grads"][k])
    del dp
    torch.cuda.empty_cache()
