"""GPU parity of the whole training-side backward of a routed stack, chained through the C ABI,
against the oracle's routed_stack_backward: a forward of L_R routed layers layer by layer
(hero_routed_layer, keeping each layer's input and the router state it received), then for
j = L_R .. 1 the block's backward (hero_routed_block_backward, given dL/dh of the layer's output
and the penalty's dL/dg) followed by the router's (hero_router_backward, given that block's
dL/dlogit and the carried state gradient), the post-attention states' gradients adding up across
the calls.  Compared: dL/dh_in, the 13 shared router weight gradients, every dL/deta_j, every
layer's adapter gradients and dL/dlogit.  fp32 storage, so that the chain carries no bf16
rounding of the gradients (the bar is fp32's, 1e-4); the oracle follows the GPU's branch decisions."""
import numpy as np
import pytest

from oracle import hero_oracle as O
from paper_2609_08189_amd import synth
from tests.oracle_inputs import adapter_of, dims_of, ffn_of, router_of

pytestmark = pytest.mark.gpu

TOL = 1e-4


def _err(x, ref):
    return float(np.max(np.abs(x - ref)) / max(np.max(np.abs(ref)), 1e-30))


@pytest.mark.parametrize("L_R,T,d_m,seed,dtype", [(4, 97, 32, 3, "f32"), (5, 64, 64, 4, "f32"), (3, 200, 64, 5, "bf16")])
def test_stack_backward_chain_matches_oracle(L_R, T, d_m, seed, dtype):
    """fp32 storage: the bar is fp32's.  bf16 storage (the training dtype): the forward rounds every
    hidden state and the block backward takes dL/dh in bf16, so the chain rounds at each layer
    boundary against the oracle's unrounded float64; the bar is bf16's, 2e-2."""
    import torch
    from paper_2609_08189_amd import hero as H
    from paper_2609_08189_amd.device import DeviceProblem, LayerStats

    if dtype == "f32":
        w = synth.Workload("sbwd_f32", "f32", d=256, d_ff=688, d_r=16, L_R=L_R, d_m=d_m, T=T, mode="budget",
                           budget=0.3)
    else:
        w = synth.Workload("sbwd_bf16", "bf16", d=512, d_ff=1408, d_r=64, L_R=L_R, d_m=d_m, T=T, mode="budget",
                           budget=0.3)
    tol = TOL if dtype == "f32" else 2e-2
    print(f"case L_R={L_R} T={T} d_m={d_m} seed={seed}", flush=True)
    prob = synth.make_problem(w, seed=seed)
    dp = DeviceProblem(prob, stats=False, for_stack=True)
    dev, dims, s = dp.device, dp.dims, dp.stream()
    f32 = lambda shape: torch.zeros(*shape, dtype=torch.float32, device=dev)
    L, d = L_R, w.d

    # forward, layer by layer, keeping every layer's input and the router state it received
    hb = [dp.hbar] + [torch.empty_like(dp.hbar) for _ in range(L)]
    S, zeta, p, m = f32((T, d_m, d_m)), f32((T, d_m)), torch.ones(T, device=dev), torch.ones(T, device=dev)
    st = H.hero_state(S.data_ptr(), zeta.data_ptr(), p.data_ptr(), m.data_ptr())
    stats = [LayerStats(T, dev) for _ in range(L)]
    ws_bytes = H.hero_workspace_size(dims, T, False)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    states_in = []
    for j in range(1, L + 1):
        states_in.append([x.clone() for x in (S, zeta, p, m)])
        H.check(H.hero_routed_layer(dims, j, T, hb[j - 1], hb[j - 2] if j >= 2 else None,
                                    hb[j - 3] if j >= 3 else None, hb[j], st, dp.ffn_s[j - 1], dp.router_s,
                                    dp.adapter_s[j - 1], dp.eta[j - 1], dp.routing_s, stats[j - 1].struct, ws,
                                    ws_bytes, s), "hero_routed_layer")
    torch.cuda.synchronize()
    use_ffn = [st_.host()["mask"] for st_ in stats]

    # backward: block, then router, for j = L .. 1
    rng = np.random.default_rng(seed + 500)
    dh_out = rng.standard_normal((T, d)).astype(np.float32)
    dg_in = [rng.standard_normal(T).astype(np.float32) for _ in range(L)]
    dHB = [f32((T, d)) for _ in range(L + 2)]
    dHB[L + 1] = torch.from_numpy(dh_out).to(dev)
    carry_t = [f32((T, d_m, d_m)), f32((T, d_m)), f32((T,)), f32((T,))]
    carry = H.hero_router_carry(*[x.data_ptr() for x in carry_t])
    rgrads = {k: f32(tuple(dp.router[k].shape)) for k in H.ROUTER_FIELDS}
    rgrads_s = H.hero_router_grads(**{k: v.data_ptr() for k, v in rgrads.items()})
    deta = f32((L, 4))
    bws_bytes = H.hero_backward_workspace_size(dims, T)
    bws = torch.empty(bws_bytes, dtype=torch.uint8, device=dev)
    rws_bytes = H.hero_router_backward_workspace_size(dims, T)
    rws = torch.empty(rws_bytes, dtype=torch.uint8, device=dev)
    # the block backward writes dL/dhbar in the storage dtype
    dhb_tmp = torch.zeros(T, d, dtype=dp.hbar.dtype, device=dev)
    dgate, dlogit = f32((T,)), [f32((T,)) for _ in range(L)]
    dw1 = [f32((w.d_r, d)) for _ in range(L)]
    dw2 = [f32((d, w.d_r)) for _ in range(L)]
    gin = [torch.from_numpy(g).to(dev) for g in dg_in]
    for j in range(L, 0, -1):
        wt = torch.float32 if dtype == "f32" else torch.bfloat16
        wdt = torch.empty(w.d_ff, d, dtype=wt, device=dev)
        wgut = torch.empty(d, 2 * w.d_ff, dtype=wt, device=dev)
        H.check(H.hero_ffn_backward_weights_make(dims, dp.ffn_s[j - 1], wdt, wgut, s), "ffn_t")
        grads = H.hero_block_grads(dhb_tmp.data_ptr(), dgate.data_ptr(), dlogit[j - 1].data_ptr(),
                                   dw1[j - 1].data_ptr(), dw2[j - 1].data_ptr())
        sj = stats[j - 1]
        dh_in = dHB[j + 1] if dtype == "f32" else dHB[j + 1].to(torch.bfloat16)
        H.check(H.hero_routed_block_backward(dims, T, hb[j - 1], dh_in, sj.gate, sj.idx_ffn, sj.idx_ad,
                                             sj.counts, None, gin[j - 1], dp.ffn_s[j - 1],
                                             H.hero_ffn_backward_weights(wdt.data_ptr(), wgut.data_ptr()),
                                             dp.adapter_s[j - 1], grads, bws, bws_bytes, s), "block backward")
        dHB[j] += dhb_tmp.float()
        Sj, zj, pj, mj = states_in[j - 1]
        H.check(H.hero_router_backward(dims, j, T, hb[j - 1], hb[j - 2] if j >= 2 else None,
                                       hb[j - 3] if j >= 3 else None,
                                       H.hero_state(Sj.data_ptr(), zj.data_ptr(), pj.data_ptr(), mj.data_ptr()),
                                       dp.router_s, dp.eta[j - 1], dlogit[j - 1], carry, dHB[j],
                                       dHB[j - 1] if j >= 2 else None, dHB[j - 2] if j >= 3 else None, rgrads_s,
                                       deta[j - 1], rws, rws_bytes, s), "router backward")
    torch.cuda.synchronize()

    dims_o = dims_of(w)
    ref = O.routed_stack_backward(dims_o, prob.hbar.f64, [ffn_of(prob.ffn[l]) for l in range(L)], router_of(prob),
                                  [adapter_of(prob.adapter[l]) for l in range(L)], [float(e) for e in prob.eta],
                                  use_ffn, dh_out.astype(np.float64), [g.astype(np.float64) for g in dg_in])
    got = lambda t: t.cpu().numpy().astype(np.float64)
    errs = {"dh_in": _err(got(dHB[1]), ref.dh_in)}
    for name in H.ROUTER_FIELDS:
        x = got(rgrads[name])
        if name == "th1":
            x = x[:, :w.d_s + d_m + 1]
        r = getattr(ref.router, name)
        if name in ("w_q", "w_k"):
            # in these short synthetic stacks the memory read barely depends on q and k (the oracle's
            # dW_q, dW_k are ~1e-12 and ~1e-9 against dW_v's ~1e-2): both are sums of cancelling terms,
            # measured against the companion projection's scale (the per-layer tests, with informative
            # carried gradients, check them relative to themselves)
            print(f"  {name}: max|ref| {np.max(np.abs(r)):.2e}, max|gpu| {np.max(np.abs(x)):.2e}, "
                  f"max|dW_v| {np.max(np.abs(ref.router.w_v)):.2e}", flush=True)
            errs["d" + name] = float(np.max(np.abs(x - r)) / np.max(np.abs(ref.router.w_v)))
        else:
            errs["d" + name] = _err(x, r)
    eta_ref = ref.deta
    errs["deta"] = float(np.max(np.abs(got(deta)[:, 0] - eta_ref)) / np.max(np.abs(eta_ref)))
    errs["dw1"] = max(_err(got(dw1[l]), ref.dw1[l]) for l in range(L) if np.any(ref.dw1[l]))
    errs["dw2"] = max(_err(got(dw2[l]), ref.dw2[l]) for l in range(L) if np.any(ref.dw2[l]))
    errs["dlogit"] = max(_err(got(dlogit[l]), ref.dlogit[l]) for l in range(L))
    print("  errors:", {k: f"{v:.2e}" for k, v in errs.items()}, flush=True)
    assert got(deta)[0, 0] == 0.0 and got(deta)[L - 1, 0] == 0.0   # the structural zeros
    for k, v in errs.items():
        assert v <= tol, f"{k}: {v:.3e} > {tol:.0e}"
