"""Pins for the CPU oracle: checks against what the paper and the mathematics fix.

None of these re-types an oracle formula.  Each compares the oracle with a
different computation of the same quantity: a closed form (the unrolled
memory recurrence, the rank-one first read), a library routine (torch
RMSNorm / SiLU / ELU / cosine similarity / Linear stacks, scipy's logistic),
brute force over tiny inputs, or an invariant the equations imply.
"""
import math

import numpy as np
import pytest
import scipy.special
import torch
import torch.nn.functional as F

from oracle import hero_oracle as O
from paper_2609_08189_amd import synth
from tests.oracle_inputs import adapter_of, dims_of, ffn_of, router_of

SMALL = synth.Workload("pin_small", "f32", d=64, d_ff=96, d_r=8, L_R=4, d_m=8, T=24,
                       mode="threshold", d_s=16, d_h=12, d_a=4, d_e=32, d_p=16, d_head=32)


def _problem(w=SMALL, seed=1, router_std=None):
    prob = synth.make_problem(w, seed=seed)
    if router_std is not None:
        prob.router = synth.router_weights(w, seed, std=router_std)
    return prob


def _stack(prob, w=SMALL, mode="threshold", budget=0.0, beta=None, etas=None, **kw):
    dims = dims_of(w)
    etas = prob.eta.astype("f8") if etas is None else etas
    return O.routed_stack(dims, prob.hbar.f64, [ffn_of(l) for l in prob.ffn], router_of(prob),
                          [adapter_of(l) for l in prob.adapter], etas, mode=mode,
                          budget=budget, beta=beta, **kw)


def _t(x):
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float64))


# ---------------------------------------------------------------------------
# elementary functions against library routines
# ---------------------------------------------------------------------------


def test_sigmoid_silu_phi_match_library():
    x = np.linspace(-40, 40, 2001)
    np.testing.assert_allclose(O.sigmoid(x), scipy.special.expit(x), rtol=1e-15, atol=0)
    np.testing.assert_allclose(O.silu(x), F.silu(_t(x)).numpy(), rtol=1e-14, atol=1e-300)
    # ELU(x) + 1 through the library loses the tail to cancellation (absolute error of one
    # ulp of 1.0); the oracle evaluates exp(x) directly, so it is compared in absolute terms
    # there and checked against exp itself in relative terms
    np.testing.assert_allclose(O.phi(x), (F.elu(_t(x)) + 1.0).numpy(), rtol=1e-14, atol=2.3e-16)
    neg = x <= 0
    np.testing.assert_allclose(O.phi(x)[neg], np.exp(x[neg]), rtol=1e-15, atol=0)
    # extreme logits used for forcing give exact gates
    assert O.sigmoid(np.array([1e4]))[0] == 1.0 and O.sigmoid(np.array([-1e4]))[0] == 0.0


def test_round_bf16_matches_torch():
    rng = np.random.default_rng(0)
    x = (rng.standard_normal(100000) * np.exp(rng.uniform(-20, 20, 100000))).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(O.round_bf16(x.astype("f8")), ref)
    # exact halfway points between neighbouring bf16 values: ties go to the even code
    base = torch.from_numpy(rng.standard_normal(1000).astype(np.float32)).to(torch.bfloat16)
    bits = base.view(torch.int16).numpy().astype(np.int32) & 0xFFFF
    lo = (bits.astype(np.uint32) << 16).view(np.float32).astype("f8")
    hi = ((bits.astype(np.uint32) + 1) << 16).view(np.float32).astype("f8")
    mid = (lo + hi) / 2
    ref_mid = torch.from_numpy(mid.astype(np.float32)).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(O.round_bf16(mid), ref_mid)


def test_cosine_matches_torch_far_from_eps():
    rng = np.random.default_rng(2)
    a, b = rng.standard_normal((50, 33)), rng.standard_normal((50, 33))
    ref = F.cosine_similarity(_t(a), _t(b), dim=-1).numpy()
    np.testing.assert_allclose(O.cosine_eps(a, b, 1e-6), ref, rtol=1e-6, atol=0)


def test_rmsnorm_matches_torch():
    rng = np.random.default_rng(3)
    h, w = rng.standard_normal((7, 64)) * 3, 1 + 0.1 * rng.standard_normal(64)
    ref = F.rms_norm(_t(h), (64,), weight=_t(w), eps=1e-5).numpy()
    np.testing.assert_allclose(O.rmsnorm(h, w, 1e-5), ref, rtol=1e-13)


# ---------------------------------------------------------------------------
# router sub-networks against torch module stacks (the readings' architecture)
# ---------------------------------------------------------------------------


def _mlp(w1, w2):
    l1 = torch.nn.Linear(w1.shape[1], w1.shape[0], bias=False, dtype=torch.float64)
    l2 = torch.nn.Linear(w2.shape[-1], 1 if w2.ndim == 1 else w2.shape[0], bias=False,
                         dtype=torch.float64)
    with torch.no_grad():
        l1.weight.copy_(_t(w1))
        l2.weight.copy_(_t(w2.reshape(1, -1) if w2.ndim == 1 else w2))
    return torch.nn.Sequential(l1, torch.nn.SiLU(), l2)


def test_router_subnetworks_match_torch_modules():
    prob = _problem(router_std=0.3)
    R, dims = router_of(prob), dims_of(SMALL)
    h = prob.hbar.f64
    with torch.no_grad():
        enc = torch.nn.Sequential(torch.nn.RMSNorm(SMALL.d, eps=SMALL.eps_norm,
                                                   elementwise_affine=False, dtype=torch.float64),
                                  _mlp(R.w_hd, R.w_hu))
        np.testing.assert_allclose(O.hidden_encoder(h, R, dims), enc(_t(h)).numpy(), rtol=1e-12, atol=1e-14)
        np.testing.assert_allclose(O.local_head(h, R), _mlp(R.ps1, R.ps2)(_t(h)).numpy()[:, 0],
                                   rtol=1e-12, atol=1e-14)
        x = np.random.default_rng(5).standard_normal((9, 6))
        np.testing.assert_allclose(O.path_encoder(x, R), _mlp(R.w_p1, R.w_p2)(_t(x)).numpy(),
                                   rtol=1e-12, atol=1e-14)
        s = np.random.default_rng(6).standard_normal((9, SMALL.d_s))
        c = np.random.default_rng(7).standard_normal((9, SMALL.d_m))
        nu = np.random.default_rng(8).uniform(0, 2, 9)
        a, p = O.history_head(s, c, nu, R, 0.9)
        ref = _mlp(R.th1, R.th2)(torch.cat([_t(s), _t(c), _t(nu[:, None])], -1)).numpy()[:, 0]
        np.testing.assert_allclose(a, ref, rtol=1e-12, atol=1e-14)
        np.testing.assert_allclose(p, scipy.special.expit(ref / 0.9), rtol=1e-12)
        ref_nu = 1 - F.cosine_similarity(_t(s @ R.w_n.T), _t(c @ R.w_c.T), dim=-1).numpy()
        np.testing.assert_allclose(O.history_dissimilarity(2, s, c, R, 1e-6), ref_nu, rtol=1e-6, atol=1e-9)


def test_hidden_encoder_is_scale_invariant_local_head_is_not():
    """z^h sees RMSNorm(hbar), so rescaling hbar leaves it unchanged (exactly so with a zero
    norm epsilon); f_psi sees raw hbar."""
    prob = _problem(router_std=0.3)
    R, dims = router_of(prob), dims_of(SMALL.replace(eps_norm=0.0))
    h = prob.hbar.f64
    np.testing.assert_allclose(O.hidden_encoder(3.0 * h, R, dims), O.hidden_encoder(h, R, dims),
                               rtol=1e-9, atol=1e-12)
    assert np.max(np.abs(O.local_head(3.0 * h, R) - O.local_head(h, R))) > 1e-3


# ---------------------------------------------------------------------------
# P1 / P5: the memory recurrence against its explicit sum and brute-force linear attention
# ---------------------------------------------------------------------------


def _brute_phi(x):
    return (F.elu(_t(x)) + 1.0).numpy()


@pytest.mark.parametrize("L_R", [1, 2, 5])
def test_memory_from_pairs_equals_the_recurrence(L_R):
    """The depth-history state (the pairs of layers 1..n, weighted by decay products) equals
    the stack's memory after n layers of the recurrence, for every n."""
    w = SMALL.replace(L_R=L_R, T=4)
    prob = _problem(w, router_std=0.3)
    etas = np.linspace(-1.5, 2.5, L_R)
    res = _stack(prob, w, etas=etas)
    rhos = O.sigmoid(etas)
    phik = np.stack([_brute_phi(L.debug["k"]) for L in res.layers], axis=1)
    v = np.stack([L.debug["v"] for L in res.layers], axis=1)
    S, zeta = O.memory_from_pairs(phik, v, rhos)
    np.testing.assert_allclose(S, res.state.S, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(zeta, res.state.zeta, rtol=1e-12, atol=1e-14)
    # and for a prefix of n < L_R layers, against the state the next layer reads (its c)
    for n in range(1, L_R):
        Sn, zn = O.memory_from_pairs(phik[:, :n], v[:, :n], rhos[:n])
        c = O.memory_read(res.layers[n].debug["q"], Sn, zn, w.eps)
        np.testing.assert_allclose(c, res.layers[n].debug["c"], rtol=1e-10, atol=1e-12)
    S0, z0 = O.memory_from_pairs(phik[:, :0], v[:, :0], rhos[:0])
    assert not S0.any() and not z0.any()


@pytest.mark.parametrize("L_R", [1, 2, 3, 4, 8])
@pytest.mark.parametrize("rho_one", [False, True])
def test_memory_equals_explicit_decayed_sum(L_R, rho_one):
    w = SMALL.replace(L_R=L_R, T=5)
    prob = _problem(w, router_std=0.3)
    etas = np.full(L_R, 60.0) if rho_one else np.linspace(-1.0, 3.0, L_R)
    res = _stack(prob, w, etas=etas)
    rhos = [1.0 / (1.0 + math.exp(-e)) for e in etas]
    for t in range(w.T):
        ks = [_brute_phi(L.debug["k"][t]) for L in res.layers]
        vs = [L.debug["v"][t] for L in res.layers]
        qs = [_brute_phi(L.debug["q"][t]) for L in res.layers]
        for j in range(1, L_R + 1):
            # state after layer j: sum_{i<=j} prod_{i<m<=j} rho_m phi(k_i) v_i^T
            S = np.zeros((w.d_m, w.d_m))
            z = np.zeros(w.d_m)
            for i in range(1, j + 1):
                wgt = 1.0
                for mm in range(i + 1, j + 1):
                    wgt *= rhos[mm - 1]
                for a in range(w.d_m):
                    z[a] += wgt * ks[i - 1][a]
                    for b in range(w.d_m):
                        S[a, b] += wgt * ks[i - 1][a] * vs[i - 1][b]
            if j == L_R:
                np.testing.assert_allclose(res.state.S[t], S, rtol=1e-12, atol=1e-14)
                np.testing.assert_allclose(res.state.zeta[t], z, rtol=1e-12, atol=1e-14)
            # read at layer j uses only layers i < j: brute-force linear attention over depth
            num = np.zeros(w.d_m)
            den = 0.0
            for i in range(1, j):
                wgt = 1.0
                for mm in range(i + 1, j):
                    wgt *= rhos[mm - 1]
                sc = wgt * float(np.dot(qs[j - 1], ks[i - 1]))
                num += sc * vs[i - 1]
                den += sc
            c_ref = num / (den + w.eps)
            np.testing.assert_allclose(res.layers[j - 1].debug["c"][t], c_ref, rtol=1e-11, atol=1e-15)


def test_first_read_is_zero_second_read_is_rank_one():
    prob = _problem(router_std=0.3)
    res = _stack(prob)
    L1, L2 = res.layers[0], res.layers[1]
    assert np.all(L1.debug["c"] == 0.0) and np.all(L1.debug["nu"] == 0.0)
    # c_2 = v_1 * w / (w + eps) with w = phi(q_2) . phi(k_1): the direction of v_1 exactly
    wgt = np.sum(_brute_phi(L2.debug["q"]) * _brute_phi(L1.debug["k"]), axis=-1)
    np.testing.assert_allclose(L2.debug["c"], L1.debug["v"] * (wgt / (wgt + SMALL.eps))[:, None],
                               rtol=1e-12, atol=1e-15)


def test_first_layer_ignores_key_and_value_weights():
    """Read-before-write: layer 1's logits cannot depend on W_k, W_v; layer 2's must."""
    prob = _problem(router_std=0.3)
    base = _stack(prob)
    prob2 = _problem(router_std=0.3)
    for name in ("w_k", "w_v"):
        prob2.router[name] = synth.Tensor(prob2.router[name].store * np.float32(-1.7), "f32")
    other = _stack(prob2)
    np.testing.assert_array_equal(base.layers[0].logit, other.layers[0].logit)
    assert np.max(np.abs(base.layers[1].logit - other.layers[1].logit)) > 1e-6


# ---------------------------------------------------------------------------
# P6 / P7: path-vector boundary values and range invariants
# ---------------------------------------------------------------------------


def test_path_vector_boundaries():
    prob = _problem(router_std=0.3)
    res = _stack(prob)
    L_R = SMALL.L_R
    x1 = res.layers[0].debug["x_path"]
    np.testing.assert_array_equal(x1, np.tile([1 / L_R, 1 - 1 / L_R, 0, 0, 1, 1], (SMALL.T, 1)))
    assert np.all(res.layers[1].debug["gamma"] == 0.0) and np.all(res.layers[1].debug["d"] > 0)
    for j, L in enumerate(res.layers, start=1):
        r, q = L.debug["x_path"][0, :2]
        assert r == j / L_R and q == (L_R - j) / L_R and abs(r + q - 1) < 1e-15
    # x_path carries the previous layer's history scores, p first, then m
    for jm1, L in enumerate(res.layers[1:]):
        prev = res.layers[jm1].state
        np.testing.assert_array_equal(L.debug["x_path"][:, 4], prev.p_hist)
        np.testing.assert_array_equal(L.debug["x_path"][:, 5], prev.m_hist)
    # gamma_j is the cosine of consecutive residual transitions (library cosine, j >= 3);
    # the transitions here are small, so eps is shrunk until it is negligible against them
    w_small_eps = SMALL.replace(eps=1e-13)
    res = _stack(prob, w_small_eps)
    hb = [prob.hbar.f64] + [L.h for L in res.layers]
    for j in range(3, L_R + 1):
        dj = hb[j - 1] - hb[j - 2]
        djm1 = hb[j - 2] - hb[j - 3]
        ref = F.cosine_similarity(_t(dj), _t(djm1), dim=-1).numpy()
        np.testing.assert_allclose(res.layers[j - 1].debug["gamma"], ref, rtol=1e-6, atol=1e-9)
        assert np.max(np.abs(ref)) > 1e-3
    # d_j is the distance between consecutive post-attention states (hbar_{j+1} = h_j)
    h_prev = prob.hbar.f64
    for L, Lnext in zip(res.layers[:-1], res.layers[1:]):
        brute = np.array([math.sqrt(sum((a - b) ** 2 for a, b in zip(L.h[t], h_prev[t])))
                          for t in range(SMALL.T)])
        np.testing.assert_allclose(Lnext.debug["d"], brute, rtol=1e-12)
        h_prev = L.h


def test_range_invariants_over_seeds():
    for seed in range(4):
        w = SMALL.replace(L_R=6)
        prob = _problem(w, seed=seed, router_std=0.15)
        res = _stack(prob, w)
        m_prev = np.ones(w.T)
        vmax = np.zeros((w.T, w.d_m))
        for j, L in enumerate(res.layers, start=1):
            g = L.debug
            assert np.all(np.abs(g["gamma"]) <= 1.0 + 1e-12)
            assert np.all((g["nu"] >= -1e-12) & (g["nu"] <= 2 + 1e-12))
            assert np.all((L.state.p_hist > 0) & (L.state.p_hist < 1))   # sigma of a finite logit
            assert np.all(L.state.m_hist <= m_prev + 1e-15)
            assert np.all(L.state.zeta > 0)
            if j > 1:
                # c is a non-negative combination of past v with total weight < 1
                assert np.all(np.abs(g["c"]) <= vmax + 1e-12)
            vmax = np.maximum(vmax, np.abs(g["v"]))
            m_prev = L.state.m_hist


# ---------------------------------------------------------------------------
# P2 / P3 / P8: routing special cases that reduce to the dense backbone or the adapter
# ---------------------------------------------------------------------------


def _dense_block_torch(h, ffn, eps):
    u = F.rms_norm(_t(h), (h.shape[1],), weight=_t(ffn.norm_w), eps=eps)
    y = F.linear(F.silu(F.linear(u, _t(ffn.w_gate))) * F.linear(u, _t(ffn.w_up)), _t(ffn.w_down))
    return (_t(h) + y).numpy()


def _adapter_block_torch(h, ffn, ad, eps):
    u = F.rms_norm(_t(h), (h.shape[1],), weight=_t(ffn.norm_w), eps=eps)
    return (_t(h) + F.linear(F.silu(F.linear(u, _t(ad.w1))), _t(ad.w2))).numpy()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_all_full_routing_is_the_dense_backbone(dtype):
    w = SMALL.replace(dtype=dtype)
    prob = _problem(w)
    res = _stack(prob, w, beta=np.full(w.T, 1e4))
    h = prob.hbar.f64
    for j, L in enumerate(res.layers):
        assert L.use_ffn.all() and np.all(L.gate == 1.0)
        ref = O.round_io(_dense_block_torch(h, ffn_of(prob.ffn[j]), w.eps_norm), dtype)
        if dtype == "f32":
            np.testing.assert_allclose(L.h, ref, rtol=1e-6, atol=1e-6)
        else:
            # both round the same fp64 value; allow one bf16 ulp where fp64 sums differ at a tie
            np.testing.assert_allclose(L.h, ref, rtol=2 ** -7, atol=0)
        h = L.h


def test_all_full_routing_single_layer_exact():
    prob = _problem()
    res = _stack(prob, SMALL.replace(L_R=4), beta=np.full(SMALL.T, 1e4))
    layer = O.routed_layer(1, dims_of(SMALL), prob.hbar.f64, None, None, O.State.initial(SMALL.T, SMALL.d_m),
                           ffn_of(prob.ffn[0]), router_of(prob), adapter_of(prob.adapter[0]), prob.eta[0],
                           mode="threshold", beta=np.full(SMALL.T, 1e4), round_output=False)
    ref = _dense_block_torch(prob.hbar.f64, ffn_of(prob.ffn[0]), SMALL.eps_norm)
    np.testing.assert_allclose(layer.h, ref, rtol=1e-12, atol=1e-13)
    assert res.layers[0].use_ffn.all()


def test_all_adapter_routing_is_the_adapter_path():
    prob = _problem()
    layer = O.routed_layer(1, dims_of(SMALL), prob.hbar.f64, None, None, O.State.initial(SMALL.T, SMALL.d_m),
                           ffn_of(prob.ffn[0]), router_of(prob), adapter_of(prob.adapter[0]), prob.eta[0],
                           mode="threshold", beta=np.full(SMALL.T, -1e4), round_output=False)
    assert not layer.use_ffn.any() and np.all(layer.gate == 0.0)
    ref = _adapter_block_torch(prob.hbar.f64, ffn_of(prob.ffn[0]), adapter_of(prob.adapter[0]), SMALL.eps_norm)
    np.testing.assert_allclose(layer.h, ref, rtol=1e-12, atol=1e-13)


def test_gate_scales_the_taken_branch():
    """Unforced routing: FFN rows are hbar + g*dense, adapter rows hbar + (1-g)*adapter."""
    prob = _problem(router_std=0.5)
    hb = prob.hbar.f64
    layer = O.routed_layer(1, dims_of(SMALL), hb, None, None, O.State.initial(SMALL.T, SMALL.d_m),
                           ffn_of(prob.ffn[0]), router_of(prob), adapter_of(prob.adapter[0]), prob.eta[0],
                           mode="threshold", round_output=False)
    assert 0 < layer.use_ffn.sum() < SMALL.T
    dense = _dense_block_torch(hb, ffn_of(prob.ffn[0]), SMALL.eps_norm) - hb
    adap = _adapter_block_torch(hb, ffn_of(prob.ffn[0]), adapter_of(prob.adapter[0]), SMALL.eps_norm) - hb
    for t in range(SMALL.T):
        g = layer.gate[t]
        ref = hb[t] + (g * dense[t] if layer.use_ffn[t] else (1 - g) * adap[t])
        np.testing.assert_allclose(layer.h[t], ref, rtol=1e-12, atol=1e-13)
        assert layer.use_ffn[t] == (g >= 0.5)


def test_zero_heads_tie_goes_to_ffn():
    prob = _problem(router_std=0.3)
    prob.router["th2"] = synth.Tensor(np.zeros_like(prob.router["th2"].store), "f32")
    prob.router["ps2"] = synth.Tensor(np.zeros_like(prob.router["ps2"].store), "f32")
    res = _stack(prob)
    hb = prob.hbar.f64
    for j, L in enumerate(res.layers):
        assert np.all(L.logit == 0.0) and np.all(L.gate == 0.5) and L.use_ffn.all()
        assert np.all(L.state.p_hist == 0.5)
        dense = _dense_block_torch(hb, ffn_of(prob.ffn[j]), SMALL.eps_norm) - hb
        np.testing.assert_allclose(L.h, (hb + 0.5 * dense).astype(np.float32), rtol=1e-6, atol=1e-6)
        hb = L.h
    np.testing.assert_allclose(res.state.m_hist, 0.5 ** SMALL.L_R, rtol=1e-15)


# ---------------------------------------------------------------------------
# P4: skip budget; P9: token independence
# ---------------------------------------------------------------------------


@pytest.mark.parametrize("budget", [0.0, 0.27, 0.5, 0.9, 1.0])
def test_budget_selects_exact_count_of_smallest(budget):
    rng = np.random.default_rng(11)
    T = 157
    ell = np.round(rng.standard_normal(T), 1)       # many exact ties
    use_ffn, lam = O.decide_budget(ell, budget)
    k = int(math.floor(budget * T + 0.5))
    assert (~use_ffn).sum() == k
    skip = [t for t in range(T) if not use_ffn[t]]
    keep = [t for t in range(T) if use_ffn[t]]
    for a in skip:
        for f in keep:
            assert (ell[a], a) < (ell[f], f)
    if keep:
        assert lam == float(np.float32(min(ell[f] for f in keep)))
    else:
        assert lam == math.inf


def test_budget_realized_in_stack():
    w = synth.WORKLOADS["tiny_f32_stack"]
    prob = synth.make_problem(w, seed=0)
    res = O.routed_stack(dims_of(w), prob.hbar.f64, [ffn_of(l) for l in prob.ffn], router_of(prob),
                         [adapter_of(l) for l in prob.adapter], prob.eta.astype("f8"),
                         mode="budget", budget=w.budget)
    for L in res.layers:
        assert (~L.use_ffn).sum() == 17


def test_token_permutation_equivariance():
    prob = _problem(router_std=0.5)
    base = _stack(prob)
    perm = np.random.default_rng(4).permutation(SMALL.T)
    prob2 = _problem(router_std=0.5)
    prob2.hbar = synth.Tensor(prob.hbar.store[perm], "f32")
    other = _stack(prob2)
    np.testing.assert_array_equal(other.h, base.h[perm])
    np.testing.assert_array_equal(other.state.S, base.state.S[perm])
    # a token subset gives the same rows as the full batch
    sub = _problem(router_std=0.5)
    rows = np.array([3, 5, 17])
    sub.hbar = synth.Tensor(prob.hbar.store[rows], "f32")
    np.testing.assert_array_equal(_stack(sub).h, base.h[rows])


def test_teacher_forcing_follows_given_mask():
    prob = _problem(router_std=0.5)
    base = _stack(prob)
    flip = [~L.use_ffn for L in base.layers]
    forced = _stack(prob, forced_ffn=flip)
    for L, f in zip(forced.layers, flip):
        np.testing.assert_array_equal(L.use_ffn, f)
    np.testing.assert_array_equal(forced.layers[0].own_ffn, base.layers[0].use_ffn)


def test_logit_bias_enters_the_gate_only():
    """beta shifts the gate logit; the history score p = sigma(a / T_hist) is unaffected."""
    prob = _problem(router_std=0.15)
    base = _stack(prob)
    for beta in (1e4, -1e4, 0.7):
        other = _stack(prob, beta=np.full(SMALL.T, beta))
        L0, L1 = base.layers[0], other.layers[0]
        np.testing.assert_array_equal(L1.state.p_hist, L0.state.p_hist)
        np.testing.assert_array_equal(L1.state.m_hist, L0.state.m_hist)
        np.testing.assert_allclose(L1.logit, L0.logit + beta, rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(L1.gate, scipy.special.expit(L0.logit + beta), rtol=1e-12, atol=1e-300)
    a = base.layers[0].debug["a"]
    np.testing.assert_allclose(base.layers[0].state.p_hist, scipy.special.expit(a / SMALL.T_hist), rtol=1e-13)


def test_bf16_state_is_the_rounded_memory():
    """S stored in bf16: every stored element is a bf16 value; at the first layer it is exactly
    torch's bf16 rounding of the exact outer product; over the stack it stays within the rounding
    error accumulated by one half-ulp per layer, and the logits barely move."""
    w16 = SMALL.replace(state_dtype="bf16")
    prob = _problem(router_std=0.3)
    exact = _stack(prob, SMALL)
    rounded = _stack(prob, w16)
    for L in rounded.layers:
        S = L.state.S
        np.testing.assert_array_equal(_t(S).to(torch.bfloat16).double().numpy(), S)
    np.testing.assert_array_equal(rounded.layers[0].state.S,
                                  _t(exact.layers[0].state.S).to(torch.bfloat16).double().numpy())
    for j, (Le, Lr) in enumerate(zip(exact.layers, rounded.layers), start=1):
        scale = np.abs(Le.state.S).max()
        assert np.abs(Lr.state.S - Le.state.S).max() <= j * 2.0 ** -8 * scale
        assert Lr.state.S is not Le.state.S and not np.array_equal(Lr.state.S, Le.state.S)
        if j == 1:   # the first layer reads no memory: same zeta and logits
            np.testing.assert_array_equal(Lr.state.zeta, Le.state.zeta)
            np.testing.assert_array_equal(Lr.logit, Le.logit)
        assert np.abs(Lr.logit - Le.logit).max() < 5e-3 * np.abs(Le.logit).max()
