"""Forward pins of the router's concatenation orders (Sec. 3.2).

The router state is s = [z^h; z^a] (eq:router_state): the hidden encoder's output
first, the path encoder's second; the history head reads [s; c; nu].  These tests
pin both orders in the forward pass, independently of the oracle's own code:

* a whole routed layer's router (state, memory read and write, both heads, p, m and
  the logit) is assembled from torch modules in the paper's order and compared with
  the oracle's layer;
* structural zeros: with W_hu = 0 the first d_h entries of s vanish, with W_p2 = 0
  the last d_a do;
* a planted swap of the state order inside the oracle (on the CPU) is caught.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import hero_oracle as O
from paper_2609_08189_amd import synth
from tests.oracle_inputs import adapter_of, dims_of, ffn_of, router_of, state_of

# d_h != d_a and d_s != d_m so that a swapped or misplaced slice cannot line up by accident
W = synth.Workload("order_pin", "f32", d=64, d_ff=96, d_r=8, L_R=6, d_m=8, T=20,
                   mode="threshold", d_s=14, d_h=9, d_a=5, d_e=24, d_p=12, d_head=20)


def _t(x):
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float64))


def _lin(w):
    w = np.asarray(w)
    l = torch.nn.Linear(w.shape[-1], 1 if w.ndim == 1 else w.shape[0], bias=False, dtype=torch.float64)
    with torch.no_grad():
        l.weight.copy_(_t(w.reshape(1, -1) if w.ndim == 1 else w))
    return l


def _problem(j, seed=4):
    prob = synth.make_problem(W, seed=seed, layer_j=j)
    prob.router = synth.router_weights(W, seed, std=0.3)   # gates well away from 1/2
    return prob


def torch_router(j, prob, eta):
    """The router of routed layer j assembled from torch modules, in the paper's order:
    z^h, x^path, z^a, s = [z^h; z^a], q/k/v, read then write, nu, a over [s; c; nu], p, m,
    b and the logit."""
    R = router_of(prob)
    h = _t(prob.hbar.f64)
    T = h.shape[0]
    with torch.no_grad():
        z_h = _lin(R.w_hu)(F.silu(_lin(R.w_hd)(F.rms_norm(h, (W.d,), eps=W.eps_norm))))
        delta = h - _t(prob.hbar_prev1.f64)
        delta_prev = _t(prob.hbar_prev1.f64) - _t(prob.hbar_prev2.f64)
        d_j = torch.linalg.vector_norm(delta, dim=-1)
        gamma = (delta * delta_prev).sum(-1) / (d_j * torch.linalg.vector_norm(delta_prev, dim=-1) + W.eps)
        p_prev, m_prev = _t(prob.p_hist.astype("f8")), _t(prob.m_hist.astype("f8"))
        x_path = torch.stack([torch.full((T,), j / W.L_R, dtype=torch.float64),
                              torch.full((T,), (W.L_R - j) / W.L_R, dtype=torch.float64),
                              d_j, gamma, p_prev, m_prev], dim=-1)
        z_a = _lin(R.w_p2)(F.silu(_lin(R.w_p1)(x_path)))
        s = torch.cat([z_h, z_a], dim=-1)
        q, k, v = _lin(R.w_q)(s), _lin(R.w_k)(s), _lin(R.w_v)(s)
        fq, fk = F.elu(q) + 1.0, F.elu(k) + 1.0
        S0, z0 = _t(prob.S.astype("f8")), _t(prob.zeta.astype("f8"))
        c = torch.bmm(fq[:, None, :], S0)[:, 0, :] / ((fq * z0).sum(-1, keepdim=True) + W.eps)
        rho = torch.sigmoid(torch.tensor(eta, dtype=torch.float64))
        S1 = rho * S0 + fk[:, :, None] * v[:, None, :]
        z1 = rho * z0 + fk
        ns, nc = _lin(R.w_n)(s), _lin(R.w_c)(c)
        nu = 1.0 - (ns * nc).sum(-1) / (torch.linalg.vector_norm(ns, dim=-1) *
                                        torch.linalg.vector_norm(nc, dim=-1) + W.eps)
        f_theta = torch.nn.Sequential(_lin(R.th1), torch.nn.SiLU(), _lin(R.th2))
        a = f_theta(torch.cat([s, c, nu[:, None]], dim=-1))[:, 0]
        p = torch.sigmoid(a / W.T_hist)
        m = m_prev * p
        f_psi = torch.nn.Sequential(_lin(R.ps1), torch.nn.SiLU(), _lin(R.ps2))
        b = f_psi(h)[:, 0]
    return {"s": s.numpy(), "c": c.numpy(), "logit": (a + b).numpy(), "p": p.numpy(), "m": m.numpy(),
            "S": S1.numpy(), "zeta": z1.numpy()}


def oracle_layer(j, prob):
    dims = dims_of(W)
    return O.routed_layer(j, dims, prob.hbar.f64, prob.hbar_prev1.f64, prob.hbar_prev2.f64,
                          state_of(prob), ffn_of(prob.ffn[0]), router_of(prob), adapter_of(prob.adapter[0]),
                          float(prob.eta[j - 1]), mode="threshold", tau=0.5)


def _match(res, ref):
    np.testing.assert_allclose(res.debug["s"], ref["s"], rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(res.debug["c"], ref["c"], rtol=1e-11, atol=1e-13)
    np.testing.assert_allclose(res.logit, ref["logit"], rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(res.state.p_hist, ref["p"], rtol=1e-12)
    np.testing.assert_allclose(res.state.m_hist, ref["m"], rtol=1e-12)
    np.testing.assert_allclose(res.state.S, ref["S"], rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(res.state.zeta, ref["zeta"], rtol=1e-12, atol=1e-14)


@pytest.mark.parametrize("j", [3, 5])
def test_router_forward_equals_torch_assembly_in_paper_order(j):
    prob = _problem(j)
    res = oracle_layer(j, prob)
    ref = torch_router(j, prob, float(prob.eta[j - 1]))
    # the comparison must see a live memory read and history term
    assert np.max(np.abs(ref["c"])) > 1e-2 and np.ptp(ref["logit"]) > 0.1
    _match(res, ref)


def test_state_slices_follow_their_encoders():
    """s = [z^h; z^a]: zeroing W_hu empties the first d_h entries of s and only those;
    zeroing W_p2 empties the last d_a and only those."""
    j = 3
    for name, dead, live in (("w_hu", slice(0, W.d_h), slice(W.d_h, W.d_s)),
                             ("w_p2", slice(W.d_h, W.d_s), slice(0, W.d_h))):
        prob = _problem(j)
        prob.router[name] = synth.Tensor(np.zeros_like(prob.router[name].store), "f32")
        s = oracle_layer(j, prob).debug["s"]
        assert s.shape == (W.T, W.d_s)
        assert np.all(s[:, dead] == 0.0), name
        assert np.min(np.max(np.abs(s[:, live]), axis=0)) > 1e-6, name


def test_planted_state_order_swap_is_caught(monkeypatch):
    """A swap of the state order inside the oracle ([z^a; z^h]) must fail the forward pin."""
    j = 3
    prob = _problem(j)
    ref = torch_router(j, prob, float(prob.eta[j - 1]))
    monkeypatch.setattr(O, "router_state", lambda z_h, z_a: np.concatenate([z_a, z_h], axis=-1))
    res = oracle_layer(j, prob)
    with pytest.raises(AssertionError):
        _match(res, ref)
    # the logit alone already tells the two orders apart by far more than rounding
    assert np.max(np.abs(res.logit - ref["logit"])) > 1e-3
