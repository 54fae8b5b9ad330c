"""Pins for the oracle's training-side backward: the routed block through the gate scaling
(Sec. 3.1, eq:ffn_route and the remark after it) and the utilisation penalty (Sec. 3.3,
Eq. 17-18).

The analytic gradients are checked against central finite differences of the oracle's
forward (routed_block, itself tied to routed_layer's output), element by element on a tiny
problem with both branches present; the penalty against finite differences and its closed
form for constant gates."""
import numpy as np
import pytest

from oracle import hero_oracle as O
from paper_2609_08189_amd import synth
from tests.oracle_inputs import adapter_of, dims_of, ffn_of, router_of, state_of

D, DFF, DR, T = 16, 24, 4, 7


def _tiny(seed=0):
    rng = np.random.default_rng(seed)
    dims = O.Dims(d=D, d_ff=DFF, d_r=DR, L_R=4, d_m=8)
    ffn = O.FFNParams(norm_w=1.0 + 0.2 * rng.standard_normal(D),
                      w_gate=0.4 * rng.standard_normal((DFF, D)),
                      w_up=0.4 * rng.standard_normal((DFF, D)),
                      w_down=0.4 * rng.standard_normal((D, DFF)))
    ad = O.AdapterParams(w1=0.5 * rng.standard_normal((DR, D)), w2=0.5 * rng.standard_normal((D, DR)))
    hbar = rng.standard_normal((T, D)) * rng.uniform(0.5, 2.0, (T, 1))
    gate = rng.uniform(0.05, 0.95, T)
    use_ffn = np.array([1, 0, 1, 1, 0, 0, 1], dtype=bool)
    dh = rng.standard_normal((T, D))
    dgate_in = rng.standard_normal(T)
    return dims, ffn, ad, hbar, gate, use_ffn, dh, dgate_in


def _objective(dims, ffn, ad, hbar, gate, use_ffn, dh, dgate_in):
    """J = <dh, h_out> + <dgate_in, g>: its gradient is what routed_block_backward returns."""
    return float(np.sum(dh * O.routed_block(hbar, gate, use_ffn, ffn, ad, dims)) + np.dot(dgate_in, gate))


def _fd(f, x, h=1e-6):
    """Central differences of the scalar f() over every element of the array x (in place)."""
    g = np.zeros_like(x)
    it = np.nditer(x, flags=["multi_index"])
    for _ in it:
        i = it.multi_index
        v = x[i]
        x[i] = v + h
        fp = f()
        x[i] = v - h
        fm = f()
        x[i] = v
        g[i] = (fp - fm) / (2 * h)
    return g


def _close(a, b, rtol=1e-6):
    scale = max(np.max(np.abs(b)), 1e-12)
    assert np.max(np.abs(a - b)) <= rtol * scale, (np.max(np.abs(a - b)), scale)


@pytest.mark.parametrize("seed", [0, 1])
def test_block_gradients_match_finite_differences(seed):
    dims, ffn, ad, hbar, gate, use_ffn, dh, dgate_in = _tiny(seed)
    grad = O.routed_block_backward(hbar, gate, use_ffn, ffn, ad, dims, dh, dgate_in)
    J = lambda: _objective(dims, ffn, ad, hbar, gate, use_ffn, dh, dgate_in)
    _close(grad.dhbar, _fd(J, hbar))
    _close(grad.dgate, _fd(J, gate))
    _close(grad.dw1, _fd(J, ad.w1))
    _close(grad.dw2, _fd(J, ad.w2))
    # the logit gradient: g = sigma(logit), the branch held fixed
    logit = np.log(gate / (1 - gate))
    Jl = lambda: _objective(dims, ffn, ad, hbar, O.sigmoid(logit), use_ffn, dh, dgate_in)
    _close(grad.dlogit, _fd(Jl, logit))


def test_frozen_backbone_gets_no_adapter_gradient_from_ffn_tokens():
    """With every token on the FFN branch the adapter is never used: dW = 0, and dL/dg is the
    inner product of the upstream gradient with the FFN output alone."""
    dims, ffn, ad, hbar, gate, _, dh, _ = _tiny(3)
    use_ffn = np.ones(T, dtype=bool)
    grad = O.routed_block_backward(hbar, gate, use_ffn, ffn, ad, dims, dh)
    assert not grad.dw1.any() and not grad.dw2.any()
    y = (O.routed_block(hbar, np.ones(T), use_ffn, ffn, ad, dims) - hbar)
    np.testing.assert_allclose(grad.dgate, np.sum(dh * y, axis=1), rtol=1e-12)


def test_gate_half_splits_the_scaling_evenly():
    """At g = 1/2 both branches are scaled by 1/2, so flipping every decision leaves the
    residual's share and halves of the branch gradients; the logit gradient is dg / 4."""
    dims, ffn, ad, hbar, _, use_ffn, dh, _ = _tiny(4)
    gate = np.full(T, 0.5)
    grad = O.routed_block_backward(hbar, gate, use_ffn, ffn, ad, dims, dh)
    np.testing.assert_allclose(grad.dlogit, grad.dgate / 4, rtol=1e-14)


def test_block_output_is_the_routed_layer_output():
    """routed_block with the layer's own gate and decision reproduces routed_layer's h."""
    w = synth.Workload("blk", "f32", d=64, d_ff=96, d_r=8, L_R=5, d_m=8, T=24, mode="budget",
                       budget=0.4, d_s=16, d_h=12, d_a=4, d_e=32, d_p=16, d_head=32, layer_j=3)
    prob = synth.make_problem(w, seed=2, layer_j=3)
    res = O.routed_layer(3, dims_of(w), prob.hbar.f64, prob.hbar_prev1.f64, prob.hbar_prev2.f64,
                         state_of(prob), ffn_of(prob.ffn[0]), router_of(prob),
                         adapter_of(prob.adapter[0]), float(prob.eta[2]), mode="budget",
                         budget=0.4, round_output=False)
    assert 0 < res.use_ffn.sum() < w.T
    h = O.routed_block(prob.hbar.f64, res.gate, res.use_ffn, ffn_of(prob.ffn[0]),
                       adapter_of(prob.adapter[0]), dims_of(w))
    np.testing.assert_allclose(h, res.h, rtol=0, atol=1e-12)


def test_rmsnorm_backward_matches_finite_differences():
    rng = np.random.default_rng(9)
    h = rng.standard_normal((3, 10))
    w = rng.uniform(0.5, 1.5, 10)
    du = rng.standard_normal((3, 10))
    J = lambda: float(np.sum(du * O.rmsnorm(h, w, 1e-5)))
    _close(O.rmsnorm_backward(h, w, 1e-5, du), _fd(J, h))


def test_skip_penalty_matches_finite_differences():
    rng = np.random.default_rng(5)
    L_R, B, S = 3, 2, 5
    g = rng.uniform(0.05, 0.95, (L_R, B * S))
    val, grad = O.skip_penalty(g, B, S, alpha=0.7)
    _close(grad, _fd(lambda: O.skip_penalty(g, B, S, alpha=0.7)[0], g))
    # the last position of every sequence has no next token: no penalty, no gradient
    last = np.arange(B) * S + S - 1
    assert not grad[:, last].any()
    g2 = g.copy()
    g2[:, last] = rng.uniform(0, 1, (L_R, B))
    assert O.skip_penalty(g2, B, S, alpha=0.7)[0] == val


def test_skip_penalty_constant_gates():
    """Every gate c: each position's sum is L_R c, so L_skip = (L_R c)^2 and the gradient at a
    position with a next token is 2 L_R c / (B (S - 1))."""
    L_R, B, S, c = 4, 3, 6, 0.3
    val, grad = O.skip_penalty(np.full((L_R, B * S), c), B, S)
    assert val == pytest.approx((L_R * c) ** 2, rel=1e-14)
    pos = np.ones(B * S, dtype=bool)
    pos[np.arange(B) * S + S - 1] = False
    np.testing.assert_allclose(grad[:, pos], 2 * L_R * c / (B * (S - 1)), rtol=1e-14)
    assert O.skip_penalty(np.full((L_R, B), c), B, 1) == (0.0, pytest.approx(np.zeros((L_R, B))))
