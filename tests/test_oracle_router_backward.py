"""Pins for the oracle's backward through the whole routed stack: the gradients that reach the
router through the gate scaling (Sec. 3.1, the remark after eq:ffn_route) and flow through its
heads, depth memory, encoders and path features (Sec. 3.2) across routed layers, together with
the adapters' and the input's (Sec. 3.3: adapters, state encoders, depth memory and router
heads are the trained parts).

Every analytic gradient is checked element by element against central finite differences of
the float64 forward (routed_stack_f64, the same equations as routed_stack without rounding) on a
tiny stack of four layers with both branches present; structural zeros that follow from the
equations (the first layer's memory decay multiplies an empty memory, the last layer's write is
never read, a one-layer stack never reads its memory) are checked exactly."""
import numpy as np
import pytest

from oracle import hero_oracle as O

D, DFF, DR, T, L = 12, 16, 4, 5, 4
DIMS = O.Dims(d=D, d_ff=DFF, d_r=DR, L_R=L, d_m=4, d_s=8, d_h=6, d_a=2, d_e=8, d_p=6, d_head=10)
SHAPES = {"w_hd": (8, D), "w_hu": (6, 8), "w_p1": (6, 6), "w_p2": (2, 6), "w_q": (4, 8), "w_k": (4, 8),
          "w_v": (4, 8), "w_n": (4, 8), "w_c": (4, 4), "th1": (10, 8 + 4 + 1), "th2": (10,),
          "ps1": (10, D), "ps2": (10,)}


def _problem(seed=0, dims=DIMS, all_ffn=False):
    rng = np.random.default_rng(seed)
    nrm = lambda shape, s: s * rng.standard_normal(shape)
    R = O.RouterParams(**{k: nrm(sh, 0.6 / np.sqrt(sh[-1]) if len(sh) == 2 else 0.5)
                          for k, sh in SHAPES.items()})
    ffns = [O.FFNParams(norm_w=1.0 + nrm(D, 0.2), w_gate=nrm((DFF, D), 0.4), w_up=nrm((DFF, D), 0.4),
                        w_down=nrm((D, DFF), 0.3)) for _ in range(dims.L_R)]
    ads = [O.AdapterParams(w1=nrm((DR, D), 0.5), w2=nrm((D, DR), 0.5)) for _ in range(dims.L_R)]
    h_in = rng.standard_normal((T, D)) * rng.uniform(0.5, 2.0, (T, 1))
    etas = np.array([0.3, -0.5, 1.0, 0.2][:dims.L_R])
    use = [np.ones(T, bool) if all_ffn else rng.uniform(size=T) < 0.6 for _ in range(dims.L_R)]
    if not all_ffn:
        use[0][:2] = [True, False]                  # both branches at every layer
        for u in use[1:]:
            u[:2] = [False, True]
    dh = rng.standard_normal((T, D))
    dg = [rng.standard_normal(T) for _ in range(dims.L_R)]
    return R, ffns, ads, h_in, etas, use, dh, dg


def _J(dims, R, ffns, ads, h_in, etas, use, dh, dg):
    tr = O.routed_stack_f64(dims, h_in, ffns, R, ads, etas, use)
    return float(np.sum(dh * tr.h_out) + sum(np.dot(g, lr.gate) for g, lr in zip(dg, tr.layers)))


def _fd(f, x, h=1e-4):
    """Central differences over every element of x (in place).  h = 1e-4 keeps the rounding of a
    loss of size ~10 (about 1e-16 * 10 / h) and the O(h^2) truncation both near 1e-9."""
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


def _close(a, b, rtol=1e-6, atol=1e-9):
    scale = max(np.max(np.abs(b)), 1e-12)
    assert np.max(np.abs(a - b)) <= rtol * scale + atol, (np.max(np.abs(a - b)), scale)


@pytest.fixture(scope="module")
def case():
    P = _problem()
    return P, O.routed_stack_backward(DIMS, P[3], P[1], P[0], P[2], P[4], P[5], P[6], P[7])


def test_gates_are_not_saturated_and_memory_is_read(case):
    (R, ffns, ads, h_in, etas, use, dh, dg), _ = case
    tr = O.routed_stack_f64(DIMS, h_in, ffns, R, ads, etas, use)
    g = np.array([lr.gate for lr in tr.layers])
    assert 0.02 < g.min() and g.max() < 0.98
    assert all(np.abs(lr.debug["c"]).max() > 1e-3 for lr in tr.layers[1:])


@pytest.mark.parametrize("name", list(SHAPES))
def test_router_weight_gradients_match_finite_differences(case, name):
    (R, ffns, ads, h_in, etas, use, dh, dg), grad = case
    x = getattr(R, name)
    fd = _fd(lambda: _J(DIMS, R, ffns, ads, h_in, etas, use, dh, dg), x)
    _close(getattr(grad.router, name), fd)
    assert np.max(np.abs(fd)) > 1e-6          # the weight does reach the loss


def test_input_and_decay_gradients_match_finite_differences(case):
    (R, ffns, ads, h_in, etas, use, dh, dg), grad = case
    J = lambda: _J(DIMS, R, ffns, ads, h_in, etas, use, dh, dg)
    _close(grad.dh_in, _fd(J, h_in))
    _close(grad.deta, _fd(J, etas), rtol=1e-5)


def test_adapter_gradients_match_finite_differences(case):
    (R, ffns, ads, h_in, etas, use, dh, dg), grad = case
    J = lambda: _J(DIMS, R, ffns, ads, h_in, etas, use, dh, dg)
    for l in range(L):
        _close(grad.dw1[l], _fd(J, ads[l].w1))
        _close(grad.dw2[l], _fd(J, ads[l].w2))


def test_structural_zeros_of_the_memory_decay(case):
    """rho_1 multiplies the empty initial memory and the last layer's write is never read: their
    decay gradients are exactly zero; the layers in between have nonzero ones."""
    _, grad = case
    assert grad.deta[0] == 0.0 and grad.deta[-1] == 0.0
    assert np.all(np.abs(grad.deta[1:-1]) > 1e-8)


def test_one_layer_stack_never_reads_its_memory():
    """With L_R = 1 the only read is of the initial (zero) memory and nu = 0: no gradient reaches
    W_q, W_k, W_v, W_n, W_c, eta, or the c and nu inputs of f_theta."""
    dims = O.Dims(**{**DIMS.__dict__, "L_R": 1})
    R, ffns, ads, h_in, etas, use, dh, dg = _problem(seed=3, dims=dims)
    grad = O.routed_stack_backward(dims, h_in, ffns, R, ads, etas, use, dh, dg)
    for name in ("w_q", "w_k", "w_v", "w_n", "w_c"):
        assert not np.any(getattr(grad.router, name)), name
    assert not np.any(grad.router.th1[:, dims.d_s:])
    assert np.any(grad.router.th1[:, :dims.d_s]) and grad.deta[0] == 0.0


def test_last_layer_hand_off_equals_the_block_backward(case):
    """The gradient reaching the last router through its gate is the routed block's dL/dlogit for
    the loss's dL/dh_out and dL/dg alone (no later layer exists)."""
    (R, ffns, ads, h_in, etas, use, dh, dg), grad = case
    tr = O.routed_stack_f64(DIMS, h_in, ffns, R, ads, etas, use)
    bg = O.routed_block_backward(tr.hbars[-1], tr.layers[-1].gate, use[-1], ffns[-1], ads[-1], DIMS, dh, dg[-1])
    np.testing.assert_array_equal(grad.dlogit[-1], bg.dlogit)


def test_all_ffn_stack_gives_the_adapters_nothing():
    R, ffns, ads, h_in, etas, use, dh, dg = _problem(seed=5, all_ffn=True)
    grad = O.routed_stack_backward(DIMS, h_in, ffns, R, ads, etas, use, dh, dg)
    assert all(not np.any(a) for a in grad.dw1) and all(not np.any(a) for a in grad.dw2)
    assert np.any(grad.router.ps1) and np.any(grad.router.w_q)


def test_forward_matches_the_routed_stack_before_rounding():
    """routed_stack_f64 is routed_stack's computation: with fp32 I/O and the same forced branches,
    the two agree to the float32 rounding routed_stack applies at each layer boundary."""
    R, ffns, ads, h_in, etas, use, dh, dg = _problem(seed=7)
    tr = O.routed_stack_f64(DIMS, h_in, ffns, R, ads, etas, use)
    ref = O.routed_stack(DIMS, h_in, ffns, R, ads, etas, mode="threshold", forced_ffn=use)
    np.testing.assert_allclose(tr.h_out, ref.h, rtol=1e-5, atol=1e-5)
