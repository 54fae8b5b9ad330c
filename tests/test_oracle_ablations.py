"""Pins for the oracle's router ablations (Table 3, Sec. 4.3).

Each ablation bit is compared with the full router run on weights that make the removed
component contribute exactly nothing (zeroed columns or output rows of the sub-network
that carried it), and with invariances: an ablated router's logit does not move when the
inputs it no longer sees are changed.  Neither re-types the ablated code path.
"""
import dataclasses

import numpy as np
import pytest

from oracle import hero_oracle as O
from paper_2609_08189_amd import synth
from tests.oracle_inputs import adapter_of, dims_of, ffn_of, router_of, state_of

W = synth.Workload("abl_small", "f32", d=64, d_ff=96, d_r=8, L_R=5, d_m=8, T=32,
                   mode="threshold", d_s=16, d_h=12, d_a=4, d_e=32, d_p=16, d_head=32)


def _problem(seed=3):
    prob = synth.make_problem(W, seed=seed)
    prob.router = synth.router_weights(W, seed, std=0.3)   # router effects well above rounding
    return prob


def _stack(prob, R=None, ablation=0, w=W):
    return O.routed_stack(dims_of(w), prob.hbar.f64, [ffn_of(l) for l in prob.ffn],
                          router_of(prob) if R is None else R,
                          [adapter_of(l) for l in prob.adapter], prob.eta.astype("f8"),
                          mode="threshold", tau=0.5, ablation=ablation)


def _logits(res):
    return np.stack([L.logit for L in res.layers])


def _assert_same_path(a, b):
    np.testing.assert_array_equal(_logits(a), _logits(b))
    for La, Lb in zip(a.layers, b.layers):
        np.testing.assert_array_equal(La.use_ffn, Lb.use_ffn)
    np.testing.assert_array_equal(a.h, b.h)


def _differs(a, b, min_diff=1e-3):
    return np.max(np.abs(_logits(a) - _logits(b))) > min_diff


def test_no_aux_state_is_a_zero_path_encoder():
    prob = _problem()
    R = router_of(prob)
    abl = _stack(prob, ablation=O.NO_AUX_STATE)
    zeroed = _stack(prob, dataclasses.replace(R, w_p2=np.zeros_like(R.w_p2)))
    _assert_same_path(abl, zeroed)
    np.testing.assert_array_equal(abl.state.S, zeroed.state.S)
    np.testing.assert_array_equal(abl.state.m_hist, zeroed.state.m_hist)
    assert _differs(abl, _stack(prob))


def test_no_pos_state_drops_the_first_four_path_features():
    prob = _problem()
    R = router_of(prob)
    w_p1 = R.w_p1.copy()
    w_p1[:, :4] = 0.0          # columns of r, q_rem, d, gamma (p and m stay)
    abl = _stack(prob, ablation=O.NO_POS_STATE)
    zeroed = _stack(prob, dataclasses.replace(R, w_p1=w_p1))
    _assert_same_path(abl, zeroed)
    np.testing.assert_array_equal(abl.state.S, zeroed.state.S)
    assert _differs(abl, _stack(prob))


def test_no_memread_is_a_history_head_blind_to_the_context():
    prob = _problem()
    R = router_of(prob)
    th1 = R.th1.copy()
    th1[:, W.d_s:] = 0.0       # the c and nu inputs of f_theta
    abl = _stack(prob, ablation=O.NO_MEMREAD)
    blind = _stack(prob, dataclasses.replace(R, th1=th1))
    _assert_same_path(abl, blind)
    np.testing.assert_array_equal(abl.state.p_hist, blind.state.p_hist)
    np.testing.assert_array_equal(abl.state.m_hist, blind.state.m_hist)
    # the memory is never written: the stack ends with its initial (zero) state
    assert not abl.state.S.any() and not abl.state.zeta.any()
    assert blind.state.S.any()
    assert _differs(abl, _stack(prob))


def test_no_history_is_the_local_router():
    prob = _problem()
    R = router_of(prob)
    abl = _stack(prob, ablation=O.NO_HISTORY)
    local = _stack(prob, dataclasses.replace(R, th2=np.zeros_like(R.th2)))
    _assert_same_path(abl, local)
    # no history scores exist: p = m = 1 throughout; no memory is kept
    for L in abl.layers:
        assert np.all(L.state.p_hist == 1.0) and np.all(L.state.m_hist == 1.0)
    assert not abl.state.S.any()
    assert _differs(abl, _stack(prob))


def _layer(prob, j, ablation, S=None, zeta=None, p=None, prev1=None, prev2=None, w=W):
    st = state_of(prob)
    if S is not None:
        st = O.State(S, zeta, st.p_hist if p is None else p, st.m_hist)
    elif p is not None:
        st = O.State(st.S, st.zeta, p, st.m_hist)
    hp1 = prob.hbar_prev1.f64 if prev1 is None else prev1
    hp2 = prob.hbar_prev2.f64 if prev2 is None else prev2
    return O.routed_layer(j, dims_of(w), prob.hbar.f64, hp1, hp2, st, ffn_of(prob.ffn[0]),
                          router_of(prob), adapter_of(prob.adapter[0]), float(prob.eta[j - 1]),
                          mode="threshold", tau=0.5, ablation=ablation)


@pytest.mark.parametrize("ablation", [O.NO_MEMREAD, O.NO_HISTORY])
def test_memoryless_logits_ignore_the_memory(ablation):
    prob = synth.make_problem(W.replace(layer_j=3), seed=5)
    rng = np.random.default_rng(11)
    base = _layer(prob, 3, ablation)
    S = rng.standard_normal(prob.S.shape) ** 2
    zeta = rng.standard_normal(prob.zeta.shape) ** 2
    moved = _layer(prob, 3, ablation, S=S, zeta=zeta)
    np.testing.assert_array_equal(base.logit, moved.logit)
    np.testing.assert_array_equal(moved.state.S, S)     # left as it came in
    full = _layer(prob, 3, 0, S=S, zeta=zeta)
    assert np.max(np.abs(full.logit - _layer(prob, 3, 0).logit)) > 1e-6


def test_no_aux_logits_ignore_the_path_vector():
    prob = synth.make_problem(W.replace(layer_j=4), seed=6)
    rng = np.random.default_rng(12)
    base = _layer(prob, 4, O.NO_AUX_STATE)
    p = rng.uniform(0.05, 0.95, W.T)
    prev1 = prob.hbar_prev1.f64 + rng.standard_normal(prob.hbar.shape)
    prev2 = prob.hbar_prev2.f64 - rng.standard_normal(prob.hbar.shape)
    moved = _layer(prob, 4, O.NO_AUX_STATE, p=p, prev1=prev1, prev2=prev2)
    np.testing.assert_array_equal(base.logit, moved.logit)
    # ... while the full router's logit does move with it
    assert np.max(np.abs(_layer(prob, 4, 0, p=p, prev1=prev1, prev2=prev2).logit
                         - _layer(prob, 4, 0).logit)) > 1e-6


def test_no_pos_logits_ignore_depth_and_transitions():
    prob = synth.make_problem(W.replace(layer_j=4), seed=7)
    rng = np.random.default_rng(13)
    base = _layer(prob, 4, O.NO_POS_STATE)
    prev1 = prob.hbar_prev1.f64 + rng.standard_normal(prob.hbar.shape)
    prev2 = prob.hbar_prev2.f64 - rng.standard_normal(prob.hbar.shape)
    moved = _layer(prob, 4, O.NO_POS_STATE, prev1=prev1, prev2=prev2, w=W.replace(L_R=9))
    np.testing.assert_array_equal(base.logit, moved.logit)
    # the history scores still enter the path vector
    p = rng.uniform(0.05, 0.95, W.T)
    assert np.max(np.abs(_layer(prob, 4, O.NO_POS_STATE, p=p).logit - base.logit)) > 1e-6
