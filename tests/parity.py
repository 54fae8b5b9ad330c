"""GPU-versus-oracle comparison protocol (test helper).

Branch decisions are integers taken from floating point, so they are compared
exactly except for tokens whose gate lies within BAND of the layer's threshold
(tau in threshold mode, sigma(lambda) in budget mode); such tokens are counted
and reported, and the oracle then follows the GPU's decision (teacher forcing)
so that everything downstream stays comparable.  In budget mode the GPU's
selection is also checked exactly against the budget rule applied to its own
logits.  Index lists are checked bit-exactly against the GPU's own mask.
Real-valued outputs are compared per token row:
    err = max_i |x_gpu - x_ref| / max(max_i |x_ref|, 1e-30),  reported as the max over rows.
"""
import math

import numpy as np

from oracle import hero_oracle as O
from tests.oracle_inputs import adapter_of, dims_of, ffn_of, router_of, state_of

BAND = 1e-3
TOL = {"f32": 1e-4, "bf16": 2e-2}
# the router's outputs are fp32 arithmetic on exactly stored inputs in every workload, so they are
# held to the fp32 tolerance even where hidden states and weights are bf16
ROUTER_KEYS = ("logit", "gate", "p", "m", "S", "zeta")


def tol_of(w, key, own_inputs=True):
    """Tolerance of one output: the workload dtype's, except that
    * a memory matrix stored in bf16 is a bf16 quantity (the GPU rounds its fp32 value, the
      oracle its fp64 one, so the two may differ by one bf16 ulp);
    * the router's outputs are held to the fp32 tolerance when the layer ran on the same inputs on
      both sides (a single layer call, or each layer of a stack fed the GPU's own inputs).  Through
      a bf16 stack compared end to end, the hidden states the router reads differ by bf16
      rounding from layer 2 on, and the workload's tolerance applies."""
    if key == "S" and w.state_dtype == "bf16":
        return TOL["bf16"]
    if key in ROUTER_KEYS and own_inputs:
        return TOL["f32"]
    return TOL[w.dtype]


def row_rel_err(x, ref):
    x = np.asarray(x, np.float64).reshape(len(x), -1)
    ref = np.asarray(ref, np.float64).reshape(len(ref), -1)
    if x.size == 0:
        return 0.0
    den = np.maximum(np.max(np.abs(ref), axis=1), 1e-30)
    return float(np.max(np.max(np.abs(x - ref), axis=1) / den))


def scalar_err(x, ref):
    x, ref = np.asarray(x, np.float64), np.asarray(ref, np.float64)
    if x.size == 0:
        return 0.0
    return float(np.max(np.abs(x - ref) / np.maximum(np.abs(ref), 1.0)))


def check_compaction(L, T):
    mask = L["mask"]
    assert L["n_ffn"] == int(mask.sum()) and L["n_ad"] == T - int(mask.sum())
    np.testing.assert_array_equal(L["idx_ffn"][:L["n_ffn"]], np.nonzero(mask)[0])
    np.testing.assert_array_equal(L["idx_ad"][:L["n_ad"]], np.nonzero(~mask)[0])


def check_budget_selection(L, budget, T):
    """The GPU picked exactly the n_skip smallest (logit, index) of its own logits."""
    own, lam = O.decide_budget(L["logit"].astype(np.float64), budget)
    np.testing.assert_array_equal(L["mask"], own)
    assert (~L["mask"]).sum() == O.n_skip_for(budget, T)
    if math.isinf(lam):
        assert math.isinf(L["lam"])
    else:
        assert L["lam"] == np.float32(lam)


def band_threshold(w, lam_ref):
    if w.mode == "threshold":
        return w.tau
    return float(O.sigmoid(np.array([lam_ref]))[0]) if math.isfinite(lam_ref) else 1.0


def compare_decisions(w, L, ref, lam_ref):
    """Mask mismatches must all lie in the band; returns the number of band tokens that differ."""
    mism = L["mask"] != ref.own_ffn
    thr = band_threshold(w, lam_ref)
    far = mism & (np.abs(ref.gate - thr) >= BAND)
    assert not far.any(), (f"{int(far.sum())} decisions differ outside the band: tokens "
                           f"{np.nonzero(far)[0][:10]}, gates {ref.gate[far][:10]}, thr {thr}")
    return int(mism.sum())


def oracle_layer(prob, j, forced_ffn=None, rows=None, lam_given=None):
    w = prob.w
    hp1 = prob.hbar_prev1.f64 if prob.hbar_prev1 is not None else None
    hp2 = prob.hbar_prev2.f64 if prob.hbar_prev2 is not None else None
    return O.routed_layer(j, dims_of(w), prob.hbar.f64, hp1, hp2, state_of(prob), ffn_of(prob.ffn[0]),
                          router_of(prob), adapter_of(prob.adapter[0]), float(prob.eta[j - 1]),
                          mode=w.mode, budget=w.budget, tau=w.tau,
                          beta=None if prob.beta is None else prob.beta.astype(np.float64),
                          forced_ffn=forced_ffn, compute_rows=rows, lam_given=lam_given,
                          ablation=w.ablation)


def check_layer(prob, gpu_res, j, rows=None, report=None):
    """Full comparison of one routed layer call (GPU results vs the teacher-forced oracle)."""
    w = prob.w
    T = prob.hbar.shape[0]
    tol = TOL[w.dtype]
    L = gpu_res["layers"][0]
    check_compaction(L, T)
    if w.mode == "budget":
        check_budget_selection(L, w.budget, T)
    ref = oracle_layer(prob, j, forced_ffn=L["mask"], rows=rows)
    # the oracle's own (untouched) decision for the band check
    if w.mode == "budget":
        _, lam_ref = O.decide_budget(ref.logit, w.budget)
    else:
        lam_ref = ref.lam
    n_band = compare_decisions(w, L, ref, lam_ref)
    sel = np.arange(T) if rows is None else np.nonzero(rows)[0]
    if w.ablation & (O.NO_MEMREAD | O.NO_HISTORY):
        # no memory access: the buffers must come back exactly as they went in
        # (the oracle's own S, zeta are its initial zeros at j = 1)
        assert np.array_equal(gpu_res["S"], prob.S), "S was written"
        assert np.array_equal(gpu_res["zeta"], prob.zeta), "zeta was written"
        S_ref, zeta_ref = prob.S.astype(np.float64), prob.zeta.astype(np.float64)
    else:
        S_ref, zeta_ref = ref.state.S, ref.state.zeta
    errs = dict(
        logit=scalar_err(L["logit"], ref.logit),
        gate=scalar_err(L["gate"], ref.gate),
        h=row_rel_err(gpu_res["h"][sel], ref.h[sel]),
        S=row_rel_err(gpu_res["S"], S_ref),
        zeta=row_rel_err(gpu_res["zeta"], zeta_ref),
        p=scalar_err(gpu_res["p_hist"], ref.state.p_hist),
        m=scalar_err(gpu_res["m_hist"], ref.state.m_hist),
        band_flips=n_band, n_ffn=L["n_ffn"],
    )
    if report is not None:
        report.update(errs)
    for k in ("logit", "gate", "h", "S", "zeta", "p", "m"):
        t = tol_of(w, k)
        assert errs[k] <= t, f"{k}: max rel err {errs[k]:.3e} > {t:.0e} ({errs})"
    return errs


class _LazyMap:
    """Sequence view applying f to the items of a lazily generated sequence."""

    def __init__(self, seq, f):
        self.seq, self.f = seq, f

    def __len__(self):
        return len(self.seq)

    def __getitem__(self, i):
        return self.f(self.seq[i])


def check_stack(prob, gpu_res, rows=None, report=None):
    """Routed stack: per-layer decisions, logits and gates, and the final hidden state and
    router state, against the oracle stack teacher-forced to the GPU's decisions.  With
    ``rows`` (a token subset) the oracle's own budget decisions use the GPU's per-layer
    lambda, since the quantile is over the whole batch."""
    w = prob.w
    T = prob.hbar.shape[0]
    tol = TOL[w.dtype]
    layers = gpu_res["layers"]
    sel = np.arange(T) if rows is None else np.asarray(rows)
    for L in layers:
        check_compaction(L, T)
        if w.mode == "budget":
            check_budget_selection(L, w.budget, T)
    forced = [L["mask"][sel] for L in layers]
    lam_given = [L["lam"] for L in layers] if (rows is not None and w.mode == "budget") else None
    beta = None if prob.beta is None else prob.beta[sel].astype(np.float64)
    ref = O.routed_stack(dims_of(w), prob.hbar.f64[sel], _LazyMap(prob.ffn, ffn_of), router_of(prob),
                         _LazyMap(prob.adapter, adapter_of), prob.eta.astype(np.float64),
                         mode=w.mode, budget=w.budget, tau=w.tau, beta=beta,
                         forced_ffn=forced, lam_given=lam_given, ablation=w.ablation)
    if w.ablation & (O.NO_MEMREAD | O.NO_HISTORY):
        # no memory access: the caller's buffers come back exactly as they went in
        assert np.array_equal(gpu_res["S"], prob.S) and np.array_equal(gpu_res["zeta"], prob.zeta)
        S_ref, zeta_ref = prob.S[sel].astype(np.float64), prob.zeta[sel].astype(np.float64)
    else:
        S_ref, zeta_ref = ref.state.S, ref.state.zeta
    n_band = 0
    errs = dict(logit=0.0, gate=0.0)
    for L, R in zip(layers, ref.layers):
        if w.mode == "budget" and rows is None:
            _, lam_ref = O.decide_budget(R.logit, w.budget)
        else:
            lam_ref = R.lam
        mism = L["mask"][sel] != R.own_ffn
        thr = band_threshold(w, lam_ref)
        far = mism & (np.abs(R.gate - thr) >= BAND)
        assert not far.any(), (f"{int(far.sum())} decisions differ outside the band at layer "
                               f"{len(errs) and layers.index(L) + 1}: gates {R.gate[far][:4]}, thr {thr}, "
                               f"logit err so far {errs['logit']:.2e}")
        n_band += int(mism.sum())
        errs["logit"] = max(errs["logit"], scalar_err(L["logit"][sel], R.logit))
        errs["gate"] = max(errs["gate"], scalar_err(L["gate"][sel], R.gate))
    errs.update(h=row_rel_err(gpu_res["h"][sel], ref.h), S=row_rel_err(gpu_res["S"][sel], S_ref),
                zeta=row_rel_err(gpu_res["zeta"][sel], zeta_ref),
                p=scalar_err(gpu_res["p_hist"][sel], ref.state.p_hist),
                m=scalar_err(gpu_res["m_hist"][sel], ref.state.m_hist), band_flips=n_band)
    if report is not None:
        report.update(errs)
    for k in ("logit", "gate", "h", "S", "zeta", "p", "m"):
        t = tol_of(w, k, own_inputs=False)
        assert errs[k] <= t, f"{k}: max rel err {errs[k]:.3e} > {t:.0e} ({errs})"
    return errs


def check_stack_layerwise(prob, layer_io, rows=None, report=None, verbose=False):
    """Deep stacks: every routed layer checked on the GPU's own inputs.

    ``layer_io[j-1]`` holds, for the selected token rows, what the GPU fed into and got out
    of routed layer j: ``hbar`` (its post-attention input), ``S``/``zeta``/``p``/``m``
    before the layer, the layer's stats, and ``h``/``S1``/``zeta1``/``p1``/``m1`` after it.
    The oracle runs each layer from the GPU's inputs with the GPU's decisions (so errors
    cannot compound over depth) and each layer is held to the single-layer tolerance.
    """
    w = prob.w
    tol = TOL[w.dtype]
    T = prob.hbar.shape[0]
    sel = np.arange(T) if rows is None else np.asarray(rows)
    worst = dict(logit=0.0, gate=0.0, h=0.0, S=0.0, zeta=0.0, p=0.0, m=0.0)
    n_band = 0
    far_info = []
    for j in range(1, w.L_R + 1):
        io = layer_io[j - 1]
        L = io["stats"]
        check_compaction(L, T)
        if w.mode == "budget":
            check_budget_selection(L, w.budget, T)
        prev1 = layer_io[j - 2]["hbar"] if j >= 2 else None
        prev2 = layer_io[j - 3]["hbar"] if j >= 3 else None
        st = O.State(io["S"], io["zeta"], io["p"], io["m"])
        beta = None if prob.beta is None else prob.beta[sel].astype(np.float64)
        lam_given = L["lam"] if (rows is not None and w.mode == "budget") else None
        R = O.routed_layer(j, dims_of(w), io["hbar"], prev1, prev2, st, ffn_of(prob.ffn[j - 1]), router_of(prob),
                           adapter_of(prob.adapter[j - 1]), float(prob.eta[j - 1]), mode=w.mode,
                           budget=w.budget, tau=w.tau, beta=beta, forced_ffn=L["mask"][sel],
                           lam_given=lam_given, ablation=w.ablation)
        if w.mode == "budget" and rows is None:
            _, lam_ref = O.decide_budget(R.logit, w.budget)
        else:
            lam_ref = R.lam
        mism = L["mask"][sel] != R.own_ffn
        thr = band_threshold(w, lam_ref)
        far = mism & (np.abs(R.gate - thr) >= BAND)
        if far.any():
            far_info.append((j, R.gate[far][:4].tolist(), thr))
        n_band += int(mism.sum())
        if verbose:
            print(f"  layer {j}: n_ffn {L['n_ffn']}, logit err {scalar_err(L['logit'][sel], R.logit):.2e}, "
                  f"{int(mism.sum())} band flips", flush=True)
        e = dict(logit=scalar_err(L["logit"][sel], R.logit), gate=scalar_err(L["gate"][sel], R.gate),
                 h=row_rel_err(io["h"], R.h), S=row_rel_err(io["S1"], R.state.S),
                 zeta=row_rel_err(io["zeta1"], R.state.zeta), p=scalar_err(io["p1"], R.state.p_hist),
                 m=scalar_err(io["m1"], R.state.m_hist))
        for k in worst:
            worst[k] = max(worst[k], e[k])
    worst["band_flips"] = n_band
    if report is not None:
        report.update(worst)
    assert not far_info, f"decisions outside the band (layer, gates, threshold): {far_info}"
    for k in ("logit", "gate", "h", "S", "zeta", "p", "m"):
        t = tol_of(w, k)
        assert worst[k] <= t, f"{k}: max rel err {worst[k]:.3e} > {t:.0e} ({worst})"
    return worst


def check_decoder(prob, gpu_res, report=None):
    """Full decoder (attention at every block, routing at the last L_R): per routed block the
    decisions, logits and gates, then the output and the router state, against the oracle
    decoder teacher-forced to the GPU's decisions."""
    from tests.oracle_inputs import adims_of, attn_of
    w = prob.w
    T = prob.hbar.shape[0]
    layers = gpu_res["layers"]
    for L in layers:
        check_compaction(L, T)
        if w.mode == "budget":
            check_budget_selection(L, w.budget, T)
    beta = None if prob.beta is None else prob.beta.astype(np.float64)
    ref = O.decoder_stack(dims_of(w), adims_of(w), w.n_layers, w.batch, w.seq, prob.hbar.f64,
                          _LazyMap(prob.attn, lambda a: attn_of(a, w, prob.inv_freq)),
                          _LazyMap(prob.ffn, ffn_of), router_of(prob), _LazyMap(prob.adapter, adapter_of),
                          prob.eta.astype(np.float64), mode=w.mode, budget=w.budget, tau=w.tau, beta=beta,
                          forced_ffn=[L["mask"] for L in layers], ablation=w.ablation)
    n_band = 0
    errs = dict(logit=0.0, gate=0.0)
    for jj, (L, R) in enumerate(zip(layers, ref.routed), start=1):
        lam_ref = O.decide_budget(R.logit, w.budget)[1] if w.mode == "budget" else R.lam
        mism = L["mask"] != R.own_ffn
        thr = band_threshold(w, lam_ref)
        far = mism & (np.abs(R.gate - thr) >= BAND)
        assert not far.any(), (f"{int(far.sum())} decisions differ outside the band at routed block {jj}: "
                               f"gates {R.gate[far][:4]}, thr {thr}")
        n_band += int(mism.sum())
        errs["logit"] = max(errs["logit"], scalar_err(L["logit"], R.logit))
        errs["gate"] = max(errs["gate"], scalar_err(L["gate"], R.gate))
    errs.update(h=row_rel_err(gpu_res["h"], ref.h), S=row_rel_err(gpu_res["S"], ref.state.S),
                zeta=row_rel_err(gpu_res["zeta"], ref.state.zeta),
                p=scalar_err(gpu_res["p_hist"], ref.state.p_hist),
                m=scalar_err(gpu_res["m_hist"], ref.state.m_hist), band_flips=n_band)
    if report is not None:
        report.update(errs)
    for k in ("logit", "gate", "h", "S", "zeta", "p", "m"):
        t = tol_of(w, k, own_inputs=False)
        assert errs[k] <= t, f"{k}: max rel err {errs[k]:.3e} > {t:.0e} ({errs})"
    return errs
