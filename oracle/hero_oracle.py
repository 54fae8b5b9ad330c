"""CPU oracle for HeRo's history-aware routed FFN stack.  TEST INFRASTRUCTURE ONLY.

Only the tests, the smoke check and the CPU-baseline leg of the benchmark may
import this module.  The product (the HIP library and its Python binding) never
does, and this module imports nothing from the product.

What it is: the method of the paper (HeRo, "History-Aware Routing", arxiv
2609.08189, Sec. 3), written out step by step in plain float64 numpy, one
function per equation, in the paper's order and notation.  There is no
blocking, fusion or reordering; a matrix product over a batch of tokens is the
only library primitive used, and each token's row is independent of the others
except for the skip-budget selection.

Readings of points the paper leaves open (each one is a named argument or
constant here):
  * the routed FFN stack has no attention between routed layers, so the next
    layer's post-attention state is this layer's output (hbar_{j+1} = h_j);
  * the frozen FFN is Llama's bias-free SwiGLU W_d (SiLU(W_g u) * (W_u u)), and
    LN^ffn is Llama's RMSNorm with gain w and eps_norm;
  * the router's own RMSNorm (hidden encoder) has unit gain and eps_norm;
  * every router/adapter linear map is bias-free; FFN_path is
    Linear(6->d_p) -> SiLU -> Linear(d_p->d_a); f_theta and f_psi are
    Linear(in->d_head) -> SiLU -> Linear(d_head->1);
  * the comparison space of W_n and W_c has width d_m; the three epsilons of the
    transition cosine, the memory read and the history cosine are one eps, and
    both cosines use <a,b> / (|a||b| + eps);
  * phi(x) = x + 1 for x > 0 and exp(x) otherwise (ELU + 1 evaluated directly);
  * the gate decision g >= tau_exec is taken in logit space, logit >= ln(tau/(1-tau)),
    on the float32 rounding of the logit (the precision the kernels decide in);
    ties go to the FFN;
  * an optional per-token logit bias beta enters the gate only: g = sigma(a + b + beta);
  * skip-budget mode (not in the paper; needed because untrained routers give
    gates near 1/2): per layer, n_skip = floor(budget * T + 1/2) tokens with the
    smallest (float32 logit, token index) take the adapter;
  * at layer j = 1 the state is the paper's initial value (S = 0, zeta = 0,
    p = m = 1) whatever the incoming buffers hold;
  * hidden-state outputs are rounded to the storage dtype (bfloat16 nearest-even
    for bf16 workloads) at every layer boundary; with ``state_dtype = "bf16"`` (an
    option of this implementation, not of the paper) the memory matrix S is also
    rounded to bfloat16 where it is written; nothing else is rounded;
  * the component ablations of Table 3 (Sec. 4.3) are a bit set ``ablation``:
    w/o Pos State zeroes the routing-progress and residual-transition features
    (r, q_rem, d, gamma) of the path vector; w/o Aux State drops the path
    encoder (z_a = 0); w/o MemRead keeps the history head but gives it no memory
    (c = 0 and nu = 0 at every layer, as at the first routed block) and leaves S,
    zeta as they came in; w/o History removes the history branch (a = 0, so the
    logit is the local one), writes p = m = 1 and leaves S, zeta as they came in;
  * the training-side backward (last section) holds the branch decision fixed, gives the
    frozen backbone no gradient, hands the router dL/dlogit = dL/dg g (1 - g), and takes
    the utilisation penalty over the first T - 1 positions of each sequence;
  * the router's backward through the stack treats the initial state (S = 0, zeta = 0,
    p = m = 1) and the depth features r, q_rem as constants, takes d_j = |delta_j| to have
    zero gradient where delta_j = 0, and covers the full router with S in full precision
    (no ablation bits, no bf16 S); the logit bias beta takes no gradient.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional

import numpy as np

f64 = np.float64


# ---------------------------------------------------------------------------
# elementary functions
# ---------------------------------------------------------------------------


def sigmoid(x):
    """Logistic function sigma(x) = 1 / (1 + e^-x), evaluated without overflow."""
    x = np.asarray(x, dtype=f64)
    out = np.empty_like(x)
    pos = x >= 0
    out[pos] = 1.0 / (1.0 + np.exp(-x[pos]))
    ex = np.exp(x[~pos])
    out[~pos] = ex / (1.0 + ex)
    return out


def silu(x):
    """SiLU(x) = x * sigma(x)."""
    x = np.asarray(x, dtype=f64)
    return x * sigmoid(x)


def phi(x):
    """Positive feature map ELU(x) + 1 of the linear-attention memory (Sec. 3.2, router memory)."""
    x = np.asarray(x, dtype=f64)
    return np.where(x > 0, x + 1.0, np.exp(np.minimum(x, 0.0)))


def cosine_eps(a, b, eps):
    """<a, b> / (|a| |b| + eps), row-wise over the last axis."""
    num = np.sum(a * b, axis=-1)
    den = np.linalg.norm(a, axis=-1) * np.linalg.norm(b, axis=-1) + eps
    return num / den


def round_bf16(x):
    """Round float64 values to the nearest bfloat16 (8 significant bits), ties to even.

    Written from the definition of the format (same exponent range as IEEE
    binary32, 7 stored fraction bits).  Values in this workload never reach the
    subnormal or overflow range; those are not handled.
    """
    x = np.asarray(x, dtype=f64)
    m, e = np.frexp(x)                      # x = m * 2^e, 0.5 <= |m| < 1
    return np.ldexp(np.rint(np.ldexp(m, 8)), e - 8)


def round_io(x, dtype):
    if dtype == "bf16":
        return round_bf16(x)
    if dtype == "f32":
        return np.asarray(x, dtype=np.float32).astype(f64)
    raise ValueError(dtype)


# ---------------------------------------------------------------------------
# parameters
# ---------------------------------------------------------------------------


@dataclasses.dataclass
class Dims:
    d: int
    d_ff: int
    d_r: int
    L_R: int
    d_m: int
    d_s: int = 64
    d_h: int = 48
    d_a: int = 16
    d_e: int = 256
    d_p: int = 64
    d_head: int = 256
    eps_norm: float = 1e-5
    eps: float = 1e-6
    T_hist: float = 0.9
    io_dtype: str = "f32"
    state_dtype: str = "f32"   # storage of S between layers: "f32" (exact) or "bf16"


@dataclasses.dataclass
class RouterParams:
    """Router parameters shared by every routed layer (Sec. 3.2, last sentence of 'Router memory')."""
    w_hd: np.ndarray   # [d_e, d]        hidden encoder, down
    w_hu: np.ndarray   # [d_h, d_e]      hidden encoder, up
    w_p1: np.ndarray   # [d_p, 6]        path encoder FFN_path, first layer
    w_p2: np.ndarray   # [d_a, d_p]      path encoder, second layer
    w_q: np.ndarray    # [d_m, d_s]
    w_k: np.ndarray    # [d_m, d_s]
    w_v: np.ndarray    # [d_m, d_s]
    w_n: np.ndarray    # [d_m, d_s]      state -> comparison space
    w_c: np.ndarray    # [d_m, d_m]      context -> comparison space
    th1: np.ndarray    # [d_head, d_s + d_m + 1]  history head f_theta
    th2: np.ndarray    # [d_head]
    ps1: np.ndarray    # [d_head, d]     local head f_psi
    ps2: np.ndarray    # [d_head]


@dataclasses.dataclass
class FFNParams:
    norm_w: np.ndarray  # [d]          LN^ffn gain
    w_gate: np.ndarray  # [d_ff, d]
    w_up: np.ndarray    # [d_ff, d]
    w_down: np.ndarray  # [d, d_ff]


@dataclasses.dataclass
class AdapterParams:
    w1: np.ndarray      # [d_r, d]     down projection W_1
    w2: np.ndarray      # [d, d_r]     up projection W_2


@dataclasses.dataclass
class State:
    """Per-token router state carried across routed layers."""
    S: np.ndarray       # [T, d_m, d_m]  memory matrix, key index first
    zeta: np.ndarray    # [T, d_m]       normaliser
    p_hist: np.ndarray  # [T]            previous history score
    m_hist: np.ndarray  # [T]            cumulative history score

    @staticmethod
    def initial(T, d_m):
        """Zero memory and p = m = 1 at the start of a forward pass (Sec. 3.2)."""
        return State(np.zeros((T, d_m, d_m)), np.zeros((T, d_m)), np.ones(T), np.ones(T))

    def copy(self):
        return State(self.S.copy(), self.zeta.copy(), self.p_hist.copy(), self.m_hist.copy())


# ---------------------------------------------------------------------------
# Sec. 3.1  Router computation: FFN input, branches, routed output
# ---------------------------------------------------------------------------


def rmsnorm(h, gain, eps_norm):
    """RMSNorm h / sqrt(mean(h^2) + eps) * gain, per token row."""
    h = np.asarray(h, dtype=f64)
    r = 1.0 / np.sqrt(np.mean(h * h, axis=-1, keepdims=True) + eps_norm)
    out = h * r
    if gain is not None:
        out = out * gain
    return out


def ffn_input(hbar, ffn: FFNParams, dims: Dims):
    """u = LN^ffn(hbar), the normalised FFN input (Sec. 3.1, eq:dense_attention second line)."""
    return rmsnorm(hbar, ffn.norm_w, dims.eps_norm)


def frozen_ffn(u, ffn: FFNParams):
    """Frozen pretrained FFN, read as Llama SwiGLU: W_d (SiLU(W_g u) * (W_u u))."""
    gate = u @ ffn.w_gate.T
    up = u @ ffn.w_up.T
    return (silu(gate) * up) @ ffn.w_down.T


def adapter(u, ad: AdapterParams):
    """Bottleneck adapter W_2 SiLU(W_1 u) (Sec. 3.1, adapter equation)."""
    return silu(u @ ad.w1.T) @ ad.w2.T


def routed_output(hbar, g, use_ffn, ffn_out, adapter_out):
    """Thresholded single-branch output (Sec. 3.1, eq:ffn_route).

    FFN tokens: hbar + g * FFN(u); adapter tokens: hbar + (1 - g) * Adapter(u).
    ``ffn_out``/``adapter_out`` only need valid rows where the branch is taken.
    """
    g = g[:, None]
    return np.where(use_ffn[:, None], hbar + g * ffn_out, hbar + (1.0 - g) * adapter_out)


# ---------------------------------------------------------------------------
# Sec. 3.2  HeRo router: router state
# ---------------------------------------------------------------------------


def hidden_encoder(hbar, R: RouterParams, dims: Dims):
    """z^h = W_hu SiLU(W_hd RMSNorm(hbar)) in R^{d_h} (Sec. 3.2, 'Router state')."""
    return silu(rmsnorm(hbar, None, dims.eps_norm) @ R.w_hd.T) @ R.w_hu.T


def depth_features(j, L_R):
    """Routing progress r = j / L_R and remaining fraction q_rem = (L_R - j) / L_R."""
    return j / L_R, (L_R - j) / L_R


def residual_transitions(j, hbar, hbar_prev1, hbar_prev2, eps):
    """delta_j = hbar_j - hbar_{j-1} (zero at j = 1), d_j = |delta_j|, and
    gamma_j = cos(delta_j, delta_{j-1}) with eps (zero for j <= 2)
    (Sec. 3.2, transition equation and eq:transition_features)."""
    T = hbar.shape[0]
    if j < 2:
        return np.zeros(T), np.zeros(T)
    delta = hbar - hbar_prev1
    d_j = np.linalg.norm(delta, axis=-1)
    if j <= 2:
        return d_j, np.zeros(T)
    delta_prev = hbar_prev1 - hbar_prev2
    return d_j, cosine_eps(delta, delta_prev, eps)


def path_vector(j, L_R, d_j, gamma_j, p_prev, m_prev):
    """x^path = [r, q_rem, d, gamma, p^hist_{j-1}, m^hist_{j-1}] in R^6 (eq:path_vector)."""
    T = d_j.shape[0]
    r, q_rem = depth_features(j, L_R)
    return np.stack([np.full(T, r), np.full(T, q_rem), d_j, gamma_j, p_prev, m_prev], axis=-1)


def path_encoder(x_path, R: RouterParams):
    """z^a = FFN_path(x^path) in R^{d_a}."""
    return silu(x_path @ R.w_p1.T) @ R.w_p2.T


def router_state(z_h, z_a):
    """s = [z^h; z^a] in R^{d_s} (eq:router_state)."""
    return np.concatenate([z_h, z_a], axis=-1)


# ---------------------------------------------------------------------------
# Sec. 3.2  HeRo router: router memory (linear attention over depth)
# ---------------------------------------------------------------------------


def memory_projections(s, R: RouterParams):
    """q = W_q s, k = W_k s, v = W_v s in R^{d_m}."""
    return s @ R.w_q.T, s @ R.w_k.T, s @ R.w_v.T


def memory_read(q, S_prev, zeta_prev, eps):
    """c = phi(q)^T S_{j-1} / (phi(q)^T zeta_{j-1} + eps) (eq:memory_read)."""
    fq = phi(q)
    num = np.einsum("tk,tkv->tv", fq, S_prev)
    den = np.sum(fq * zeta_prev, axis=-1) + eps
    return num / den[:, None]


def memory_write(k, v, S_prev, zeta_prev, rho):
    """S_j = rho S_{j-1} + phi(k) v^T,  zeta_j = rho zeta_{j-1} + phi(k) (eq:memory_update)."""
    fk = phi(k)
    S = rho * S_prev + fk[:, :, None] * v[:, None, :]
    zeta = rho * zeta_prev + fk
    return S, zeta


def memory_from_pairs(phik, v, rho):
    """The memory after n routed layers, from their key/value pairs (eq:memory_update unrolled).

    With the zero initial state of Sec. 3.2, n applications of memory_write give
        S_n = sum_{i=1..n} (prod_{l=i+1..n} rho_l) phi(k_i) v_i^T,   zeta_n likewise with phi(k_i),
    phik, v: [T, n, d_m] (phi(k_i) and v_i of layers 1..n), rho: [n] (rho_l of layers 1..n).
    This is the state behind the depth-history form of the memory.
    """
    T, n, dm = phik.shape
    S = np.zeros((T, dm, dm))
    zeta = np.zeros((T, dm))
    for i in range(n):
        w = 1.0
        for l in range(i + 1, n):
            w *= rho[l]
        S += w * phik[:, i, :, None] * v[:, i, None, :]
        zeta += w * phik[:, i, :]
    return S, zeta


# ---------------------------------------------------------------------------
# Sec. 3.2  HeRo router: gate computation
# ---------------------------------------------------------------------------

# Component ablations of Table 3 (bits of ``ablation``)
NO_POS_STATE, NO_AUX_STATE, NO_MEMREAD, NO_HISTORY = 1, 2, 4, 8


def history_dissimilarity(j, s, c, R: RouterParams, eps):
    """nu = 1 - cos(W_n s, W_c c) for j > 1, nu = 0 at the first routed layer."""
    if j == 1:
        return np.zeros(s.shape[0])
    return 1.0 - cosine_eps(s @ R.w_n.T, c @ R.w_c.T, eps)


def history_head(s, c, nu, R: RouterParams, T_hist):
    """a = f_theta([s; c; nu]) and p^hist = sigma(a / T_hist)."""
    x = np.concatenate([s, c, nu[:, None]], axis=-1)
    a = silu(x @ R.th1.T) @ R.th2
    return a, sigmoid(a / T_hist)


def cumulative_history(m_prev, p):
    """m^hist_j = m^hist_{j-1} * p^hist_j."""
    return m_prev * p


def local_head(hbar, R: RouterParams):
    """b = f_psi(hbar), on the post-attention representation itself (eq:final_gate)."""
    return silu(hbar @ R.ps1.T) @ R.ps2


def execution_gate(a, b, beta=None):
    """Logit a + b (+ optional per-token bias) and gate g = sigma(logit) (eq:final_gate)."""
    ell = a + b
    if beta is not None:
        ell = ell + beta
    return ell, sigmoid(ell)


# ---------------------------------------------------------------------------
# branch decision
# ---------------------------------------------------------------------------


def logit_f32(ell):
    return np.asarray(ell, dtype=np.float32).astype(f64)


def decide_threshold(ell, tau):
    """g >= tau_exec taken as logit >= ln(tau / (1 - tau)) on float32 logits; ties -> FFN (eq:ffn_route)."""
    lam = math.log(tau / (1.0 - tau))
    use_ffn = logit_f32(ell) >= np.float32(lam)
    return use_ffn, float(np.float32(lam))


def n_skip_for(budget, T):
    return int(math.floor(budget * T + 0.5))


def decide_budget(ell, budget):
    """The n_skip smallest (float32 logit, token index) take the adapter.

    Returns (use_ffn, lambda) where lambda is the smallest logit left on the FFN
    branch (+inf when every token skips).
    """
    T = ell.shape[0]
    k = n_skip_for(budget, T)
    l32 = logit_f32(ell)
    order = np.lexsort((np.arange(T), l32))     # primary: logit, secondary: index
    use_ffn = np.ones(T, dtype=bool)
    use_ffn[order[:k]] = False
    lam = float(l32[order[k]]) if k < T else math.inf
    return use_ffn, lam


# ---------------------------------------------------------------------------
# one routed layer and the routed stack
# ---------------------------------------------------------------------------


@dataclasses.dataclass
class LayerResult:
    h: np.ndarray          # [T, d] layer output (rounded to the storage dtype)
    state: State           # updated router state
    logit: np.ndarray      # [T]
    gate: np.ndarray       # [T]
    use_ffn: np.ndarray    # [T] bool: the branch actually taken
    own_ffn: np.ndarray    # [T] bool: the oracle's own decision
    lam: float
    debug: Dict[str, np.ndarray]


def routed_layer(j, dims: Dims, hbar, hbar_prev1, hbar_prev2, state: State,
                 ffn: FFNParams, R: RouterParams, ad: AdapterParams, eta,
                 mode="budget", budget=0.0, tau=0.5, beta=None,
                 forced_ffn=None, round_output=True, compute_rows=None, lam_given=None,
                 ablation=0):
    """Routed layer l_j for a batch of tokens, in the order of Sec. 3 (overview paragraph).

    ``forced_ffn`` (bool [T]) makes the branch follow a given decision (teacher
    forcing); the oracle's own decision is still returned.  ``compute_rows``
    (bool [T]) restricts the expensive branch evaluation to those rows; other
    rows of ``h`` are left as NaN.  ``lam_given`` (budget mode on a subset of a
    larger batch) replaces the subset's own quantile: a token's own decision is
    then FFN iff its float32 logit >= lam_given.  ``ablation`` selects a Table 3
    router variant (bits NO_POS_STATE, NO_AUX_STATE, NO_MEMREAD, NO_HISTORY).
    """
    hbar = np.asarray(hbar, dtype=f64)
    T = hbar.shape[0]
    if j == 1:
        state = State.initial(T, dims.d_m)
    # router state (eq:path_vector .. eq:router_state)
    z_h = hidden_encoder(hbar, R, dims)
    d_j, gamma_j = residual_transitions(j, hbar, hbar_prev1, hbar_prev2, dims.eps)
    x_path = path_vector(j, dims.L_R, d_j, gamma_j, state.p_hist, state.m_hist)
    if ablation & NO_POS_STATE:
        x_path = x_path.copy()
        x_path[:, :4] = 0.0
    z_a = path_encoder(x_path, R)
    if ablation & NO_AUX_STATE:
        z_a = np.zeros_like(z_a)
    s = router_state(z_h, z_a)
    # memory: read before write
    q, k, v = memory_projections(s, R)
    rho = float(sigmoid(np.array([eta]))[0])
    if ablation & (NO_MEMREAD | NO_HISTORY):
        c = np.zeros_like(q)
        S_new, zeta_new = state.S.copy(), state.zeta.copy()
        nu = np.zeros(T)
    else:
        c = memory_read(q, state.S, state.zeta, dims.eps)
        S_new, zeta_new = memory_write(k, v, state.S, state.zeta, rho)
        if dims.state_dtype == "bf16":
            S_new = round_bf16(S_new)       # the memory matrix as stored for the next layer
        nu = history_dissimilarity(j, s, c, R, dims.eps)
    # gate
    if ablation & NO_HISTORY:
        a, p, m = np.zeros(T), np.ones(T), np.ones(T)
    else:
        a, p = history_head(s, c, nu, R, dims.T_hist)
        m = cumulative_history(state.m_hist, p)
    b = local_head(hbar, R)
    ell, g = execution_gate(a, b, beta)
    # decision
    if mode == "threshold":
        own, lam = decide_threshold(ell, tau)
    elif mode == "budget" and lam_given is not None:
        own, lam = logit_f32(ell) >= np.float32(lam_given), float(lam_given)
    elif mode == "budget":
        own, lam = decide_budget(ell, budget)
    else:
        raise ValueError(mode)
    use_ffn = own if forced_ffn is None else np.asarray(forced_ffn, dtype=bool)
    # branches and routed output (eq:ffn_route)
    rows = np.ones(T, dtype=bool) if compute_rows is None else np.asarray(compute_rows, bool)
    ffn_out = np.full(hbar.shape, np.nan)
    adapter_out = np.full(hbar.shape, np.nan)
    fr = np.nonzero(rows & use_ffn)[0]
    ar = np.nonzero(rows & ~use_ffn)[0]
    if fr.size:
        ffn_out[fr] = frozen_ffn(ffn_input(hbar[fr], ffn, dims), ffn)
    if ar.size:
        adapter_out[ar] = adapter(ffn_input(hbar[ar], ffn, dims), ad)
    h = routed_output(hbar, g, use_ffn, ffn_out, adapter_out)
    h[~rows] = np.nan
    if round_output:
        h = round_io(h, dims.io_dtype)
    debug = dict(z_h=z_h, d=d_j, gamma=gamma_j, x_path=x_path, z_a=z_a, s=s, q=q, k=k, v=v,
                 c=c, nu=nu, a=a, b=b, rho=rho)
    return LayerResult(h, State(S_new, zeta_new, p, m), ell, g, use_ffn, own, lam, debug)


@dataclasses.dataclass
class StackResult:
    h: np.ndarray
    state: State
    layers: List[LayerResult]


def routed_stack(dims: Dims, h_in, ffns: List[FFNParams], R: RouterParams,
                 adapters: List[AdapterParams], etas, mode="budget", budget=0.0, tau=0.5,
                 beta=None, forced_ffn=None, lam_given=None, ablation=0):
    """L_R routed layers with zero initial state; hbar_{j+1} = h_j between them.

    ``forced_ffn`` is an optional list (one bool [T] per layer) for teacher
    forcing, ``lam_given`` an optional list of per-layer budget thresholds (for
    a token subset of a larger batch).
    """
    T = h_in.shape[0]
    state = State.initial(T, dims.d_m)
    hist = [None, None]                  # hbar_{j-1}, hbar_{j-2}
    hbar = np.asarray(h_in, dtype=f64)
    layers = []
    for j in range(1, dims.L_R + 1):
        ff = None if forced_ffn is None else forced_ffn[j - 1]
        lg = None if lam_given is None else lam_given[j - 1]
        res = routed_layer(j, dims, hbar, hist[0], hist[1], state, ffns[j - 1], R,
                           adapters[j - 1], etas[j - 1], mode, budget, tau, beta, ff,
                           lam_given=lg, ablation=ablation)
        layers.append(res)
        state = res.state
        hist = [hbar, hist[0]]
        hbar = res.h
    return StackResult(hbar, state, layers)


# ---------------------------------------------------------------------------
# The full decoder: dense attention before every FFN (Sec. 3.1, eq:dense_attention, first
# line) and routing at the last L_R blocks ("latter half" placement, Sec. 4.1)
#
# Readings: Attn is Llama's bias-free grouped-query self-attention.  LN^attn is RMSNorm
# with gain; q = W_q x, k = W_k x, v = W_v x per head of width hd; the rotary position
# embedding turns each interleaved pair (x_{2i}, x_{2i+1}) of q and k by the angle
# pos * inv_freq[i] (the frequency table is an input, so plain and rescaled variants are
# both expressible); attention is causal within each sequence, softmax(q k^T / sqrt(hd)) v,
# query head h reading key/value head floor(h / (n_heads / n_kv_heads)); the heads are
# concatenated and projected by W_o.  Tokens are laid out as [batch][seq], position = index
# in the sequence.  Non-routed blocks keep their pretrained FFN: h = hbar + FFN(LN^ffn(hbar)).
# ---------------------------------------------------------------------------


@dataclasses.dataclass
class AttnDims:
    n_heads: int
    n_kv_heads: int
    head_dim: int


@dataclasses.dataclass
class AttnParams:
    norm_w: np.ndarray    # [d]                               LN^attn gain
    w_q: np.ndarray       # [n_heads * hd, d]
    w_k: np.ndarray       # [n_kv_heads * hd, d]
    w_v: np.ndarray       # [n_kv_heads * hd, d]
    w_o: np.ndarray       # [d, n_heads * hd]
    inv_freq: np.ndarray  # [hd / 2]                          rotary frequencies


def rope(x, pos, inv_freq):
    """Rotary embedding of the rows of x [n, hd]: pair (x_{2i}, x_{2i+1}) turned by
    pos * inv_freq[i] (pos [n])."""
    x = np.asarray(x, dtype=f64)
    ang = np.asarray(pos, dtype=f64)[:, None] * np.asarray(inv_freq, dtype=f64)[None, :]
    c, s = np.cos(ang), np.sin(ang)
    a, b = x[:, 0::2], x[:, 1::2]
    out = np.empty_like(x)
    out[:, 0::2] = a * c - b * s
    out[:, 1::2] = a * s + b * c
    return out


def causal_attention(q, k, v):
    """One head of one sequence: softmax(q k^T / sqrt(hd)) v with key i visible to query t iff
    i <= t.  q, k, v: [seq, hd]."""
    S = q.shape[0]
    scores = (q @ k.T) / math.sqrt(q.shape[1])
    scores = np.where(np.tril(np.ones((S, S), dtype=bool)), scores, -np.inf)
    scores = scores - scores.max(axis=1, keepdims=True)
    p = np.exp(scores)
    p = p / p.sum(axis=1, keepdims=True)
    return p @ v


def attention_block(h, attn: AttnParams, adims: AttnDims, batch, seq, dims: Dims, rows=None):
    """hbar = h + Attn(LN^attn(h)) for tokens laid out as [batch][seq] (eq:dense_attention).

    ``rows`` (token indices) restricts the output to those rows, each computed from its own
    query and all keys up to it; other rows are NaN."""
    h = np.asarray(h, dtype=f64)
    hd, nh, nkv = adims.head_dim, adims.n_heads, adims.n_kv_heads
    x = rmsnorm(h, attn.norm_w, dims.eps_norm)
    k, v = x @ attn.w_k.T, x @ attn.w_v.T
    pos = np.tile(np.arange(seq), batch)
    group = nh // nkv
    k_rot = [rope(k[:, g * hd:(g + 1) * hd], pos, attn.inv_freq) for g in range(nkv)]
    if rows is None:
        q = x @ attn.w_q.T
        o = np.empty_like(q)
        for hh in range(nh):
            g = hh // group
            qh = rope(q[:, hh * hd:(hh + 1) * hd], pos, attn.inv_freq)
            vh = v[:, g * hd:(g + 1) * hd]
            for b in range(batch):
                sl = slice(b * seq, (b + 1) * seq)
                o[sl, hh * hd:(hh + 1) * hd] = causal_attention(qh[sl], k_rot[g][sl], vh[sl])
        return h + o @ attn.w_o.T
    rows = np.asarray(rows)
    out = np.full(h.shape, np.nan)
    q = x[rows] @ attn.w_q.T
    o = np.empty((len(rows), nh * hd))
    for i, t in enumerate(rows):
        b, s_ = divmod(int(t), seq)
        keys = slice(b * seq, b * seq + s_ + 1)          # the token itself and the ones before it
        for hh in range(nh):
            g = hh // group
            qh = rope(q[i:i + 1, hh * hd:(hh + 1) * hd], [s_], attn.inv_freq)[0]
            sc = k_rot[g][keys] @ qh / math.sqrt(hd)
            p = np.exp(sc - sc.max())
            o[i, hh * hd:(hh + 1) * hd] = (p / p.sum()) @ v[keys, g * hd:(g + 1) * hd]
    out[rows] = h[rows] + o @ attn.w_o.T
    return out


def dense_ffn_block(hbar, ffn: FFNParams, dims: Dims):
    """A non-routed block's pretrained FFN: h = hbar + FFN(LN^ffn(hbar))."""
    return hbar + frozen_ffn(ffn_input(hbar, ffn, dims), ffn)


@dataclasses.dataclass
class DecoderResult:
    h: np.ndarray
    state: State
    hbars: List[np.ndarray]        # post-attention state of every block
    routed: List[LayerResult]      # the routed blocks, in order


def decoder_stack(dims: Dims, adims: AttnDims, n_layers, batch, seq, h_in,
                  attns: List[AttnParams], ffns: List[FFNParams], R: RouterParams,
                  adapters: List[AdapterParams], etas, mode="budget", budget=0.0, tau=0.5,
                  beta=None, forced_ffn=None, ablation=0):
    """n_layers decoder blocks; blocks n_layers - L_R + 1 .. n_layers are routed (j = 1..L_R,
    adapters[j-1], etas[j-1]), the others keep their FFN.  Every block starts with dense
    attention.  Hidden states are rounded to the storage dtype after every sub-block."""
    L_R = dims.L_R
    first = n_layers - L_R
    T = h_in.shape[0]
    state = State.initial(T, dims.d_m)
    hist = [None, None]
    h = np.asarray(h_in, dtype=f64)
    hbars, routed = [], []
    for l in range(n_layers):
        hbar = round_io(attention_block(h, attns[l], adims, batch, seq, dims), dims.io_dtype)
        hbars.append(hbar)
        if l < first:
            h = round_io(dense_ffn_block(hbar, ffns[l], dims), dims.io_dtype)
            continue
        j = l - first + 1
        ff = None if forced_ffn is None else forced_ffn[j - 1]
        res = routed_layer(j, dims, hbar, hist[0], hist[1], state, ffns[l], R, adapters[j - 1],
                           etas[j - 1], mode, budget, tau, beta, ff, ablation=ablation)
        routed.append(res)
        state = res.state
        hist = [hbar, hist[0]]
        h = res.h
    return DecoderResult(h, state, hbars, routed)


# ---------------------------------------------------------------------------
# Training side: the backward of the routed block through the gate scaling (Sec. 3.1,
# eq:ffn_route and the remark after it) and the gate-utilisation penalty (Sec. 3.3, Eq. 17-18)
#
# Readings: the branch decision is a constant of the backward (the threshold is not
# differentiated); the backbone (LN^ffn gain and the FFN weights) is frozen, so it takes no
# gradient but passes one on to hbar; the gradient leaves the block at hbar (the residual, and
# LN^ffn through the branch taken) and at the gate g, and the router receives it as
# dL/dlogit = dL/dg g (1 - g) (g = sigma(logit)).  Only the adapter weights of the block are
# trained here.  The penalty's positions are the first T - 1 of every length-T sequence (those
# with a next token; none when T = 1), tokens ordered sequence-major (t = b T + pos), and the
# weight alpha_t is an input.  Everything is float64 with no rounding.
# ---------------------------------------------------------------------------


@dataclasses.dataclass
class BlockGrad:
    dhbar: np.ndarray   # [T, d]   dL/dhbar
    dgate: np.ndarray   # [T]      dL/dg (including a gradient passed in for g)
    dlogit: np.ndarray  # [T]      dL/dlogit
    dw1: np.ndarray     # [d_r, d] dL/dW_1
    dw2: np.ndarray     # [d, d_r] dL/dW_2


def routed_block(hbar, gate, use_ffn, ffn: FFNParams, ad: AdapterParams, dims: Dims):
    """The routed block's output (eq:ffn_route) for a given gate and branch decision, in float64
    without rounding: the function whose gradient routed_block_backward forms."""
    hbar = np.asarray(hbar, dtype=f64)
    gate = np.asarray(gate, dtype=f64)
    use_ffn = np.asarray(use_ffn, dtype=bool)
    u = ffn_input(hbar, ffn, dims)
    ffn_out = np.zeros_like(hbar)
    ad_out = np.zeros_like(hbar)
    if use_ffn.any():
        ffn_out[use_ffn] = frozen_ffn(u[use_ffn], ffn)
    if (~use_ffn).any():
        ad_out[~use_ffn] = adapter(u[~use_ffn], ad)
    return routed_output(hbar, gate, use_ffn, ffn_out, ad_out)


def silu_grad(x):
    """d SiLU(x) / dx = sigma(x) (1 + x (1 - sigma(x)))."""
    s = sigmoid(x)
    return s * (1.0 + x * (1.0 - s))


def rmsnorm_backward(h, gain, eps_norm, du):
    """dL/dh of u = h r gain with r = (mean(h^2) + eps)^(-1/2), given dL/du, per token row:
    dh = r (gain du) - (r^3 / d) h <gain du, h>."""
    h = np.asarray(h, dtype=f64)
    d = h.shape[-1]
    r = 1.0 / np.sqrt(np.mean(h * h, axis=-1, keepdims=True) + eps_norm)
    gdu = du * gain
    return r * gdu - (r ** 3 / d) * h * np.sum(gdu * h, axis=-1, keepdims=True)


def routed_block_backward(hbar, gate, use_ffn, ffn: FFNParams, ad: AdapterParams, dims: Dims,
                          dh_out, dgate_in=None) -> BlockGrad:
    """Gradients of the routed block, given dL/dh_out (and optionally a further dL/dg, e.g. the
    utilisation penalty's), by the chain rule through eq:ffn_route:
      FFN token:     h = hbar + g y,       y = W_d (SiLU(G) * U), G = W_g u, U = W_u u
      adapter token: h = hbar + (1 - g) y, y = W_2 SiLU(z),       z = W_1 u
    with u = LN^ffn(hbar) and the branch fixed."""
    hbar = np.asarray(hbar, dtype=f64)
    gate = np.asarray(gate, dtype=f64)
    use_ffn = np.asarray(use_ffn, dtype=bool)
    dh = np.asarray(dh_out, dtype=f64)
    T = hbar.shape[0]
    u = ffn_input(hbar, ffn, dims)
    du = np.zeros_like(u)
    dgate = np.zeros(T)
    f = use_ffn
    if f.any():
        uf = u[f]
        G = uf @ ffn.w_gate.T
        U = uf @ ffn.w_up.T
        y = (silu(G) * U) @ ffn.w_down.T
        dgate[f] = np.sum(dh[f] * y, axis=-1)
        dact = (gate[f, None] * dh[f]) @ ffn.w_down
        dG = dact * U * silu_grad(G)
        dU = dact * silu(G)
        du[f] = dG @ ffn.w_gate + dU @ ffn.w_up
    a = ~use_ffn
    dw1 = np.zeros_like(np.asarray(ad.w1, dtype=f64))
    dw2 = np.zeros_like(np.asarray(ad.w2, dtype=f64))
    if a.any():
        ua = u[a]
        z = ua @ ad.w1.T
        hid = silu(z)
        y = hid @ ad.w2.T
        dgate[a] = -np.sum(dh[a] * y, axis=-1)
        dy = (1.0 - gate[a, None]) * dh[a]
        dw2 = dy.T @ hid
        dz = (dy @ ad.w2) * silu_grad(z)
        dw1 = dz.T @ ua
        du[a] = dz @ ad.w1
    dhbar = dh + rmsnorm_backward(hbar, ffn.norm_w, dims.eps_norm, du)
    if dgate_in is not None:
        dgate = dgate + np.asarray(dgate_in, dtype=f64)
    dlogit = dgate * gate * (1.0 - gate)
    return BlockGrad(dhbar, dgate, dlogit, dw1, dw2)


def skip_penalty(gates, batch, seq, alpha=1.0):
    """alpha L_skip of Eq. 18 and its gradient over the gates.

    gates [L_R, batch * seq] (token t = b seq + pos).  L_skip is the mean over the
    batch (seq - 1) positions with a next token of the squared sum of the token's gates over
    the routed blocks; the gradient at such a position is 2 alpha (sum_j g) / (batch (seq - 1))
    for every block, and 0 at each sequence's last position.  Returns (value, [L_R, batch*seq])."""
    g = np.asarray(gates, dtype=f64).reshape(gates.shape[0], batch, seq)
    grad = np.zeros_like(g)
    if seq < 2:
        return 0.0, grad.reshape(gates.shape)
    n = batch * (seq - 1)
    tot = g[:, :, : seq - 1].sum(axis=0)            # [batch, seq - 1]
    value = alpha * float(np.sum(tot * tot)) / n
    grad[:, :, : seq - 1] = (2.0 * alpha / n) * tot[None]
    return value, grad.reshape(gates.shape)


# ---------------------------------------------------------------------------
# Training side, continued: gradients reach the router through the gate scaling
# (Sec. 3.1, the remark after eq:ffn_route), and the router's encoders, depth memory and
# heads are trained with the adapters (Sec. 3.3, training objective).  Below: the routed
# stack's backward with every routed layer's branch held fixed, by the chain rule through the
# router equations of Sec. 3.2 in reverse order (gate <- heads <- memory read/write <- router
# state <- encoders and path features), the memory carried backwards across depth.  float64
# throughout, no rounding; the full router (no ablation) and S kept in full precision.
# ---------------------------------------------------------------------------


@dataclasses.dataclass
class StackTrace:
    hbars: List[np.ndarray]        # post-attention state entering routed layer j (index j - 1)
    states: List[State]            # router state entering layer j (index j - 1)
    layers: List[LayerResult]
    h_out: np.ndarray


def routed_stack_f64(dims: Dims, h_in, ffns: List[FFNParams], R: RouterParams,
                     adapters: List[AdapterParams], etas, use_ffn, beta=None) -> StackTrace:
    """The routed stack in float64 with no rounding at layer boundaries and each layer's branch
    given (use_ffn: one bool [T] per layer): the function whose gradient routed_stack_backward
    forms.  Same equations as routed_stack otherwise."""
    if dims.state_dtype != "f32":
        raise ValueError("the backward keeps S in full precision")
    T = np.asarray(h_in).shape[0]
    state = State.initial(T, dims.d_m)
    hbar = np.asarray(h_in, dtype=f64)
    hbars, states, layers = [], [], []
    prev = [None, None]
    for j in range(1, dims.L_R + 1):
        hbars.append(hbar)
        states.append(state)
        res = routed_layer(j, dims, hbar, prev[0], prev[1], state, ffns[j - 1], R, adapters[j - 1],
                           etas[j - 1], mode="threshold", beta=beta, forced_ffn=use_ffn[j - 1],
                           round_output=False)
        layers.append(res)
        prev = [hbar, prev[0]]
        state = res.state
        hbar = res.h
    return StackTrace(hbars, states, layers, hbar)


@dataclasses.dataclass
class StackGrad:
    dh_in: np.ndarray                 # [T, d]
    router: RouterParams              # dL/d(router weights), summed over tokens and layers
    deta: np.ndarray                  # [L_R] dL/d eta_j
    dw1: List[np.ndarray]             # per layer, dL/dW_1
    dw2: List[np.ndarray]             # per layer, dL/dW_2
    dlogit: List[np.ndarray]          # per layer, dL/dlogit [T]


def phi_grad(x):
    """d phi / dx: 1 for x > 0, exp(x) otherwise."""
    x = np.asarray(x, dtype=f64)
    return np.where(x > 0, 1.0, np.exp(np.minimum(x, 0.0)))


def cosine_eps_backward(a, b, eps, dcos):
    """Gradients over a and b of cos = <a, b> / (|a| |b| + eps) (row-wise), given dL/dcos [T]:
    with N = <a, b> and D = |a| |b| + eps,
      dcos/da = b / D - (N / D^2) |b| a / |a|   (the last term taken as 0 where a = 0),
    and symmetrically for b."""
    na = np.linalg.norm(a, axis=-1)
    nb = np.linalg.norm(b, axis=-1)
    N = np.sum(a * b, axis=-1)
    D = na * nb + eps
    ua = np.divide(a, na[:, None], out=np.zeros_like(a), where=na[:, None] > 0)
    ub = np.divide(b, nb[:, None], out=np.zeros_like(b), where=nb[:, None] > 0)
    k = (N / (D * D))[:, None]
    da = dcos[:, None] * (b / D[:, None] - k * nb[:, None] * ua)
    db = dcos[:, None] * (a / D[:, None] - k * na[:, None] * ub)
    return da, db


def _zero_router(R: RouterParams) -> RouterParams:
    return RouterParams(**{f.name: np.zeros_like(np.asarray(getattr(R, f.name), dtype=f64))
                           for f in dataclasses.fields(RouterParams)})


def router_layer_backward(j, dims: Dims, hbar, hbar_prev1, hbar_prev2, state_in: State,
                          res: LayerResult, R: RouterParams, dl, dS, dzeta, dp, dm, G: RouterParams):
    """Reverse of the router at routed layer j (Sec. 3.2), given dL/dlogit and the gradients
    over the state it hands on (S_j, zeta_j, p_j, m_j).  Adds the weight gradients into G and
    returns (dhbar_j, dhbar_{j-1}, dhbar_{j-2}, dL/drho_j, dS_{j-1}, dzeta_{j-1}, dp_{j-1},
    dm_{j-1}); entries for absent predecessors are None."""
    dbg = res.debug
    s, q, k, v, c, nu = dbg["s"], dbg["q"], dbg["k"], dbg["v"], dbg["c"], dbg["nu"]
    rho = dbg["rho"]
    p, m_prev, p_prev = res.state.p_hist, state_in.m_hist, state_in.p_hist
    T = s.shape[0]
    dl = np.asarray(dl, dtype=f64)
    # gate logit ell = a + b (+ beta)
    da = dl.copy()
    db = dl.copy()
    # cumulative history m_j = m_{j-1} p_j and p_j = sigma(a / T_hist)
    dp_tot = dp + dm * m_prev
    dm_prev = dm * p
    da = da + dp_tot * p * (1.0 - p) / dims.T_hist
    # local head b = f_psi(hbar)
    pre_b = hbar @ R.ps1.T
    G.ps2 += silu(pre_b).T @ db
    dpre_b = db[:, None] * R.ps2[None, :] * silu_grad(pre_b)
    G.ps1 += dpre_b.T @ hbar
    dhbar = dpre_b @ R.ps1
    # history head a = f_theta([s; c; nu])
    x_th = np.concatenate([s, c, nu[:, None]], axis=-1)
    pre_a = x_th @ R.th1.T
    G.th2 += silu(pre_a).T @ da
    dpre_a = da[:, None] * R.th2[None, :] * silu_grad(pre_a)
    G.th1 += dpre_a.T @ x_th
    dx_th = dpre_a @ R.th1
    ds = dx_th[:, :dims.d_s].copy()
    dc = dx_th[:, dims.d_s:dims.d_s + dims.d_m].copy()
    dnu = dx_th[:, -1]
    # history dissimilarity nu = 1 - cos(W_n s, W_c c) (a constant 0 at j = 1)
    if j > 1:
        du1, du2 = cosine_eps_backward(s @ R.w_n.T, c @ R.w_c.T, dims.eps, -dnu)
        G.w_n += du1.T @ s
        ds += du1 @ R.w_n
        G.w_c += du2.T @ c
        dc += du2 @ R.w_c
    # memory write S_j = rho S_{j-1} + phi(k) v^T, zeta_j = rho zeta_{j-1} + phi(k)
    S_prev, z_prev = state_in.S, state_in.zeta
    fk = phi(k)
    drho = float(np.sum(dS * S_prev) + np.sum(dzeta * z_prev))
    dS_prev = rho * dS
    dz_prev = rho * dzeta
    dfk = np.einsum("tkv,tv->tk", dS, v) + dzeta
    dv = np.einsum("tkv,tk->tv", dS, fk)
    dk = dfk * phi_grad(k)
    # memory read c = phi(q)^T S_{j-1} / (phi(q)^T zeta_{j-1} + eps), before the write
    fq = phi(q)
    den = np.sum(fq * z_prev, axis=-1) + dims.eps
    dnum = dc / den[:, None]
    dden = -np.sum(dc * c, axis=-1) / den
    dfq = np.einsum("tkv,tv->tk", S_prev, dnum) + z_prev * dden[:, None]
    dS_prev += fq[:, :, None] * dnum[:, None, :]
    dz_prev += fq * dden[:, None]
    dq = dfq * phi_grad(q)
    # projections q, k, v = W s
    G.w_q += dq.T @ s
    G.w_k += dk.T @ s
    G.w_v += dv.T @ s
    ds += dq @ R.w_q + dk @ R.w_k + dv @ R.w_v
    # router state s = [z^h; z^a]
    dzh = ds[:, :dims.d_h]
    dza = ds[:, dims.d_h:]
    # path encoder z^a = FFN_path(x^path), x^path = [r, q_rem, d_j, gamma_j, p_{j-1}, m_{j-1}]
    x_path = dbg["x_path"]
    pre_p = x_path @ R.w_p1.T
    G.w_p2 += dza.T @ silu(pre_p)
    dpre_p = (dza @ R.w_p2) * silu_grad(pre_p)
    G.w_p1 += dpre_p.T @ x_path
    dx = dpre_p @ R.w_p1
    dp_prev = dx[:, 4]
    dm_prev = dm_prev + dx[:, 5]
    # residual transitions delta_j = hbar_j - hbar_{j-1}: d_j = |delta_j| (j >= 2),
    # gamma_j = cos(delta_j, delta_{j-1}) (j >= 3)
    dh1 = dh2 = None
    if j >= 2:
        delta = hbar - hbar_prev1
        nd = np.linalg.norm(delta, axis=-1)
        ddelta = np.divide(dx[:, 2:3] * delta, nd[:, None], out=np.zeros_like(delta),
                           where=nd[:, None] > 0)
        dh1 = np.zeros_like(hbar)
        if j >= 3:
            delta_prev = hbar_prev1 - hbar_prev2
            dd1, dd0 = cosine_eps_backward(delta, delta_prev, dims.eps, dx[:, 3])
            ddelta += dd1
            dh1 += dd0
            dh2 = -dd0
        dhbar += ddelta
        dh1 -= ddelta
    # hidden encoder z^h = W_hu SiLU(W_hd RMSNorm(hbar)) (unit gain)
    hh = rmsnorm(hbar, None, dims.eps_norm)
    pre_h = hh @ R.w_hd.T
    G.w_hu += dzh.T @ silu(pre_h)
    dpre_h = (dzh @ R.w_hu) * silu_grad(pre_h)
    G.w_hd += dpre_h.T @ hh
    dhbar += rmsnorm_backward(hbar, 1.0, dims.eps_norm, dpre_h @ R.w_hd)
    return dhbar, dh1, dh2, drho, dS_prev, dz_prev, dp_prev, dm_prev


def routed_stack_backward(dims: Dims, h_in, ffns: List[FFNParams], R: RouterParams,
                          adapters: List[AdapterParams], etas, use_ffn, dh_out, dgates_in=None,
                          beta=None) -> StackGrad:
    """Gradients of J = <dh_out, h_{L_R}> + sum_j <dgates_in[j], g_j> through the routed stack
    with every layer's branch fixed (routed_stack_f64 is the forward).  Layer by layer from the
    last: the block's backward gives dL/dhbar_j and dL/dlogit_j; the router's backward turns
    dL/dlogit_j and the gradients over the state it handed on into its weight gradients, the
    post-attention states' share (hbar_j, and hbar_{j-1}, hbar_{j-2} through the residual
    transitions) and the gradients over the state it received.  hbar_{j+1} = h_j, so dL/dh_j is
    everything that reached hbar_{j+1}.  The initial state is a constant."""
    tr = routed_stack_f64(dims, h_in, ffns, R, adapters, etas, use_ffn, beta)
    L, T = dims.L_R, tr.h_out.shape[0]
    dHB = [np.zeros((T, dims.d)) for _ in range(L + 2)]     # dHB[j]: dL/dhbar_j, j = 1 .. L + 1
    dHB[L + 1] = np.asarray(dh_out, dtype=f64).copy()
    G = _zero_router(R)
    deta = np.zeros(L)
    dw1, dw2, dlogits = [None] * L, [None] * L, [None] * L
    dS = np.zeros((T, dims.d_m, dims.d_m))
    dz = np.zeros((T, dims.d_m))
    dp = np.zeros(T)
    dm = np.zeros(T)
    for j in range(L, 0, -1):
        res = tr.layers[j - 1]
        hbar = tr.hbars[j - 1]
        dgi = None if dgates_in is None else dgates_in[j - 1]
        bg = routed_block_backward(hbar, res.gate, use_ffn[j - 1], ffns[j - 1], adapters[j - 1], dims,
                                   dHB[j + 1], dgi)
        dHB[j] += bg.dhbar
        dw1[j - 1], dw2[j - 1], dlogits[j - 1] = bg.dw1, bg.dw2, bg.dlogit
        h1 = tr.hbars[j - 2] if j >= 2 else None
        h2 = tr.hbars[j - 3] if j >= 3 else None
        dhb, dh1, dh2, drho, dS, dz, dp, dm = router_layer_backward(
            j, dims, hbar, h1, h2, tr.states[j - 1], res, R, bg.dlogit, dS, dz, dp, dm, G)
        dHB[j] += dhb
        if dh1 is not None:
            dHB[j - 1] += dh1
        if dh2 is not None:
            dHB[j - 2] += dh2
        rho = res.debug["rho"]
        deta[j - 1] = drho * rho * (1.0 - rho)
    return StackGrad(dHB[1], G, deta, dw1, dw2, dlogits)
