"""Seeded synthetic inputs for the HeRo routed FFN stack.

This module is the one piece shared by the GPU harness and the CPU oracle's
callers.  It draws hidden states, frozen-backbone weights, router weights,
adapter weights and (for a mid-stack layer call) a plausible incoming router
state, and stores them in the storage dtype of a workload.  It holds none of the
method's arithmetic: no feature map, no norm, no gate, no routing.  Inputs are
returned twice over: ``store`` arrays (np.float32, or np.uint16 bf16 bit
patterns) to upload to the device, and exact float64 decodings of those same
stored values for the oracle.

Recipe (the paper trains Llama backbones on instruction data; neither the
weights nor the data are available, so Gaussian stand-ins of the same shapes
are used):
  * hidden states ~ N(0, 1);
  * every weight matrix ~ N(0, 0.02), frozen FFN gate/up/down included;
  * the FFN-input RMSNorm gain ~ 1 + N(0, 0.02) (a gain near zero would all but
    switch the FFN branch off);
  * forgetting parameter eta = ln 49 for every routed layer, so that
    sigma(eta) = 0.98, the initial value the paper states for rho (Sec. 4.1);
  * a mid-stack layer call (layer j > 1) also draws an incoming state: a
    geometrically decayed sum of j-1 outer products a_i b_i^T with strictly
    positive a_i (log-normal), its matching normaliser sum, history scores
    p ~ U(0.2, 0.8), m ~ U(0, p), and two earlier post-attention states that
    differ from the current one by N(0, 0.5^2) steps;
  * the 13B prefill workload adds a per-token logit bias that is constant over
    runs of 64 positions: a seeded 29 % of the runs draw N(-2, 1), the rest
    N(2, 1), so that skip decisions cluster by position;
  * a full-decoder workload adds per block an attention-input RMSNorm gain
    ~ 1 + N(0, 0.02), a fused [W_q; W_k; W_v] and W_o ~ N(0, 0.02), and the
    standard rotary frequency table theta^(-2i/hd) of the model;
  * the backward of a routed block takes an upstream gradient dL/dh ~ N(0, 1), gates
    g ~ U(0.02, 0.98) and a branch per token drawn apart from g (adapter with probability
    equal to the workload's budget), so that both branches meet gates on either side of 1/2.
Every draw comes from numpy's PCG64 keyed by (seed, tensor id, layer), drawn in
float32 and rounded once, round-to-nearest-even, to the storage dtype.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional

import numpy as np

# ---------------------------------------------------------------------------
# workload definitions
# ---------------------------------------------------------------------------


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    dtype: str                 # "f32" or "bf16": hidden states and every weight
    d: int                     # model width
    d_ff: int                  # SwiGLU intermediate width
    d_r: int                   # adapter rank
    L_R: int                   # number of routed layers
    d_m: int                   # router-memory key/value width
    T: int                     # tokens per call (batch x positions, flattened)
    mode: str                  # "budget" or "threshold"
    budget: float = 0.0        # skip fraction (budget mode)
    tau: float = 0.5           # execution threshold (threshold mode)
    layer_j: int = 0           # >0: a single layer call at routed index j
    bias: str = "none"         # "none" or "bimodal_runs"
    batch: int = 1
    seq: int = 0
    # router sub-network widths (Sec. 4.1 gives d_s=64 = 48 + 16 and heads of 256)
    d_s: int = 64
    d_h: int = 48
    d_a: int = 16
    d_e: int = 256
    d_p: int = 64
    d_head: int = 256
    eps_norm: float = 1e-5
    eps: float = 1e-6
    T_hist: float = 0.9
    # router variant of Table 3: bits 1 w/o Pos State, 2 w/o Aux State, 4 w/o MemRead,
    # 8 w/o History (0 = the full router)
    ablation: int = 0
    # storage of the router memory S between layers: "f32" or "bf16" (zeta, p, m stay fp32)
    state_dtype: str = "f32"
    # standard deviation of the frozen FFN's and the adapters' weights (0.02 everywhere but in
    # high-contrast parity cases, where larger branch outputs make scaling mistakes visible)
    ffn_std: float = 0.02
    adapter_std: float = 0.02
    # full decoder (n_layers > 0): every block has dense attention, the last L_R are routed
    n_layers: int = 0
    n_heads: int = 32
    n_kv_heads: int = 8
    head_dim: int = 128
    rope_theta: float = 500000.0

    @property
    def d_c(self) -> int:
        return self.d_m

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


WORKLOADS: Dict[str, Workload] = {
    # tiny fp32 stack: 4 routed layers, d=256, d_ff=688, r=16, d_m=32, T=64, ~27 % skip
    "tiny_f32_stack": Workload("tiny_f32_stack", "f32", 256, 688, 16, 4, 32, 64,
                               "budget", budget=0.27, batch=1, seq=64),
    # Llama-3.1-8B shape, one routed layer (j=17 of 32), bf16, T=4096 prefill tokens
    "llama31_8b_layer": Workload("llama31_8b_layer", "bf16", 4096, 14336, 64, 32, 128,
                                 4096, "budget", budget=0.2687, layer_j=17,
                                 batch=1, seq=4096),
    # Llama-3.1-8B shape, 32-layer routed stack, 16 x 2048 tokens, tight budget
    "llama31_8b_stack": Workload("llama31_8b_stack", "bf16", 4096, 14336, 64, 32, 128,
                                 32768, "budget", budget=0.3882, batch=16, seq=2048),
    # Llama-2-7B shape, 32-layer decode step, 256 sequences x 1 token
    "llama2_7b_decode": Workload("llama2_7b_decode", "bf16", 4096, 11008, 64, 32, 128,
                                 256, "budget", budget=0.27, batch=256, seq=1),
    # the paper's operating point on the Llama-3.1-8B shape: adapter rank 896, memory dim 64
    # (Sec. 4.1), one routed layer (j=17 of 32), 25 % skip, T=4096 prefill tokens
    "llama31_8b_paper": Workload("llama31_8b_paper", "bf16", 4096, 14336, 896, 32, 64,
                                 4096, "budget", budget=0.25, layer_j=17, batch=1, seq=4096),
    # Llama-2-13B shape, 40-layer prefill, 8 x 4096 tokens, bimodal position-clustered bias
    "llama2_13b_prefill": Workload("llama2_13b_prefill", "bf16", 5120, 13824, 64, 40, 128,
                                   32768, "threshold", tau=0.5, bias="bimodal_runs",
                                   batch=8, seq=4096),
    # the whole Llama-3.1-8B decoder (32 blocks, GQA 32/8 heads of 128, rotary base 5e5) with
    # the latter half routed (Sec. 4.1), 2 x 2048 prefill tokens, 75 % of routed FFN calls
    # skipped (the rate the paper's 25 % parameter budget implies)
    "llama31_8b_decoder": Workload("llama31_8b_decoder", "bf16", 4096, 14336, 64, 16, 128,
                                   4096, "budget", budget=0.75, batch=2, seq=2048,
                                   n_layers=32, n_heads=32, n_kv_heads=8, head_dim=128,
                                   rope_theta=500000.0),
}

# ---------------------------------------------------------------------------
# storage rounding (input preparation only)
# ---------------------------------------------------------------------------


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (nearest, ties to even); return the bits."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounded = (b + np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return rounded.astype(np.uint16)


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact float64 value of stored bfloat16 bit patterns."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def to_store(x32: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "f32":
        return np.ascontiguousarray(x32, dtype=np.float32)
    if dtype == "bf16":
        flat = np.ascontiguousarray(x32, dtype=np.float32).reshape(-1)
        if flat.size <= 4 * _CHUNK:
            return f32_to_bf16_bits(flat).reshape(x32.shape)
        out = np.empty(flat.size, dtype=np.uint16)

        def conv(c):
            lo, hi = c * _CHUNK, min(flat.size, (c + 1) * _CHUNK)
            out[lo:hi] = f32_to_bf16_bits(flat[lo:hi])

        list(_pool().map(conv, range((flat.size + _CHUNK - 1) // _CHUNK)))
        return out.reshape(x32.shape)
    raise ValueError(dtype)


def store_to_f64(a: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "f32":
        return np.asarray(a, dtype=np.float32).astype(np.float64)
    if dtype == "bf16":
        return bf16_bits_to_f64(a)
    raise ValueError(dtype)


# ---------------------------------------------------------------------------
# seeded draws
# ---------------------------------------------------------------------------

# fixed tensor ids: they key the random streams, so they never change
_TID = {
    "hbar": 1, "hbar_prev1": 2, "hbar_prev2": 3,
    "norm_w": 10, "w_gate": 11, "w_up": 12, "w_down": 13,
    "w1": 20, "w2": 21,
    "w_hd": 30, "w_hu": 31, "w_p1": 32, "w_p2": 33, "w_q": 34, "w_k": 35, "w_v": 36,
    "w_n": 37, "w_c": 38, "th1": 39, "th2": 40, "ps1": 41, "ps2": 42,
    "state_a": 50, "state_b": 51, "p_hist": 52, "m_hist": 53,
    "bias_runs": 60, "bias_vals": 61, "bias_spread": 62,
    "attn_norm": 70, "w_qkv": 71, "w_o": 72,
    "dh_out": 80, "bwd_gate": 81, "bwd_branch": 82,
}


def _rng(seed: int, name: str, layer: int = 0) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64([seed, _TID[name], layer]))


_CHUNK = 1 << 20   # elements per independent stream of a large tensor
_POOL = None


def _pool():
    global _POOL
    if _POOL is None:
        import concurrent.futures
        import os
        n = min(16, os.cpu_count() or 1)
        _POOL = concurrent.futures.ThreadPoolExecutor(max_workers=n)
    return _POOL


def normal32(seed: int, name: str, shape, std: float = 1.0, mean: float = 0.0,
             layer: int = 0) -> np.ndarray:
    """N(mean, std^2) in float32.  Chunk c of 2^20 elements comes from PCG64 keyed by
    (seed, tensor id, layer, c), so large tensors are drawn in parallel."""
    n = int(np.prod(shape))
    x = np.empty(n, dtype=np.float32)

    def fill(c):
        lo, hi = c * _CHUNK, min(n, (c + 1) * _CHUNK)
        g = np.random.Generator(np.random.PCG64([seed, _TID[name], layer, c]))
        g.standard_normal(size=hi - lo, dtype=np.float32, out=x[lo:hi])
        if std != 1.0:
            x[lo:hi] *= np.float32(std)
        if mean != 0.0:
            x[lo:hi] += np.float32(mean)

    nch = (n + _CHUNK - 1) // _CHUNK
    if nch <= 2:
        for c in range(nch):
            fill(c)
    else:
        list(_pool().map(fill, range(nch)))
    return x.reshape(shape)


class Tensor:
    """A stored tensor plus the exact float64 decoding of what was stored."""

    __slots__ = ("store", "dtype", "_f64")

    def __init__(self, store: np.ndarray, dtype: str):
        self.store = store
        self.dtype = dtype
        self._f64 = None

    @property
    def f64(self) -> np.ndarray:
        if self._f64 is None:
            self._f64 = store_to_f64(self.store, self.dtype)
        return self._f64

    @property
    def shape(self):
        return self.store.shape


def _t(x32: np.ndarray, dtype: str) -> Tensor:
    return Tensor(to_store(x32, dtype), dtype)


ROUTER_SHAPES = {
    "w_hd": lambda w: (w.d_e, w.d),
    "w_hu": lambda w: (w.d_h, w.d_e),
    "w_p1": lambda w: (w.d_p, 6),
    "w_p2": lambda w: (w.d_a, w.d_p),
    "w_q": lambda w: (w.d_m, w.d_s),
    "w_k": lambda w: (w.d_m, w.d_s),
    "w_v": lambda w: (w.d_m, w.d_s),
    "w_n": lambda w: (w.d_c, w.d_s),
    "w_c": lambda w: (w.d_c, w.d_m),
    "th1": lambda w: (w.d_head, w.d_s + w.d_m + 1),
    "th2": lambda w: (w.d_head,),
    "ps1": lambda w: (w.d_head, w.d),
    "ps2": lambda w: (w.d_head,),
}


def router_weights(w: Workload, seed: int = 0, std: float = 0.02) -> Dict[str, Tensor]:
    return {k: _t(normal32(seed, k, fn(w), std), w.dtype) for k, fn in ROUTER_SHAPES.items()}


def ffn_layer(w: Workload, layer: int, seed: int = 0) -> Dict[str, Tensor]:
    return {
        "norm_w": _t(normal32(seed, "norm_w", (w.d,), 0.02, 1.0, layer), w.dtype),
        "w_gate": _t(normal32(seed, "w_gate", (w.d_ff, w.d), w.ffn_std, layer=layer), w.dtype),
        "w_up": _t(normal32(seed, "w_up", (w.d_ff, w.d), w.ffn_std, layer=layer), w.dtype),
        "w_down": _t(normal32(seed, "w_down", (w.d, w.d_ff), w.ffn_std, layer=layer), w.dtype),
    }


def adapter_layer(w: Workload, layer: int, seed: int = 0) -> Dict[str, Tensor]:
    return {
        "w1": _t(normal32(seed, "w1", (w.d_r, w.d), w.adapter_std, layer=layer), w.dtype),
        "w2": _t(normal32(seed, "w2", (w.d, w.d_r), w.adapter_std, layer=layer), w.dtype),
    }


def attn_layer(w: Workload, layer: int, seed: int = 0) -> Dict[str, Tensor]:
    n_qkv = (w.n_heads + 2 * w.n_kv_heads) * w.head_dim
    return {
        "norm_w": _t(normal32(seed, "attn_norm", (w.d,), 0.02, 1.0, layer), w.dtype),
        "w_qkv": _t(normal32(seed, "w_qkv", (n_qkv, w.d), 0.02, layer=layer), w.dtype),
        "w_o": _t(normal32(seed, "w_o", (w.d, w.n_heads * w.head_dim), 0.02, layer=layer), w.dtype),
    }


def rope_inv_freq(w: Workload) -> np.ndarray:
    """The model's rotary frequency table theta^(-2i/hd), i < hd/2, as float32."""
    i = np.arange(w.head_dim // 2, dtype=np.float64)
    return (w.rope_theta ** (-2.0 * i / w.head_dim)).astype(np.float32)


def eta_values(w: Workload) -> np.ndarray:
    return np.full(w.L_R, math.log(49.0), dtype=np.float32)


def hidden(w: Workload, seed: int = 0, T: Optional[int] = None) -> Tensor:
    T = w.T if T is None else T
    return _t(normal32(seed, "hbar", (T, w.d)), w.dtype)


def incoming_history(w: Workload, hbar: Tensor, seed: int = 0):
    """Earlier post-attention states for a mid-stack layer call (j >= 2)."""
    T = hbar.shape[0]
    h0 = store_to_f64(hbar.store, w.dtype).astype(np.float32)
    p1 = h0 - normal32(seed, "hbar_prev1", (T, w.d), 0.5)
    prev1 = _t(p1, w.dtype)
    p2 = store_to_f64(prev1.store, w.dtype).astype(np.float32) - normal32(seed, "hbar_prev2", (T, w.d), 0.5)
    prev2 = _t(p2, w.dtype)
    return prev1, prev2


def incoming_memory_pairs(w: Workload, j: int, T: int, seed: int = 0):
    """The key/value pairs of the j-1 routed layers before layer j behind a synthesized state:
    log-normal (strictly positive) a_i in the role of phi(k_i) and Gaussian b_i in the role of
    v_i, each [T, j-1, d_m] float32 (None, None for j == 1)."""
    if j <= 1:
        return None, None
    n, dm = j - 1, w.d_m
    a = np.exp(np.float32(0.5) * _rng(seed, "state_a").standard_normal((T, n, dm), dtype=np.float32))
    b = _rng(seed, "state_b").standard_normal((T, n, dm), dtype=np.float32)
    return a, b


def incoming_state(w: Workload, j: int, T: int, seed: int = 0, decay: float = 0.98):
    """A plausible router state as it stands before routed layer j (fp32 storage).

    S = sum_{i<j} decay^(j-1-i) a_i b_i^T and zeta = sum_{i<j} decay^(j-1-i) a_i over the pairs
    of incoming_memory_pairs; p ~ U(0.2, 0.8), m ~ U(0, p).
    For j == 1 the state is the all-zero matrix/normaliser with p = m = 1.
    """
    dm = w.d_m
    S = np.zeros((T, dm, dm), dtype=np.float32)
    zeta = np.zeros((T, dm), dtype=np.float32)
    if j <= 1:
        return S, zeta, np.ones(T, np.float32), np.ones(T, np.float32)
    a, b = incoming_memory_pairs(w, j, T, seed)
    wgt = np.array([decay ** (j - 1 - i) for i in range(1, j)], dtype=np.float32)
    aw = a * wgt[None, :, None]
    S = np.matmul(aw.transpose(0, 2, 1), b)          # [T, dm, dm] = sum_i w_i a_i b_i^T
    zeta = aw.sum(axis=1)
    gp = _rng(seed, "p_hist")
    p = gp.uniform(0.2, 0.8, size=T).astype(np.float32)
    gm = _rng(seed, "m_hist")
    m = (gm.uniform(0.0, 1.0, size=T).astype(np.float32) * p).astype(np.float32)
    return S, zeta, p, m


def logit_bias(w: Workload, seed: int = 0, T: Optional[int] = None) -> Optional[np.ndarray]:
    """Per-token logit bias: position-clustered bimodal runs ("bimodal_runs"), or U(-3, 3) drawn
    per token ("spread": gates spread over about (0.05, 0.95) whatever the router gives); else None."""
    if w.bias == "none":
        return None
    T = w.T if T is None else T
    if w.bias == "spread":
        return _rng(seed, "bias_spread").uniform(-3.0, 3.0, size=T).astype(np.float32)
    run = 64
    n_runs = (T + run - 1) // run
    n_neg = int(math.floor(0.29 * n_runs + 0.5))
    perm = _rng(seed, "bias_runs").permutation(n_runs)
    neg = np.zeros(n_runs, dtype=bool)
    neg[perm[:n_neg]] = True
    vals = _rng(seed, "bias_vals").standard_normal(T, dtype=np.float32)
    run_of = np.arange(T) // run
    beta = np.where(neg[run_of], vals - np.float32(2.0), vals + np.float32(2.0)).astype(np.float32)
    return beta


def backward_inputs(w: Workload, seed: int = 0, T: Optional[int] = None, n_adapter: Optional[int] = None):
    """Inputs of one routed block's backward besides the layer's own: dL/dh [T, d] in the storage
    dtype, the gates [T] (float32) and the branch taken [T] (True = FFN).  The adapter tokens are
    each token with probability w.budget, or exactly n_adapter tokens at random positions."""
    T = w.T if T is None else T
    dh = _t(normal32(seed, "dh_out", (T, w.d)), w.dtype)
    gate = _rng(seed, "bwd_gate").uniform(0.02, 0.98, size=T).astype(np.float32)
    draw = _rng(seed, "bwd_branch").uniform(0.0, 1.0, size=T)
    if n_adapter is None:
        use_ffn = draw >= w.budget
    else:
        use_ffn = np.ones(T, dtype=bool)
        use_ffn[np.argsort(draw, kind="stable")[:n_adapter]] = False
    return dh, gate, use_ffn


# ---------------------------------------------------------------------------
# a whole problem instance
# ---------------------------------------------------------------------------


class LazyLayers:
    """Per-layer weights drawn on first access (the most recent layers are cached)."""

    def __init__(self, make, layers, keep: int = 2):
        self._make = make
        self._layers = list(layers)
        self._keep = keep
        self._cache: Dict[int, Dict[str, Tensor]] = {}

    def __len__(self):
        return len(self._layers)

    def __getitem__(self, i):
        if i < 0:
            i += len(self._layers)
        if i not in self._cache:
            while len(self._cache) >= self._keep:
                self._cache.pop(next(iter(self._cache)))
            self._cache[i] = self._make(self._layers[i])
        return self._cache[i]

    def __iter__(self):
        for i in range(len(self._layers)):
            yield self[i]


@dataclasses.dataclass
class Problem:
    w: Workload
    hbar: Tensor                      # [T, d]: h_in for a stack, hbar_j for a layer call
    hbar_prev1: Optional[Tensor]
    hbar_prev2: Optional[Tensor]
    S: np.ndarray                     # [T, d_m, d_m] f32 (incoming, layer calls)
    zeta: np.ndarray                  # [T, d_m] f32
    p_hist: np.ndarray                # [T] f32
    m_hist: np.ndarray                # [T] f32
    router: Dict[str, Tensor]
    ffn: "LazyLayers"                 # one per routed layer (a layer call: one entry)
    adapter: "LazyLayers"
    eta: np.ndarray                   # [L_R] f32 (a layer call uses eta[j-1])
    beta: Optional[np.ndarray]        # [T] f32 or None
    # a layer call at j > 1: the pairs of layers 1..j-1 ([T, j-1, d_m] f32), for the depth-history
    # form of the memory; S and zeta above are their decayed sums with decay 0.98
    mem_k: Optional[np.ndarray] = None
    # full decoder: attention weights of every block, and the rotary frequency table
    attn: Optional["LazyLayers"] = None
    inv_freq: Optional[np.ndarray] = None
    mem_v: Optional[np.ndarray] = None


def make_problem(w: Workload, seed: int = 0, T: Optional[int] = None,
                 layer_j: Optional[int] = None) -> Problem:
    """Draw every input of a workload.  ``layer_j`` overrides the workload's layer index."""
    T = w.T if T is None else T
    j = w.layer_j if layer_j is None else layer_j
    hb = hidden(w, seed, T)
    prev1 = prev2 = None
    if j >= 1:
        # a single routed-layer call at index j
        if j >= 2:
            prev1, prev2 = incoming_history(w, hb, seed)
            if j == 2:
                prev2 = None
        S, zeta, p, m = incoming_state(w, j, T, seed)
        mem_k, mem_v = incoming_memory_pairs(w, j, T, seed)
        layers = [j - 1]
    else:
        S = np.zeros((T, w.d_m, w.d_m), np.float32)
        zeta = np.zeros((T, w.d_m), np.float32)
        p = np.ones(T, np.float32)
        m = np.ones(T, np.float32)
        mem_k = mem_v = None
        layers = list(range(w.L_R))
    if w.state_dtype == "bf16":
        # the incoming memory as the caller stores it
        S = bf16_bits_to_f64(f32_to_bf16_bits(S)).astype(np.float32)
    if w.n_layers > 0:
        # full decoder: a frozen FFN and attention in every block, adapters in the routed ones
        return Problem(
            w=w, hbar=hb, hbar_prev1=None, hbar_prev2=None,
            S=S, zeta=zeta, p_hist=p, m_hist=m,
            router=router_weights(w, seed),
            ffn=LazyLayers(lambda l: ffn_layer(w, l, seed), range(w.n_layers)),
            adapter=LazyLayers(lambda l: adapter_layer(w, l, seed), range(w.L_R), keep=4),
            eta=eta_values(w), beta=logit_bias(w, seed, T),
            attn=LazyLayers(lambda l: attn_layer(w, l, seed), range(w.n_layers)),
            inv_freq=rope_inv_freq(w),
        )
    return Problem(
        w=w, hbar=hb, hbar_prev1=prev1, hbar_prev2=prev2,
        S=S, zeta=zeta, p_hist=p, m_hist=m,
        router=router_weights(w, seed),
        ffn=LazyLayers(lambda l: ffn_layer(w, l, seed), layers),
        adapter=LazyLayers(lambda l: adapter_layer(w, l, seed), layers, keep=4),
        eta=eta_values(w),
        beta=logit_bias(w, seed, T),
        mem_k=mem_k, mem_v=mem_v,
    )
