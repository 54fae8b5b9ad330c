"""Python binding of libhero.so: the C ABI of include/hero.h, argument marshalling only.

Every function here has the name of the C entry point it calls.  Pointer
arguments accept a torch tensor (its data_ptr is passed), an int address, or
None.  Nothing here computes any part of the routed layer; if the library has
not been built, loading fails with an error instead of falling back to
anything else.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libhero.so")
ABI_VERSION = 7          # the struct layouts below follow include/hero.h of this version

HERO_OK = 0
HERO_E_NULL = 1
HERO_E_DIM = 2
HERO_E_RANGE = 3
HERO_E_DTYPE = 4
HERO_E_ALIGN = 5
HERO_E_ALIAS = 6
HERO_E_WORKSPACE = 7
HERO_E_UNSUPPORTED = 8
HERO_E_LAUNCH = 9
HERO_E_DEVICE = 10
HERO_E_SCRATCH = 11
HERO_NOALLOC_SCRATCH_BYTES = 64 << 20

HERO_F32 = 0
HERO_BF16 = 1
HERO_MODE_THRESHOLD = 0
HERO_MODE_BUDGET = 1
HERO_ABL_NO_POS_STATE = 1
HERO_ABL_NO_AUX_STATE = 2
HERO_ABL_NO_MEMREAD = 4
HERO_ABL_NO_HISTORY = 8

KERNELS = ("rowstats", "router_gemm", "router_pre", "router_mem", "router_post", "select",
           "ffn_gate_up", "ffn_down", "adapter_down", "adapter_up",
           "attn_norm", "attn_qkv", "attn_core", "attn_out",
           "bwd_norm", "bwd_ffn_e", "bwd_ffn_gate_up", "bwd_ffn_du", "bwd_adapter", "bwd_adapter_wgrad",
           "bwd_rows", "skip_penalty",
           "router_bwd_gemm", "router_bwd_token", "router_bwd_products", "router_bwd_rows")
HERO_K = {name: i for i, name in enumerate(KERNELS)}

_vp = ctypes.c_void_p


class hero_dims(ctypes.Structure):
    _fields_ = [("d", ctypes.c_int), ("d_ff", ctypes.c_int), ("d_r", ctypes.c_int), ("L_R", ctypes.c_int),
                ("d_m", ctypes.c_int), ("d_s", ctypes.c_int), ("d_h", ctypes.c_int), ("d_a", ctypes.c_int),
                ("d_e", ctypes.c_int), ("d_p", ctypes.c_int), ("d_head", ctypes.c_int),
                ("dtype", ctypes.c_int),
                ("eps_norm", ctypes.c_float), ("eps", ctypes.c_float), ("T_hist", ctypes.c_float),
                ("state_dtype", ctypes.c_int)]


class hero_ffn_weights(ctypes.Structure):
    _fields_ = [("norm_w", _vp), ("w_gate", _vp), ("w_up", _vp), ("w_down", _vp),
                ("w_gate_up_tiled", _vp), ("w_down_tiled", _vp)]


class hero_adapter_weights(ctypes.Structure):
    _fields_ = [("w1", _vp), ("w2", _vp)]


ROUTER_FIELDS = ("w_hd", "w_hu", "w_p1", "w_p2", "w_q", "w_k", "w_v", "w_n", "w_c",
                 "th1", "th2", "ps1", "ps2")


class hero_router_weights(ctypes.Structure):
    _fields_ = [(n, _vp) for n in ROUTER_FIELDS]


class hero_state(ctypes.Structure):
    _fields_ = [("S", _vp), ("zeta", _vp), ("p_hist", _vp), ("m_hist", _vp), ("c_read", _vp)]


class hero_router_grads(ctypes.Structure):
    _fields_ = [(n, _vp) for n in ROUTER_FIELDS]


class hero_router_carry(ctypes.Structure):
    _fields_ = [("dS", _vp), ("dzeta", _vp), ("dp", _vp), ("dm", _vp)]


class hero_history(ctypes.Structure):
    _fields_ = [("kv", _vp), ("p_hist", _vp), ("m_hist", _vp)]


class hero_routing(ctypes.Structure):
    _fields_ = [("mode", ctypes.c_int), ("tau", ctypes.c_float), ("budget", ctypes.c_double),
                ("logit_bias", _vp), ("ablation", ctypes.c_int)]


class hero_attn_dims(ctypes.Structure):
    _fields_ = [("n_heads", ctypes.c_int), ("n_kv_heads", ctypes.c_int), ("head_dim", ctypes.c_int)]


class hero_attn_weights(ctypes.Structure):
    _fields_ = [("norm_w", _vp), ("w_qkv", _vp), ("w_o", _vp)]


class hero_ffn_backward_weights(ctypes.Structure):
    _fields_ = [("w_down_t", _vp), ("w_gate_up_t", _vp)]


class hero_block_grads(ctypes.Structure):
    _fields_ = [("dhbar", _vp), ("dgate", _vp), ("dlogit", _vp), ("dw1", _vp), ("dw2", _vp)]


class hero_layer_stats(ctypes.Structure):
    _fields_ = [("mask", _vp), ("idx_ffn", _vp), ("idx_ad", _vp), ("counts", _vp),
                ("logit", _vp), ("gate", _vp), ("lambda_", _vp)]


_lib = None


def lib() -> ctypes.CDLL:
    """Load libhero.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
        L = ctypes.CDLL(LIB_PATH)
        P = ctypes.POINTER
        L.hero_status_string.restype = ctypes.c_char_p
        L.hero_status_string.argtypes = [ctypes.c_int]
        L.hero_abi_version.restype = ctypes.c_int
        L.hero_abi_version.argtypes = []
        if L.hero_abi_version() != ABI_VERSION:
            raise RuntimeError(f"{LIB_PATH} has ABI version {L.hero_abi_version()}, the binding "
                               f"expects {ABI_VERSION}: rebuild it with __graft_entry__.build()")
        L.hero_kernel_timer.restype = ctypes.c_int
        L.hero_kernel_timer.argtypes = [ctypes.c_int, P(_vp), P(_vp), ctypes.c_int]
        L.hero_workspace_size.restype = ctypes.c_int
        L.hero_workspace_size.argtypes = [P(hero_dims), ctypes.c_int, ctypes.c_int, P(ctypes.c_size_t)]
        L.hero_routed_layer.restype = ctypes.c_int
        L.hero_routed_layer.argtypes = [P(hero_dims), ctypes.c_int, ctypes.c_int, _vp, _vp, _vp, _vp,
                                        P(hero_state), P(hero_ffn_weights), P(hero_router_weights),
                                        P(hero_adapter_weights), ctypes.c_float, P(hero_routing),
                                        P(hero_layer_stats), _vp, ctypes.c_size_t, _vp]
        L.hero_routed_layer_noalloc.restype = ctypes.c_int
        L.hero_routed_layer_noalloc.argtypes = [P(hero_dims), ctypes.c_int, ctypes.c_int, _vp, _vp, _vp, _vp,
                                                P(hero_state), P(hero_ffn_weights), P(hero_router_weights),
                                                P(hero_adapter_weights), ctypes.c_float, P(hero_routing),
                                                P(hero_layer_stats), _vp]
        L.hero_routed_stack.restype = ctypes.c_int
        L.hero_routed_stack.argtypes = [P(hero_dims), ctypes.c_int, _vp, _vp, P(hero_state),
                                        P(hero_ffn_weights), P(hero_router_weights),
                                        P(hero_adapter_weights), P(ctypes.c_float), P(hero_routing),
                                        P(hero_layer_stats), _vp, ctypes.c_size_t, _vp]
        L.hero_routed_layer_hist.restype = ctypes.c_int
        L.hero_routed_layer_hist.argtypes = [P(hero_dims), ctypes.c_int, ctypes.c_int, _vp, _vp, _vp, _vp,
                                             P(hero_history), P(hero_ffn_weights), P(hero_router_weights),
                                             P(hero_adapter_weights), P(ctypes.c_float), P(hero_routing),
                                             P(hero_layer_stats), _vp, ctypes.c_size_t, _vp]
        L.hero_routed_stack_hist.restype = ctypes.c_int
        L.hero_routed_stack_hist.argtypes = [P(hero_dims), ctypes.c_int, _vp, _vp, P(hero_history),
                                             P(hero_ffn_weights), P(hero_router_weights),
                                             P(hero_adapter_weights), P(ctypes.c_float), P(hero_routing),
                                             P(hero_layer_stats), _vp, ctypes.c_size_t, _vp]
        L.hero_history_state.restype = ctypes.c_int
        L.hero_history_state.argtypes = [P(hero_dims), ctypes.c_int, ctypes.c_int, _vp, P(ctypes.c_float),
                                         _vp, _vp, _vp]
        L.hero_decoder_workspace_size.restype = ctypes.c_int
        L.hero_decoder_workspace_size.argtypes = [P(hero_dims), P(hero_attn_dims), ctypes.c_int, ctypes.c_int,
                                                  ctypes.c_int, P(ctypes.c_size_t)]
        L.hero_attention_block.restype = ctypes.c_int
        L.hero_attention_block.argtypes = [P(hero_dims), P(hero_attn_dims), ctypes.c_int, ctypes.c_int, _vp, _vp,
                                           P(hero_attn_weights), P(ctypes.c_float), _vp, ctypes.c_size_t, _vp]
        L.hero_decoder_stack.restype = ctypes.c_int
        L.hero_decoder_stack.argtypes = [P(hero_dims), P(hero_attn_dims), ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                         _vp, _vp, P(hero_state), P(hero_attn_weights), P(hero_ffn_weights),
                                         P(hero_router_weights), P(hero_adapter_weights), P(ctypes.c_float),
                                         P(ctypes.c_float), P(hero_routing), P(hero_layer_stats), _vp,
                                         ctypes.c_size_t, _vp]
        L.hero_ffn_decode_weights_make.restype = ctypes.c_int
        L.hero_ffn_decode_weights_make.argtypes = [P(hero_dims), P(hero_ffn_weights), _vp, _vp, _vp]
        L.hero_ffn_backward_weights_make.restype = ctypes.c_int
        L.hero_ffn_backward_weights_make.argtypes = [P(hero_dims), P(hero_ffn_weights), _vp, _vp, _vp]
        L.hero_backward_workspace_size.restype = ctypes.c_int
        L.hero_backward_workspace_size.argtypes = [P(hero_dims), ctypes.c_int, P(ctypes.c_size_t)]
        L.hero_routed_block_backward.restype = ctypes.c_int
        L.hero_routed_block_backward.argtypes = [P(hero_dims), ctypes.c_int, _vp, _vp, _vp, _vp, _vp, _vp,
                                                 P(hero_routing), _vp, P(hero_ffn_weights), P(hero_ffn_backward_weights),
                                                 P(hero_adapter_weights), P(hero_block_grads), _vp,
                                                 ctypes.c_size_t, _vp]
        L.hero_skip_penalty.restype = ctypes.c_int
        L.hero_skip_penalty.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, _vp, ctypes.c_float, _vp, _vp,
                                        _vp]
        L.hero_router_backward_workspace_size.restype = ctypes.c_int
        L.hero_router_backward_workspace_size.argtypes = [P(hero_dims), ctypes.c_int, P(ctypes.c_size_t)]
        L.hero_router_backward.restype = ctypes.c_int
        L.hero_router_backward.argtypes = [P(hero_dims), ctypes.c_int, ctypes.c_int, _vp, _vp, _vp, P(hero_state),
                                           P(hero_router_weights), ctypes.c_float, _vp, P(hero_router_carry), _vp,
                                           _vp, _vp, P(hero_router_grads), _vp, _vp, ctypes.c_size_t, _vp]
        L.hero_peak_mfma.restype = ctypes.c_int
        L.hero_peak_mfma.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, _vp, _vp, P(ctypes.c_double)]
        L.hero_peak_read.restype = ctypes.c_int
        L.hero_peak_read.argtypes = [_vp, ctypes.c_size_t, ctypes.c_int, _vp, _vp]
        _lib = L
    return _lib


def ptr(x) -> Optional[int]:
    """Device address of a tensor, an int address, or None."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


class HeroError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {hero_status_string(status)} (status {status})")


def check(status: int, where: str) -> None:
    if status != HERO_OK:
        raise HeroError(status, where)


def hero_status_string(status: int) -> str:
    return lib().hero_status_string(status).decode()


def hero_abi_version() -> int:
    return lib().hero_abi_version()


def hero_peak_mfma(random_operands: bool, iters: int, workgroups: int, sink, stream, mi16: bool = False) -> float:
    """Launch the matrix-core rate probe on `stream`; returns the FLOPs the launch performs."""
    flop = ctypes.c_double()
    mode = int(bool(random_operands)) | (2 if mi16 else 0)
    check(lib().hero_peak_mfma(mode, iters, workgroups, ptr(sink), stream, ctypes.byref(flop)), "hero_peak_mfma")
    return flop.value


def hero_peak_read(src, nbytes: int, visit_bytes: int, sink, stream) -> None:
    """Launch the HBM read probe over nbytes of src on `stream` (0: contiguous; 128/256/512: row visits)."""
    check(lib().hero_peak_read(ptr(src), nbytes, visit_bytes, ptr(sink), stream), "hero_peak_read")


def hero_kernel_timer(kernel: int, start_events: Sequence[int], stop_events: Sequence[int]) -> None:
    """Attach caller-created hipEvent_t handles around every launch of one kernel (empty: detach)."""
    n = len(start_events)
    a = (_vp * max(n, 1))(*start_events)
    b = (_vp * max(n, 1))(*stop_events)
    check(lib().hero_kernel_timer(kernel, a, b, n), "hero_kernel_timer")


def hero_workspace_size(dims: hero_dims, T: int, for_stack: bool) -> int:
    out = ctypes.c_size_t(0)
    check(lib().hero_workspace_size(ctypes.byref(dims), T, int(bool(for_stack)), ctypes.byref(out)),
          "hero_workspace_size")
    return out.value


def _byref(s):
    return None if s is None else ctypes.byref(s)


def hero_routed_layer(dims: hero_dims, j: int, T: int, hbar, hbar_prev1, hbar_prev2, h_out,
                      state: hero_state, ffn: hero_ffn_weights, router: hero_router_weights,
                      adapter: hero_adapter_weights, eta: float, routing: hero_routing,
                      stats: Optional[hero_layer_stats], workspace, workspace_bytes: int,
                      stream=None) -> int:
    """Enqueue one routed layer; returns the hero_status code."""
    return lib().hero_routed_layer(ctypes.byref(dims), j, T, ptr(hbar), ptr(hbar_prev1), ptr(hbar_prev2),
                                   ptr(h_out), _byref(state), _byref(ffn), _byref(router), _byref(adapter),
                                   float(eta), _byref(routing), _byref(stats), ptr(workspace),
                                   int(workspace_bytes), stream)


def hero_routed_layer_noalloc(dims: hero_dims, j: int, T: int, hbar, hbar_prev1, hbar_prev2, h_out,
                              state: hero_state, ffn: hero_ffn_weights, router: hero_router_weights,
                              adapter: hero_adapter_weights, eta: float, routing: hero_routing,
                              stats: Optional[hero_layer_stats], stream=None) -> int:
    """Enqueue one routed layer on the library's fixed device scratch (no workspace, nothing
    allocated); returns the hero_status code."""
    return lib().hero_routed_layer_noalloc(ctypes.byref(dims), j, T, ptr(hbar), ptr(hbar_prev1),
                                           ptr(hbar_prev2), ptr(h_out), _byref(state), _byref(ffn),
                                           _byref(router), _byref(adapter), float(eta), _byref(routing),
                                           _byref(stats), stream)


def hero_routed_stack(dims: hero_dims, T: int, h_in, h_out, state: hero_state,
                      ffn: Sequence[hero_ffn_weights], router: hero_router_weights,
                      adapter: Sequence[hero_adapter_weights], eta: Sequence[float],
                      routing: hero_routing, stats: Optional[Sequence[hero_layer_stats]],
                      workspace, workspace_bytes: int, stream=None) -> int:
    """Enqueue the whole routed stack; returns the hero_status code."""
    L = len(ffn)
    ffn_arr = (hero_ffn_weights * L)(*ffn)
    ad_arr = (hero_adapter_weights * L)(*adapter)
    eta_arr = (ctypes.c_float * L)(*[float(e) for e in eta])
    st_arr = None if stats is None else (hero_layer_stats * L)(*stats)
    return lib().hero_routed_stack(ctypes.byref(dims), T, ptr(h_in), ptr(h_out), _byref(state), ffn_arr,
                                   _byref(router), ad_arr, eta_arr, _byref(routing), st_arr,
                                   ptr(workspace), int(workspace_bytes), stream)


def _floats(xs):
    xs = [float(x) for x in xs]
    return (ctypes.c_float * max(len(xs), 1))(*xs)


def hero_routed_layer_hist(dims: hero_dims, j: int, T: int, hbar, hbar_prev1, hbar_prev2, h_out,
                           history: hero_history, ffn: hero_ffn_weights, router: hero_router_weights,
                           adapter: hero_adapter_weights, eta: Sequence[float], routing: hero_routing,
                           stats: Optional[hero_layer_stats], workspace, workspace_bytes: int,
                           stream=None) -> int:
    """One routed layer with the memory in depth-history form; eta holds eta_1 .. eta_j."""
    return lib().hero_routed_layer_hist(ctypes.byref(dims), j, T, ptr(hbar), ptr(hbar_prev1), ptr(hbar_prev2),
                                        ptr(h_out), _byref(history), _byref(ffn), _byref(router),
                                        _byref(adapter), _floats(eta), _byref(routing), _byref(stats),
                                        ptr(workspace), int(workspace_bytes), stream)


def hero_routed_stack_hist(dims: hero_dims, T: int, h_in, h_out, history: hero_history,
                           ffn: Sequence[hero_ffn_weights], router: hero_router_weights,
                           adapter: Sequence[hero_adapter_weights], eta: Sequence[float],
                           routing: hero_routing, stats: Optional[Sequence[hero_layer_stats]],
                           workspace, workspace_bytes: int, stream=None) -> int:
    """The routed stack with the memory in depth-history form."""
    L = len(ffn)
    ffn_arr = (hero_ffn_weights * L)(*ffn)
    ad_arr = (hero_adapter_weights * L)(*adapter)
    st_arr = None if stats is None else (hero_layer_stats * L)(*stats)
    return lib().hero_routed_stack_hist(ctypes.byref(dims), T, ptr(h_in), ptr(h_out), _byref(history), ffn_arr,
                                        _byref(router), ad_arr, _floats(eta), _byref(routing), st_arr,
                                        ptr(workspace), int(workspace_bytes), stream)


def hero_history_state(dims: hero_dims, n: int, T: int, kv, eta: Sequence[float], S, zeta, stream=None) -> int:
    """Matrix-form state after n layers from a history (eta: eta_1 .. eta_n)."""
    return lib().hero_history_state(ctypes.byref(dims), n, T, ptr(kv), _floats(eta), ptr(S), ptr(zeta), stream)


def hero_decoder_workspace_size(dims: hero_dims, adims: hero_attn_dims, n_layers: int, batch: int,
                                seq: int) -> int:
    out = ctypes.c_size_t(0)
    check(lib().hero_decoder_workspace_size(ctypes.byref(dims), ctypes.byref(adims), n_layers, batch, seq,
                                            ctypes.byref(out)), "hero_decoder_workspace_size")
    return out.value


def hero_attention_block(dims: hero_dims, adims: hero_attn_dims, batch: int, seq: int, h, hbar,
                         attn: hero_attn_weights, inv_freq: Sequence[float], workspace, workspace_bytes: int,
                         stream=None) -> int:
    """hbar = h + Attn(LN^attn(h)) for batch x seq tokens; inv_freq: head_dim / 2 host floats."""
    return lib().hero_attention_block(ctypes.byref(dims), _byref(adims), batch, seq, ptr(h), ptr(hbar),
                                      _byref(attn), None if inv_freq is None else _floats(inv_freq),
                                      ptr(workspace), int(workspace_bytes), stream)


def hero_decoder_stack(dims: hero_dims, adims: hero_attn_dims, n_layers: int, batch: int, seq: int, h_in, h_out,
                       state: hero_state, attn: Sequence[hero_attn_weights], ffn: Sequence[hero_ffn_weights],
                       router: hero_router_weights, adapter: Sequence[hero_adapter_weights],
                       eta: Sequence[float], inv_freq: Sequence[float], routing: hero_routing,
                       stats: Optional[Sequence[hero_layer_stats]], workspace, workspace_bytes: int,
                       stream=None) -> int:
    """n_layers decoder blocks, the last len(adapter) of them routed."""
    n, L = len(attn), len(adapter)
    at_arr = (hero_attn_weights * n)(*attn)
    ffn_arr = (hero_ffn_weights * n)(*ffn)
    ad_arr = (hero_adapter_weights * max(L, 1))(*adapter)
    st_arr = None if stats is None else (hero_layer_stats * max(L, 1))(*stats)
    return lib().hero_decoder_stack(ctypes.byref(dims), _byref(adims), n_layers, batch, seq, ptr(h_in), ptr(h_out),
                                    _byref(state), at_arr, ffn_arr, _byref(router), ad_arr, _floats(eta),
                                    _floats(inv_freq), _byref(routing), st_arr, ptr(workspace),
                                    int(workspace_bytes), stream)


def hero_ffn_decode_weights_make(dims: hero_dims, ffn: hero_ffn_weights, w_gate_up_tiled, w_down_tiled,
                                 stream=None) -> int:
    return lib().hero_ffn_decode_weights_make(ctypes.byref(dims), _byref(ffn), ptr(w_gate_up_tiled),
                                              ptr(w_down_tiled), stream)


def hero_ffn_backward_weights_make(dims: hero_dims, ffn: hero_ffn_weights, w_down_t, w_gate_up_t,
                                   stream=None) -> int:
    """Fill the transposed copies W_d^T [d_ff][d] and [W_g; W_u]^T [d][2 d_ff] of a frozen FFN."""
    return lib().hero_ffn_backward_weights_make(ctypes.byref(dims), _byref(ffn), ptr(w_down_t), ptr(w_gate_up_t),
                                                stream)


def hero_backward_workspace_size(dims: hero_dims, T: int) -> int:
    out = ctypes.c_size_t(0)
    check(lib().hero_backward_workspace_size(ctypes.byref(dims), T, ctypes.byref(out)),
          "hero_backward_workspace_size")
    return out.value


def hero_routed_block_backward(dims: hero_dims, T: int, hbar, dh_out, gate, idx_ffn, idx_ad, counts,
                               routing: Optional[hero_routing], dgate_in, ffn: hero_ffn_weights,
                               ffn_t: hero_ffn_backward_weights, adapter: hero_adapter_weights,
                               grads: hero_block_grads, workspace, workspace_bytes: int, stream=None) -> int:
    """Gradients of one routed block given dL/dh_out (the forward's gate, branch lists and routing rule)."""
    return lib().hero_routed_block_backward(ctypes.byref(dims), T, ptr(hbar), ptr(dh_out), ptr(gate), ptr(idx_ffn),
                                            ptr(idx_ad), ptr(counts), _byref(routing), ptr(dgate_in), _byref(ffn),
                                            _byref(ffn_t),
                                            _byref(adapter), _byref(grads), ptr(workspace), int(workspace_bytes),
                                            stream)


def hero_skip_penalty(L_R: int, batch: int, seq: int, gates, alpha: float, loss, dgates, stream=None) -> int:
    """alpha L_skip (Eq. 18) into loss[0] and its gradient over gates [L_R][batch seq]."""
    return lib().hero_skip_penalty(L_R, batch, seq, ptr(gates), float(alpha), ptr(loss), ptr(dgates), stream)


def hero_router_backward_workspace_size(dims: hero_dims, T: int) -> int:
    out = ctypes.c_size_t(0)
    check(lib().hero_router_backward_workspace_size(ctypes.byref(dims), T, ctypes.byref(out)),
          "hero_router_backward_workspace_size")
    return out.value


def hero_router_backward(dims: hero_dims, j: int, T: int, hbar, hbar_prev1, hbar_prev2, state_in: hero_state,
                         router: hero_router_weights, eta: float, dlogit, carry: hero_router_carry, dhbar,
                         dhbar_prev1, dhbar_prev2, grads: hero_router_grads, deta, workspace, workspace_bytes: int,
                         stream=None) -> int:
    """Enqueue the router's backward at routed layer j; returns the hero_status code."""
    return lib().hero_router_backward(ctypes.byref(dims), j, T, ptr(hbar), ptr(hbar_prev1), ptr(hbar_prev2),
                                      _byref(state_in), _byref(router), float(eta), ptr(dlogit), _byref(carry),
                                      ptr(dhbar), ptr(dhbar_prev1), ptr(dhbar_prev2), _byref(grads), ptr(deta),
                                      ptr(workspace), workspace_bytes, stream)
