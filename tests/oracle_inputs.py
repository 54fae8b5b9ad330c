"""Convert a seeded synthetic problem into the CPU oracle's float64 parameters (test helper)."""
import numpy as np

from oracle import hero_oracle as O


def dims_of(w):
    return O.Dims(d=w.d, d_ff=w.d_ff, d_r=w.d_r, L_R=w.L_R, d_m=w.d_m, d_s=w.d_s, d_h=w.d_h,
                  d_a=w.d_a, d_e=w.d_e, d_p=w.d_p, d_head=w.d_head, eps_norm=w.eps_norm,
                  eps=w.eps, T_hist=w.T_hist, io_dtype=w.dtype, state_dtype=w.state_dtype)


def router_of(prob):
    r = prob.router
    return O.RouterParams(**{k: r[k].f64 for k in r})


def ffn_of(layer):
    return O.FFNParams(norm_w=layer["norm_w"].f64, w_gate=layer["w_gate"].f64,
                       w_up=layer["w_up"].f64, w_down=layer["w_down"].f64)


def adapter_of(layer):
    return O.AdapterParams(w1=layer["w1"].f64, w2=layer["w2"].f64)


def state_of(prob, rows=None):
    sl = slice(None) if rows is None else rows
    return O.State(prob.S[sl].astype("f8"), prob.zeta[sl].astype("f8"),
                   prob.p_hist[sl].astype("f8"), prob.m_hist[sl].astype("f8"))


def adims_of(w):
    return O.AttnDims(n_heads=w.n_heads, n_kv_heads=w.n_kv_heads, head_dim=w.head_dim)


def attn_of(layer, w, inv_freq):
    """Split the stored fused [W_q; W_k; W_v] into the oracle's three projections."""
    qkv = layer["w_qkv"].f64
    nq, nkv = w.n_heads * w.head_dim, w.n_kv_heads * w.head_dim
    return O.AttnParams(norm_w=layer["norm_w"].f64, w_q=qkv[:nq], w_k=qkv[nq:nq + nkv],
                        w_v=qkv[nq + nkv:], w_o=layer["w_o"].f64,
                        inv_freq=np.asarray(inv_freq, dtype=np.float64))
