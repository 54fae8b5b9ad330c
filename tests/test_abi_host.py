"""Host-side checks of libhero.so that need no GPU.

The library must load and export every function include/hero.h declares, and
every argument check must return its documented status before any HIP call.
Device pointers here are fake aligned addresses: each call is invalid in exactly
one way, so validation rejects it before the device check and nothing is ever
launched, on a machine with or without a GPU.
"""
import ctypes
import os
import re

import pytest

from paper_2609_08189_amd import hero as H

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
FAKE = 0x7F0000000000   # aligned, never dereferenced


def declared_functions():
    text = open(os.path.join(ROOT, "include", "hero.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(hero_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_function():
    names = declared_functions()
    assert {"hero_routed_layer", "hero_routed_stack", "hero_workspace_size"} <= set(names)
    lib = H.lib()
    for n in names:
        assert hasattr(lib, n), f"{n} declared in include/hero.h but not exported"
    assert H.hero_abi_version() == H.ABI_VERSION == 7


def test_status_strings():
    for code in range(12):
        assert H.hero_status_string(code) != "unknown status"
    assert H.hero_status_string(99) == "unknown status"


def good_dims(dtype=H.HERO_BF16, **kw):
    d = dict(d=512, d_ff=1408, d_r=64, L_R=8, d_m=128, d_s=64, d_h=48, d_a=16, d_e=256, d_p=64,
             d_head=256, dtype=dtype, eps_norm=1e-5, eps=1e-6, T_hist=0.9)
    d.update(kw)
    return H.hero_dims(**d)


def fake_structs(L=1):
    a = iter(range(1, 1000))
    nxt = lambda: FAKE + 4096 * next(a)
    ffn = [H.hero_ffn_weights(nxt(), nxt(), nxt(), nxt()) for _ in range(L)]
    ad = [H.hero_adapter_weights(nxt(), nxt()) for _ in range(L)]
    rt = H.hero_router_weights(**{k: nxt() for k in H.ROUTER_FIELDS})
    st = H.hero_state(nxt(), nxt(), nxt(), nxt())
    return ffn, ad, rt, st


def call_layer(dims=None, j=3, T=100, routing=None, ws_bytes=None, **over):
    dims = dims or good_dims()
    ffn, ad, rt, st = fake_structs()
    routing = routing or H.hero_routing(H.HERO_MODE_BUDGET, 0.5, 0.27, None)
    need = ctypes.c_size_t(0)
    if H.lib().hero_workspace_size(ctypes.byref(dims), max(T, 1), 0, ctypes.byref(need)) != H.HERO_OK:
        need.value = 1 << 20
    args = dict(hbar=FAKE + (1 << 30), prev1=FAKE + (2 << 30), prev2=FAKE + (3 << 30),
                h_out=FAKE + (4 << 30), state=st, ffn=ffn[0], router=rt, adapter=ad[0], eta=3.89,
                routing=routing, stats=None, ws=FAKE + (8 << 30),
                ws_bytes=need.value if ws_bytes is None else ws_bytes)
    args.update(over)
    return H.hero_routed_layer(dims, j, T, args["hbar"], args["prev1"], args["prev2"], args["h_out"],
                               args["state"], args["ffn"], args["router"], args["adapter"], args["eta"],
                               args["routing"], args["stats"], args["ws"], args["ws_bytes"], None)


@pytest.mark.parametrize("field,value,status", [
    ("dtype", 7, H.HERO_E_DTYPE),
    ("d", 0, H.HERO_E_DIM),
    ("d_ff", -1, H.HERO_E_DIM),
    ("d_s", 63, H.HERO_E_DIM),          # d_s != d_h + d_a
    ("eps", 0.0, H.HERO_E_RANGE),
    ("T_hist", -1.0, H.HERO_E_RANGE),
    ("d_m", 48, H.HERO_E_UNSUPPORTED),
    ("d", 640, H.HERO_E_UNSUPPORTED),    # bf16 needs d % 256 == 0
    ("d_ff", 688, H.HERO_E_UNSUPPORTED),  # bf16 needs d_ff % 128 == 0
    ("d_r", 16, H.HERO_E_UNSUPPORTED),
    ("d_e", 512, H.HERO_E_UNSUPPORTED),
    ("state_dtype", 5, H.HERO_E_DTYPE),
])
def test_dims_validation(field, value, status):
    assert call_layer(good_dims(**{field: value})) == status


def test_f32_accepts_ragged_widths_bf16_does_not():
    need = ctypes.c_size_t(0)
    dims = good_dims(H.HERO_F32, d=256, d_ff=688, d_r=16, d_m=32)
    assert H.lib().hero_workspace_size(ctypes.byref(dims), 64, 1, ctypes.byref(need)) == H.HERO_OK
    dims = good_dims(H.HERO_BF16, d=256, d_ff=688, d_r=16, d_m=32)
    assert H.lib().hero_workspace_size(ctypes.byref(dims), 64, 1, ctypes.byref(need)) == H.HERO_E_UNSUPPORTED
    # bf16 router weights are read as 16-byte rows: d_s must be a multiple of 8
    dims = good_dims(H.HERO_BF16, d_s=66, d_h=50)
    assert H.lib().hero_workspace_size(ctypes.byref(dims), 64, 1, ctypes.byref(need)) == H.HERO_E_UNSUPPORTED
    dims = good_dims(H.HERO_F32, d_s=66, d_h=50)
    assert H.lib().hero_workspace_size(ctypes.byref(dims), 64, 1, ctypes.byref(need)) == H.HERO_OK


def test_th1_pitch_macro_matches_harness():
    from paper_2609_08189_amd import device, synth
    w = synth.WORKLOADS["llama31_8b_layer"]
    assert device.th1_pitch(w) == 200 and device.th1_pitch(w) % 8 == 0
    assert device.th1_pitch(w.replace(d_s=64, d_m=32)) == 104
    text = open(os.path.join(ROOT, "include", "hero.h")).read()
    assert "#define HERO_TH1_PITCH(d_s, d_m) ((((d_s) + (d_m) + 1) + 7) / 8 * 8)" in text


def test_argument_validation():
    assert call_layer(T=0) == H.HERO_E_DIM
    assert call_layer(j=0) == H.HERO_E_RANGE
    assert call_layer(j=9) == H.HERO_E_RANGE
    assert call_layer(hbar=None) == H.HERO_E_NULL
    assert call_layer(h_out=None) == H.HERO_E_NULL
    assert call_layer(j=2, prev1=None) == H.HERO_E_NULL
    assert call_layer(j=3, prev2=None) == H.HERO_E_NULL
    assert call_layer(hbar=FAKE + 8) == H.HERO_E_ALIGN
    assert call_layer(h_out=FAKE + (1 << 30) + 512) == H.HERO_E_ALIAS       # overlaps hbar
    assert call_layer(h_out=FAKE + (2 << 30)) == H.HERO_E_ALIAS              # is hbar_prev1
    assert call_layer(state=None) == H.HERO_E_NULL
    ffn, ad, rt, st = fake_structs()
    st.S = None
    assert call_layer(state=st) == H.HERO_E_NULL
    ffn[0].w_down = None
    assert call_layer(ffn=ffn[0]) == H.HERO_E_NULL
    rt.th1 = FAKE + 2
    assert call_layer(router=rt) == H.HERO_E_ALIGN
    assert call_layer(eta=float("nan")) == H.HERO_E_RANGE
    assert call_layer(ws=None) == H.HERO_E_WORKSPACE
    assert call_layer(ws_bytes=1024) == H.HERO_E_WORKSPACE
    stats = H.hero_layer_stats(FAKE + 4, None, None, None, None, None, None)
    assert call_layer(stats=stats) == H.HERO_E_ALIGN


@pytest.mark.parametrize("routing,status", [
    (H.hero_routing(H.HERO_MODE_THRESHOLD, 0.0, 0.0, None), H.HERO_E_RANGE),
    (H.hero_routing(H.HERO_MODE_THRESHOLD, 1.0, 0.0, None), H.HERO_E_RANGE),
    (H.hero_routing(H.HERO_MODE_BUDGET, 0.5, -0.1, None), H.HERO_E_RANGE),
    (H.hero_routing(H.HERO_MODE_BUDGET, 0.5, 1.5, None), H.HERO_E_RANGE),
    (H.hero_routing(5, 0.5, 0.5, None), H.HERO_E_RANGE),
    (H.hero_routing(H.HERO_MODE_BUDGET, 0.5, 0.5, FAKE + 6), H.HERO_E_ALIGN),
    (H.hero_routing(H.HERO_MODE_BUDGET, 0.5, 0.5, None, 16), H.HERO_E_RANGE),     # unknown ablation bit
    (H.hero_routing(H.HERO_MODE_BUDGET, 0.5, 0.5, None, -1), H.HERO_E_RANGE),
])
def test_routing_validation(routing, status):
    assert call_layer(routing=routing) == status


def test_j1_and_j2_do_not_need_history():
    # with prev pointers absent, j = 1 and j = 2 pass the NULL checks and stop at the workspace
    assert call_layer(j=1, prev1=None, prev2=None, ws=None) == H.HERO_E_WORKSPACE
    assert call_layer(j=2, prev2=None, ws=None) == H.HERO_E_WORKSPACE


def test_stack_validation():
    L = 4
    dims = good_dims(L_R=L)
    ffn, ad, rt, st = fake_structs(L)
    rc = H.hero_routing(H.HERO_MODE_BUDGET, 0.5, 0.3, None)
    need = H.hero_workspace_size(dims, 100, True)

    def call(**kw):
        a = dict(h_in=FAKE + (1 << 30), h_out=FAKE + (4 << 30), ffn=ffn, ad=ad, eta=[3.9] * L,
                 ws=FAKE + (8 << 30), ws_bytes=need, st=st, rc=rc)
        a.update(kw)
        return H.hero_routed_stack(dims, 100, a["h_in"], a["h_out"], a["st"], a["ffn"], rt, a["ad"], a["eta"],
                                   a["rc"], None, a["ws"], a["ws_bytes"], None)

    assert call(h_out=FAKE + (1 << 30)) == H.HERO_E_ALIAS
    assert call(ws_bytes=need - 1) == H.HERO_E_WORKSPACE
    assert call(eta=[3.9, float("nan"), 3.9, 3.9]) == H.HERO_E_RANGE
    bad = list(ffn)
    bad[2] = H.hero_ffn_weights(FAKE, FAKE, None, FAKE)
    assert call(ffn=bad) == H.HERO_E_NULL
    # the output may not sit inside the workspace (its ring holds the layer-to-layer states)
    assert call(h_out=FAKE + (8 << 30) + 4096) == H.HERO_E_ALIAS


def test_operand_spans_past_32_bit_offsets_are_rejected():
    """The bf16 GEMM core addresses operand rows with 32-bit byte offsets: the layer, the stack and
    the decoder entry points reject shapes where an operand would span 4 GiB or more, before any
    other use of their arguments."""
    dims = good_dims(d=256, d_ff=1 << 16)          # act rows: T x 65536 x 2 B, 4 GiB at T = 32768
    assert call_layer(dims, T=32768) == H.HERO_E_UNSUPPORTED
    assert call_layer(dims, T=32767, ws=None) == H.HERO_E_WORKSPACE   # passes on to the next check
    assert call_layer(good_dims(d=4096, d_ff=1 << 19), T=1) == H.HERO_E_UNSUPPORTED   # 4 GiB of W_g
    # the fp32 path addresses rows with 64-bit offsets
    d32 = good_dims(H.HERO_F32, d=256, d_ff=1 << 16)
    assert call_layer(d32, T=32768, ws=None) == H.HERO_E_WORKSPACE
    ffn, ad, rt, st = fake_structs(dims.L_R)
    rc = H.hero_routing(H.HERO_MODE_BUDGET, 0.5, 0.3, None)
    assert H.hero_routed_stack(dims, 32768, FAKE, FAKE + (1 << 40), st, ffn, rt, ad, [3.9] * dims.L_R,
                               rc, None, None, 0, None) == H.HERO_E_UNSUPPORTED
    # decoder: the attention output [T][n_h x 128] of 64 heads spans 4 GiB at T = 262144
    out = ctypes.c_size_t(0)
    adims = H.hero_attn_dims(64, 8, 128)
    ws = lambda b, s: H.lib().hero_decoder_workspace_size(ctypes.byref(good_dims(L_R=2)), ctypes.byref(adims),
                                                          4, b, s, ctypes.byref(out))
    assert ws(2, 131072) == H.HERO_E_UNSUPPORTED
    assert ws(2, 131071) == H.HERO_OK


def test_workspace_size_monotone_and_stack_larger():
    dims = good_dims()
    a = H.hero_workspace_size(dims, 100, False)
    b = H.hero_workspace_size(dims, 1000, False)
    c = H.hero_workspace_size(dims, 1000, True)
    assert 0 < a < b < c
    # the stack adds a three-deep ring of [T][d] post-attention states
    assert c - b >= 3 * 1000 * 512 * 2


def test_no_device_means_device_error():
    """All arguments valid: without a usable gfx950 device the call stops at the device check."""
    import torch
    if torch.cuda.device_count() > 0:
        pytest.skip("a GPU is visible; this test covers hosts without one")
    assert call_layer() == H.HERO_E_DEVICE


def test_memory_read_output_validates():
    """hero_state.c_read (the layer's memory read, T x d_m fp32) must be 16-byte aligned and may not
    overlap the state, the activations or the workspace; a disjoint one passes the host checks."""
    import torch
    _, _, _, st = fake_structs()
    with_c = lambda c: H.hero_state(st.S, st.zeta, st.p_hist, st.m_hist, c)
    assert call_layer(state=with_c(FAKE + (6 << 30) + 4)) == H.HERO_E_ALIGN
    assert call_layer(state=with_c(FAKE + (4 << 30) + 256)) == H.HERO_E_ALIAS    # inside h_out
    assert call_layer(state=with_c(FAKE + (1 << 30))) == H.HERO_E_ALIAS          # is hbar
    assert call_layer(state=with_c(FAKE + (8 << 30) + 4096)) == H.HERO_E_ALIAS   # inside the workspace
    assert call_layer(state=with_c(st.zeta)) == H.HERO_E_ALIAS
    # hbar_prev2 is not read at j = 2, so a c_read over it is no overlap there
    assert call_layer(j=2, state=with_c(FAKE + (3 << 30))) != H.HERO_E_ALIAS
    if torch.cuda.device_count() == 0:
        assert call_layer(state=with_c(FAKE + (6 << 30))) == H.HERO_E_DEVICE


def test_history_entry_points_validate():
    dims = good_dims()
    ffn, ad, rt, st = fake_structs()
    hist = H.hero_history(FAKE + (5 << 30), FAKE + (6 << 30), FAKE + (7 << 30))
    rc = H.hero_routing(H.HERO_MODE_BUDGET, 0.5, 0.27, None)
    need = H.hero_workspace_size(dims, 100, False)

    def layer(j=3, eta=(3.9, 3.9, 3.9), hs=hist, d=dims, ws=FAKE + (8 << 30)):
        return H.hero_routed_layer_hist(d, j, 100, FAKE + (1 << 30), FAKE + (2 << 30), FAKE + (3 << 30),
                                        FAKE + (4 << 30), hs, ffn[0], rt, ad[0], eta, rc, None, ws, need, None)

    assert layer(hs=None) == H.HERO_E_NULL
    assert layer(hs=H.hero_history(FAKE + (5 << 30), None, FAKE)) == H.HERO_E_NULL
    assert layer(hs=H.hero_history(FAKE + 4, FAKE, FAKE)) == H.HERO_E_ALIGN
    assert layer(eta=(3.9, float("nan"), 3.9)) == H.HERO_E_RANGE
    assert layer(d=good_dims(L_R=65), j=3) == H.HERO_E_UNSUPPORTED
    assert layer(d=good_dims(state_dtype=H.HERO_BF16)) == H.HERO_E_UNSUPPORTED   # matrix form only
    assert layer(ws=None) == H.HERO_E_WORKSPACE
    S, z = FAKE + (9 << 30), FAKE + (10 << 30)
    kv = FAKE + (5 << 30)
    assert H.hero_history_state(dims, 9, 10, kv, [3.9] * 9, S, z) == H.HERO_E_RANGE      # n > L_R
    assert H.hero_history_state(dims, 2, 10, kv, [3.9] * 2, kv, z) == H.HERO_E_ALIAS     # S overlaps kv
    assert H.hero_history_state(dims, 2, 0, kv, [3.9] * 2, S, z) == H.HERO_E_DIM
    assert H.hero_history_state(dims, 2, 10, None, [3.9] * 2, S, z) == H.HERO_E_NULL
    assert H.hero_history_state(good_dims(state_dtype=H.HERO_BF16), 2, 10, kv, [3.9] * 2, S, z) == \
        H.HERO_E_UNSUPPORTED


def test_bf16_state_needs_a_wide_memory():
    assert call_layer(good_dims(state_dtype=H.HERO_BF16, d_m=32)) == H.HERO_E_UNSUPPORTED
    # a valid bf16-state call gets past validation to the device check
    assert call_layer(good_dims(state_dtype=H.HERO_BF16, d_m=64)) == H.HERO_E_DEVICE


def test_decoder_entry_points_validate():
    dims = good_dims(L_R=2)
    ad = H.hero_attn_dims(4, 2, 128)
    need = H.hero_decoder_workspace_size(dims, ad, 4, 2, 300)
    assert need > H.hero_decoder_workspace_size(dims, ad, 0, 2, 300) > H.hero_workspace_size(dims, 600, False)
    out = ctypes.c_size_t(0)
    ws_call = lambda d, a, n=4, b=2, s=300: H.lib().hero_decoder_workspace_size(
        ctypes.byref(d), None if a is None else ctypes.byref(a), n, b, s, ctypes.byref(out))
    assert ws_call(dims, None) == H.HERO_E_NULL
    assert ws_call(dims, H.hero_attn_dims(4, 3, 128)) == H.HERO_E_DIM          # heads % kv heads
    assert ws_call(dims, H.hero_attn_dims(4, 2, 64)) == H.HERO_E_UNSUPPORTED   # head width 128 only
    assert ws_call(dims, H.hero_attn_dims(3, 3, 128)) == H.HERO_E_UNSUPPORTED  # odd head count
    assert ws_call(good_dims(H.HERO_F32, d=256, d_ff=688, d_r=16, d_m=32), ad) == H.HERO_E_UNSUPPORTED
    assert ws_call(dims, ad, b=0) == H.HERO_E_DIM

    aw = H.hero_attn_weights(FAKE + 4096, FAKE + 8192, FAKE + 12288)
    freq = [1.0] * 64
    h, hb, ws = FAKE + (1 << 30), FAKE + (2 << 30), FAKE + (8 << 30)

    need_attn = H.hero_decoder_workspace_size(dims, ad, 0, 2, 300)

    def attn(**kw):
        a = dict(d=dims, ad=ad, b=2, s=300, h=h, hb=hb, w=aw, f=freq, ws=ws, n=need_attn)
        a.update(kw)
        return H.hero_attention_block(a["d"], a["ad"], a["b"], a["s"], a["h"], a["hb"], a["w"], a["f"],
                                      a["ws"], a["n"])

    assert attn(h=None) == H.HERO_E_NULL
    assert attn(hb=h) == H.HERO_E_ALIAS
    assert attn(hb=hb + 2) == H.HERO_E_ALIGN
    assert attn(w=H.hero_attn_weights(FAKE, None, FAKE)) == H.HERO_E_NULL
    assert attn(f=None) == H.HERO_E_NULL
    assert attn(f=[1.0] * 63 + [float("inf")]) == H.HERO_E_RANGE
    assert attn(n=need_attn - 1) == H.HERO_E_WORKSPACE
    assert attn(ws=hb) == H.HERO_E_ALIAS
    assert attn() == H.HERO_E_DEVICE

    ffn, adp, rt, st = fake_structs(4)
    rc = H.hero_routing(H.HERO_MODE_BUDGET, 0.5, 0.3, None)

    def dec(n_layers=4, eta=(3.9, 3.9), adapters=adp[:2], **kw):
        a = dict(h_in=h, h_out=hb, ws=ws)
        a.update(kw)
        return H.hero_decoder_stack(dims, ad, n_layers, 2, 300, a["h_in"], a["h_out"], st, [aw] * n_layers,
                                    ffn[:n_layers] + ffn[:max(0, n_layers - 4)], rt, adapters, eta, freq, rc,
                                    None, a["ws"], need)

    assert dec(n_layers=1) == H.HERO_E_RANGE           # fewer blocks than routed layers
    assert dec(h_out=h) == H.HERO_E_ALIAS
    assert dec(eta=(3.9, float("nan"))) == H.HERO_E_RANGE
    assert dec() == H.HERO_E_DEVICE


def test_backward_entry_points_validate():
    """The training-side calls check every argument before the device check."""
    dims = good_dims()
    T = 300
    need = H.hero_backward_workspace_size(dims, T)
    assert need > H.hero_backward_workspace_size(dims, T - 100) > 0
    ffn, ad, rt, st = fake_structs()
    hb, dh, gate = FAKE + (1 << 30), FAKE + (2 << 30), FAKE + (3 << 30)
    fi, ai, cnt = FAKE + (3 << 30) + 4096, FAKE + (3 << 30) + 8192, FAKE + (3 << 30) + 12288
    ft = H.hero_ffn_backward_weights(FAKE + (5 << 30), FAKE + (6 << 30))
    g = H.hero_block_grads(FAKE + (4 << 30), FAKE + (7 << 30), FAKE + (7 << 30) + 4096,
                           FAKE + (7 << 30) + 8192, FAKE + (7 << 30) + (1 << 20))
    ws = FAKE + (8 << 30)

    def bwd(d=dims, T=T, hbar=hb, dh_out=dh, gate=gate, lists=(fi, ai, cnt), dgate_in=None, ffn_t=ft,
            grads=g, ws=ws, n=need, adapter=ad[0], routing=None):
        return H.hero_routed_block_backward(d, T, hbar, dh_out, gate, *lists, routing, dgate_in, ffn[0], ffn_t, adapter,
                                            grads, ws, n)

    assert bwd(T=0) == H.HERO_E_DIM
    assert bwd(d=good_dims(dtype=9)) == H.HERO_E_DTYPE
    assert bwd(hbar=None) == H.HERO_E_NULL
    assert bwd(lists=(fi, None, cnt)) == H.HERO_E_NULL
    assert bwd(ffn_t=H.hero_ffn_backward_weights(FAKE, None)) == H.HERO_E_NULL
    assert bwd(grads=H.hero_block_grads(FAKE + (4 << 30), None, FAKE, FAKE, FAKE)) == H.HERO_E_NULL
    assert bwd(adapter=H.hero_adapter_weights(FAKE, FAKE + 2)) == H.HERO_E_ALIGN
    assert bwd(dgate_in=FAKE + 6) == H.HERO_E_ALIGN
    assert bwd(grads=H.hero_block_grads(hb + 1024, FAKE, FAKE, FAKE, FAKE)) == H.HERO_E_ALIAS   # dhbar in hbar
    assert bwd(grads=H.hero_block_grads(dh, FAKE, FAKE, FAKE, FAKE)) == H.HERO_E_ALIAS
    assert bwd(ws=None) == H.HERO_E_WORKSPACE
    assert bwd(n=need - 1) == H.HERO_E_WORKSPACE
    assert bwd(ws=hb) == H.HERO_E_ALIAS
    assert bwd(grads=H.hero_block_grads(FAKE + (4 << 30), FAKE, FAKE, ws + 4096, FAKE + (7 << 30) + (1 << 20))) == \
        H.HERO_E_ALIAS                                                       # dW_1 inside the workspace
    assert bwd(grads=H.hero_block_grads(FAKE + (4 << 30), FAKE, FAKE, FAKE + (7 << 30) + 8192,
                                        FAKE + (7 << 30) + 8192 + 4096)) == H.HERO_E_ALIAS   # dW_1, dW_2 overlap
    # operand rows the GEMM core addresses with 32-bit offsets: [dG dU] of 2^17 tokens is too big
    assert bwd(d=good_dims(d_ff=8192), T=1 << 17, n=1 << 40) == H.HERO_E_UNSUPPORTED
    assert bwd(routing=H.hero_routing(H.HERO_MODE_BUDGET, 0.5, 1.5, None)) == H.HERO_E_RANGE
    assert bwd(routing=H.hero_routing(7, 0.5, 0.5, None)) == H.HERO_E_RANGE
    assert bwd() == H.HERO_E_DEVICE
    assert bwd(dgate_in=FAKE + (9 << 30)) == H.HERO_E_DEVICE
    assert bwd(routing=H.hero_routing(H.HERO_MODE_BUDGET, 0.5, 0.27, None)) == H.HERO_E_DEVICE

    wd, wgu = FAKE + (5 << 30), FAKE + (6 << 30)
    make = lambda f=ffn[0], a=wd, b=wgu, d=dims: H.hero_ffn_backward_weights_make(d, f, a, b)
    assert make(a=None) == H.HERO_E_NULL
    assert make(b=wgu + 8) == H.HERO_E_ALIGN
    assert make(a=ffn[0].w_down) == H.HERO_E_ALIAS
    assert make(b=wd) == H.HERO_E_ALIAS
    assert make(f=H.hero_ffn_weights(FAKE, FAKE, None, FAKE)) == H.HERO_E_NULL
    assert make() == H.HERO_E_DEVICE

    gates, loss, dg = FAKE + (1 << 30), FAKE + (2 << 30), FAKE + (3 << 30)
    assert H.hero_skip_penalty(0, 2, 5, gates, 1.0, loss, dg) == H.HERO_E_DIM
    assert H.hero_skip_penalty(4, 2, 0, gates, 1.0, loss, dg) == H.HERO_E_DIM
    assert H.hero_skip_penalty(4, 2, 5, None, 1.0, loss, dg) == H.HERO_E_NULL
    assert H.hero_skip_penalty(4, 2, 5, gates, float("nan"), loss, dg) == H.HERO_E_RANGE
    assert H.hero_skip_penalty(4, 2, 5, gates, 1.0, loss, gates + 16) == H.HERO_E_ALIAS
    assert H.hero_skip_penalty(4, 2, 5, gates, 1.0, loss + 4, dg) == H.HERO_E_ALIGN
    assert H.hero_skip_penalty(4, 2, 5, gates, 1.0, loss, dg) == H.HERO_E_DEVICE


def test_ffn_decode_weights_make_validates():
    """hero_ffn_decode_weights_make and the layer call's checks of the tiled weights (fake addresses)."""
    dims = good_dims()
    ffn, _, _, _ = fake_structs()
    f = ffn[0]
    gu, dn = FAKE + (5 << 30), FAKE + (6 << 30)
    make = lambda f=f, a=gu, b=dn, d=dims: H.hero_ffn_decode_weights_make(d, f, a, b)
    assert make(d=good_dims(H.HERO_F32)) == H.HERO_E_UNSUPPORTED
    assert make(f=H.hero_ffn_weights(FAKE, FAKE, None, FAKE)) == H.HERO_E_NULL
    assert make(a=gu + 8) == H.HERO_E_ALIGN
    assert make(b=dn + 8) == H.HERO_E_ALIGN
    assert make(a=f.w_up) == H.HERO_E_ALIAS
    assert make(b=f.w_down) == H.HERO_E_ALIAS
    assert make(b=gu + 2 * 512 * 1408 * 2 - 16) == H.HERO_E_ALIAS    # W_d's copy inside [W_g; W_u]'s
    assert make(b=gu + 2 * 512 * 1408 * 2) == H.HERO_E_DEVICE        # adjacent, not overlapping
    assert make(a=None) == H.HERO_E_DEVICE
    assert make() == H.HERO_E_DEVICE
    tiled = lambda a, b: H.hero_ffn_weights(f.norm_w, f.w_gate, f.w_up, f.w_down, a, b)
    assert call_layer(ffn=tiled(gu + 8, None)) == H.HERO_E_ALIGN
    assert call_layer(ffn=tiled(None, dn + 8)) == H.HERO_E_ALIGN
    assert call_layer(good_dims(H.HERO_F32), ffn=tiled(gu, dn)) == H.HERO_E_UNSUPPORTED
    assert call_layer(ffn=tiled(gu, dn)) == H.HERO_E_DEVICE


def test_router_backward_entry_validates():
    """hero_router_backward checks everything on the host before any launch (fake addresses)."""
    dims = good_dims(L_R=4)
    T = 64
    need = H.hero_router_backward_workspace_size(dims, T)
    assert need > 0
    _, _, rt, st = fake_structs()
    import itertools
    base = FAKE + (1 << 36)
    nxt = itertools.count(1)
    at = lambda: base + (next(nxt) << 28)
    grads = H.hero_router_grads(**{k: at() for k in H.ROUTER_FIELDS})
    carry = H.hero_router_carry(at(), at(), at(), at())

    def call(**kw):
        a = dict(d=dims, j=3, T=T, hb=at(), h1=at(), h2=at(), st=st, rt=rt, eta=3.9, dl=at(), carry=carry,
                 dh=at(), dh1=at(), dh2=at(), g=grads, deta=at(), ws=at(), n=need)
        a.update(kw)
        return H.hero_router_backward(a["d"], a["j"], a["T"], a["hb"], a["h1"], a["h2"], a["st"], a["rt"], a["eta"],
                                      a["dl"], a["carry"], a["dh"], a["dh1"], a["dh2"], a["g"], a["deta"], a["ws"],
                                      a["n"], None)

    assert call(j=0) == H.HERO_E_RANGE and call(j=5) == H.HERO_E_RANGE
    assert call(T=0) == H.HERO_E_DIM
    assert call(eta=float("nan")) == H.HERO_E_RANGE
    assert call(d=good_dims(L_R=4, state_dtype=H.HERO_BF16)) == H.HERO_E_UNSUPPORTED
    assert call(dl=None) == H.HERO_E_NULL
    assert call(h2=None) == H.HERO_E_NULL and call(j=2, h2=None, dh2=None) != H.HERO_E_NULL
    assert call(g=H.hero_router_grads(**{**{k: at() for k in H.ROUTER_FIELDS}, "th1": None})) == H.HERO_E_NULL
    assert call(carry=H.hero_router_carry(at(), None, at(), at())) == H.HERO_E_NULL
    assert call(dh=FAKE + 8) == H.HERO_E_ALIGN
    same = at()
    assert call(dh=same, dh1=same) == H.HERO_E_ALIAS
    # dL/dS_{j-1} is written over dL/dS_j while S_{j-1} is read: they may not overlap
    st2 = H.hero_state(carry.dS, st.zeta, st.p_hist, st.m_hist)
    assert call(st=st2) == H.HERO_E_ALIAS
    assert call(n=need - 1) == H.HERO_E_WORKSPACE
    assert call(ws=None) == H.HERO_E_WORKSPACE
    # the received state is not read at j = 1 and may be absent there, not later
    assert call(j=1, st=None, h1=None, h2=None, dh1=None, dh2=None, ws=None) == H.HERO_E_WORKSPACE
    assert call(j=2, st=None) == H.HERO_E_NULL
    # the forward's memory read, handed in as state_in.c_read, is read after outputs are written
    with_c = lambda c: H.hero_state(st.S, st.zeta, st.p_hist, st.m_hist, c)
    assert call(st=with_c(FAKE + 8)) == H.HERO_E_ALIGN
    assert call(st=with_c(carry.dzeta)) == H.HERO_E_ALIAS
    dh = at()
    assert call(dh=dh, st=with_c(dh + 1024)) == H.HERO_E_ALIAS
    ws = at()
    assert call(ws=ws, st=with_c(ws + need - 16)) == H.HERO_E_ALIAS
    # not read at j = 1
    assert call(j=1, st=with_c(carry.dzeta), h1=None, h2=None, dh1=None, dh2=None) != H.HERO_E_ALIAS
    import torch
    if torch.cuda.device_count() == 0:
        assert call(st=with_c(at())) == H.HERO_E_DEVICE


def test_noalloc_rejects_a_call_beyond_its_scratch_before_any_launch():
    """The no-alloc entry point's fixed scratch holds a 256-token decode batch of the Llama-2-7B
    shape but not a 4096-token Llama-3.1-8B layer: that call returns HERO_E_SCRATCH from the host
    checks (fake pointers, nothing launched); an argument error keeps its own status."""
    from paper_2609_08189_amd import synth
    from paper_2609_08189_amd.device import dims_struct
    assert H.HERO_NOALLOC_SCRATCH_BYTES == 64 << 20
    assert H.hero_workspace_size(dims_struct(synth.WORKLOADS["llama2_7b_decode"]), 256, False) \
        <= H.HERO_NOALLOC_SCRATCH_BYTES
    w = synth.WORKLOADS["llama31_8b_layer"]
    dims = dims_struct(w)
    assert H.hero_workspace_size(dims, 4096, False) > H.HERO_NOALLOC_SCRATCH_BYTES
    ffn, ad, rt, st = fake_structs()
    routing = H.hero_routing(H.HERO_MODE_BUDGET, 0.5, 0.27, None)
    call = lambda T, hbar: H.hero_routed_layer_noalloc(dims, 3, T, hbar, FAKE + (2 << 30), FAKE + (3 << 30),
                                                       FAKE + (4 << 30), st, ffn[0], rt, ad[0], 3.89,
                                                       routing, None, None)
    assert call(4096, FAKE + (1 << 30)) == H.HERO_E_SCRATCH
    assert call(4096, None) == H.HERO_E_NULL
    assert call(0, FAKE + (1 << 30)) == H.HERO_E_DIM
    assert H.hero_status_string(H.HERO_E_SCRATCH) != "unknown status"


def test_peak_hooks_reject_bad_arguments_before_any_launch():
    """The measurement hooks check their arguments on the host (fake pointers: nothing is launched)."""
    lib = H.lib()
    sink = ctypes.c_void_p(FAKE)
    flop = ctypes.c_double()
    assert lib.hero_peak_mfma(4, 10, 256, sink, None, ctypes.byref(flop)) == H.HERO_E_RANGE
    assert lib.hero_peak_mfma(3, 0, 256, sink, None, ctypes.byref(flop)) == H.HERO_E_RANGE
    assert lib.hero_peak_mfma(0, 10, 256, None, None, ctypes.byref(flop)) == H.HERO_E_NULL
    rows = 96 * 8192
    assert lib.hero_peak_read(None, rows, 128, sink, None) == H.HERO_E_NULL
    assert lib.hero_peak_read(ctypes.c_void_p(FAKE + 8), rows, 128, sink, None) == H.HERO_E_ALIGN
    assert lib.hero_peak_read(ctypes.c_void_p(FAKE), rows + 8192, 128, sink, None) == H.HERO_E_DIM
    assert lib.hero_peak_read(ctypes.c_void_p(FAKE), rows, 64, sink, None) == H.HERO_E_RANGE
    assert lib.hero_peak_read(ctypes.c_void_p(FAKE), 24, 0, sink, None) == H.HERO_E_DIM
