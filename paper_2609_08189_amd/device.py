"""Device-side harness: uploads a seeded problem with torch and drives the C ABI.

torch supplies device memory and the stream; every step of the routed layer runs
in libhero.so.  This module only allocates buffers, fills the ABI structs and
copies results back for inspection.
"""
from __future__ import annotations

from typing import Dict, List, Optional

import numpy as np
import torch

from . import hero as H
from . import synth


def upload(t: synth.Tensor, device) -> torch.Tensor:
    if t.dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(t.store).view(np.int16)).to(device).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(t.store)).to(device)


def download_f64(x: torch.Tensor) -> np.ndarray:
    """Exact float64 values of a bf16 or fp32 device tensor."""
    if x.dtype == torch.bfloat16:
        return synth.bf16_bits_to_f64(x.view(torch.int16).cpu().numpy().view(np.uint16))
    return x.float().cpu().numpy().astype(np.float64)


def th1_pitch(w: synth.Workload) -> int:
    """Row pitch of the history head's input layer in the ABI layout (a multiple of 8)."""
    return (w.d_s + w.d_m + 1 + 7) // 8 * 8


def pad_th1(t: synth.Tensor, w: synth.Workload) -> synth.Tensor:
    """th1 [d_head][d_s + d_m + 1] with zero columns appended up to the ABI row pitch."""
    pad = th1_pitch(w) - t.store.shape[1]
    return synth.Tensor(np.pad(t.store, ((0, 0), (0, pad))), t.dtype)


def dims_struct(w: synth.Workload) -> H.hero_dims:
    return H.hero_dims(d=w.d, d_ff=w.d_ff, d_r=w.d_r, L_R=w.L_R, d_m=w.d_m, d_s=w.d_s, d_h=w.d_h,
                       d_a=w.d_a, d_e=w.d_e, d_p=w.d_p, d_head=w.d_head,
                       dtype=H.HERO_BF16 if w.dtype == "bf16" else H.HERO_F32,
                       eps_norm=w.eps_norm, eps=w.eps, T_hist=w.T_hist,
                       state_dtype=H.HERO_BF16 if w.state_dtype == "bf16" else H.HERO_F32)


class LayerStats:
    """Per-layer device outputs of the ABI's optional stats."""

    def __init__(self, T: int, device):
        self.mask = torch.empty(T, dtype=torch.uint8, device=device)
        self.idx_ffn = torch.empty(T, dtype=torch.int32, device=device)
        self.idx_ad = torch.empty(T, dtype=torch.int32, device=device)
        self.counts = torch.empty(4, dtype=torch.int32, device=device)
        self.logit = torch.empty(T, dtype=torch.float32, device=device)
        self.gate = torch.empty(T, dtype=torch.float32, device=device)
        self.lam = torch.empty(4, dtype=torch.float32, device=device)
        self.struct = H.hero_layer_stats(self.mask.data_ptr(), self.idx_ffn.data_ptr(),
                                         self.idx_ad.data_ptr(), self.counts.data_ptr(),
                                         self.logit.data_ptr(), self.gate.data_ptr(), self.lam.data_ptr())

    def host(self) -> Dict[str, np.ndarray]:
        c = self.counts.cpu().numpy()
        return dict(mask=self.mask.cpu().numpy().astype(bool), idx_ffn=self.idx_ffn.cpu().numpy(),
                    idx_ad=self.idx_ad.cpu().numpy(), n_ffn=int(c[0]), n_ad=int(c[1]),
                    logit=self.logit.cpu().numpy(), gate=self.gate.cpu().numpy(),
                    lam=float(self.lam.cpu().numpy()[0]))


def make_tiled(dims: H.hero_dims, ffn: List[Dict[str, torch.Tensor]], ffn_s: List[H.hero_ffn_weights],
               device) -> None:
    """The FFN weights' copies in the decode products' streaming order (hero_ffn_decode_weights_make),
    kept in ffn[i] and pointed at by ffn_s[i]."""
    stream = torch.cuda.current_stream(torch.device(device)).cuda_stream
    for f, fs in zip(ffn, ffn_s):
        f["w_gate_up_tiled"] = torch.empty(2 * f["w_gate"].numel(), dtype=f["w_gate"].dtype, device=device)
        f["w_down_tiled"] = torch.empty(f["w_down"].numel(), dtype=f["w_down"].dtype, device=device)
        fs.w_gate_up_tiled = f["w_gate_up_tiled"].data_ptr()
        fs.w_down_tiled = f["w_down_tiled"].data_ptr()
        H.check(H.hero_ffn_decode_weights_make(dims, fs, f["w_gate_up_tiled"], f["w_down_tiled"], stream),
                "hero_ffn_decode_weights_make")


class DeviceProblem:
    """A synth.Problem resident on the GPU with the ABI structs that point at it."""

    def __init__(self, prob: synth.Problem, device: str = "cuda:0", stats: bool = True,
                 for_stack: Optional[bool] = None, history: bool = False, tiled: bool = False):
        w = prob.w
        self.w = w
        self.device = device
        self.T = T = prob.hbar.shape[0]
        self.dims = dims_struct(w)
        self.hbar = upload(prob.hbar, device)
        self.prev1 = upload(prob.hbar_prev1, device) if prob.hbar_prev1 is not None else None
        self.prev2 = upload(prob.hbar_prev2, device) if prob.hbar_prev2 is not None else None
        self.h_out = torch.empty_like(self.hbar)
        self.router = {k: upload(v if k != "th1" else pad_th1(v, w), device) for k, v in prob.router.items()}
        self.router_s = H.hero_router_weights(**{k: self.router[k].data_ptr() for k in H.ROUTER_FIELDS})
        # weights are drawn and uploaded one layer at a time
        self.ffn = [{k: upload(v, device) for k, v in prob.ffn[i].items()} for i in range(len(prob.ffn))]
        self.ffn_s = [H.hero_ffn_weights(f["norm_w"].data_ptr(), f["w_gate"].data_ptr(),
                                         f["w_up"].data_ptr(), f["w_down"].data_ptr()) for f in self.ffn]
        self.tiled = tiled
        if tiled:
            make_tiled(self.dims, self.ffn, self.ffn_s, device)
        self.adapter = [{k: upload(v, device) for k, v in prob.adapter[i].items()}
                        for i in range(len(prob.adapter))]
        self.adapter_s = [H.hero_adapter_weights(a["w1"].data_ptr(), a["w2"].data_ptr()) for a in self.adapter]
        self.eta = [float(e) for e in prob.eta]
        # S in its storage dtype (the synthetic bf16 state is bf16-exact, so the cast is exact)
        self.S = torch.from_numpy(prob.S).to(device)
        if w.state_dtype == "bf16":
            self.S = self.S.to(torch.bfloat16)
        self.zeta = torch.from_numpy(prob.zeta).to(device)
        self.p_hist = torch.from_numpy(prob.p_hist).to(device)
        self.m_hist = torch.from_numpy(prob.m_hist).to(device)
        self.state_s = H.hero_state(self.S.data_ptr(), self.zeta.data_ptr(), self.p_hist.data_ptr(),
                                    self.m_hist.data_ptr())
        # depth-history form of the memory: the pairs of the earlier layers instead of S, zeta
        self.history = history
        self.n_entries = 0
        if history:
            self.kv = torch.full((T, w.L_R, 2, w.d_m), float("nan"), dtype=torch.float32, device=device)
            if prob.mem_k is not None:
                n = prob.mem_k.shape[1]
                self.kv[:, :n, 0] = torch.from_numpy(prob.mem_k).to(device)
                self.kv[:, :n, 1] = torch.from_numpy(prob.mem_v).to(device)
                self.n_entries = n
            self.hist_s = H.hero_history(self.kv.data_ptr(), self.p_hist.data_ptr(), self.m_hist.data_ptr())
        self.beta = torch.from_numpy(prob.beta).to(device) if prob.beta is not None else None
        mode = H.HERO_MODE_BUDGET if w.mode == "budget" else H.HERO_MODE_THRESHOLD
        self.routing_s = H.hero_routing(mode, w.tau, w.budget,
                                        self.beta.data_ptr() if self.beta is not None else None,
                                        w.ablation)
        if for_stack is None:
            for_stack = w.layer_j <= 0      # a stack workload (a layer workload names its j)
        self.for_stack = for_stack
        self.stats = [LayerStats(T, device) for _ in range(w.L_R if for_stack else 1)] if stats else None
        self.ws_bytes = H.hero_workspace_size(self.dims, T, for_stack)
        self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device=device)

    def stream(self):
        return torch.cuda.current_stream(torch.device(self.device)).cuda_stream

    def run_layer(self, j: int, layer: int = 0, check: bool = True) -> int:
        stats = self.stats[0].struct if self.stats else None
        if self.history:
            st = H.hero_routed_layer_hist(self.dims, j, self.T, self.hbar, self.prev1, self.prev2, self.h_out,
                                          self.hist_s, self.ffn_s[layer], self.router_s, self.adapter_s[layer],
                                          self.eta[:j], self.routing_s, stats, self.ws, self.ws_bytes,
                                          self.stream())
            self.n_entries = j
        else:
            st = H.hero_routed_layer(self.dims, j, self.T, self.hbar, self.prev1, self.prev2, self.h_out,
                                     self.state_s, self.ffn_s[layer], self.router_s, self.adapter_s[layer],
                                     self.eta[j - 1], self.routing_s, stats, self.ws, self.ws_bytes,
                                     self.stream())
        if check:
            H.check(st, "hero_routed_layer_hist" if self.history else "hero_routed_layer")
        return st

    def run_stack(self, check: bool = True) -> int:
        stats = [s.struct for s in self.stats] if self.stats else None
        if self.history:
            st = H.hero_routed_stack_hist(self.dims, self.T, self.hbar, self.h_out, self.hist_s, self.ffn_s,
                                          self.router_s, self.adapter_s, self.eta, self.routing_s, stats,
                                          self.ws, self.ws_bytes, self.stream())
            self.n_entries = self.w.L_R
        else:
            st = H.hero_routed_stack(self.dims, self.T, self.hbar, self.h_out, self.state_s, self.ffn_s,
                                     self.router_s, self.adapter_s, self.eta, self.routing_s, stats,
                                     self.ws, self.ws_bytes, self.stream())
        if check:
            H.check(st, "hero_routed_stack_hist" if self.history else "hero_routed_stack")
        return st

    def history_state(self, n: int, kv=None):
        """Matrix-form S, zeta after n layers from (a row subset of) the history, on the device."""
        kv = self.kv if kv is None else kv
        T = kv.shape[0]
        S = torch.empty((T, self.w.d_m, self.w.d_m), dtype=torch.float32, device=self.device)
        zeta = torch.empty((T, self.w.d_m), dtype=torch.float32, device=self.device)
        H.check(H.hero_history_state(self.dims, n, T, kv, self.eta[:n], S, zeta, self.stream()),
                "hero_history_state")
        return S, zeta

    def results(self) -> Dict[str, object]:
        torch.cuda.synchronize()
        S, zeta = self.history_state(self.n_entries) if self.history else (self.S, self.zeta)
        out = dict(h=download_f64(self.h_out), S=S.float().cpu().numpy().astype(np.float64),
                   zeta=zeta.cpu().numpy().astype(np.float64),
                   p_hist=self.p_hist.cpu().numpy().astype(np.float64),
                   m_hist=self.m_hist.cpu().numpy().astype(np.float64))
        if self.stats:
            out["layers"] = [s.host() for s in self.stats]
        return out

    def run_chained(self, rows=None) -> List[Dict[str, object]]:
        """Run the routed stack as chained hero_routed_layer calls and capture, for the
        selected token rows, every layer's post-attention input, the router state before and
        after it, its stats and its output (host float64).  The final output is left in
        h_out and the final state in the state buffers, as hero_routed_stack leaves them."""
        T = self.T
        idx = None if rows is None else torch.as_tensor(np.asarray(rows), device=self.device)
        pick = (lambda x: x) if idx is None else (lambda x: x.index_select(0, idx))
        ws_bytes = H.hero_workspace_size(self.dims, T, False)
        ws = torch.empty(ws_bytes, dtype=torch.uint8, device=self.device)
        stats = LayerStats(T, self.device)
        hs = [self.hbar]
        n_sel = T if idx is None else len(idx)
        prev_state = (np.zeros((n_sel, self.w.d_m, self.w.d_m)), np.zeros((n_sel, self.w.d_m)),
                      np.ones(n_sel), np.ones(n_sel))
        io = []
        for j in range(1, self.w.L_R + 1):
            out = self.h_out if j == self.w.L_R else torch.empty_like(self.hbar)
            args = (hs[-1], hs[-2] if j >= 2 else None, hs[-3] if j >= 3 else None, out)
            if self.history:
                H.check(H.hero_routed_layer_hist(self.dims, j, T, *args, self.hist_s, self.ffn_s[j - 1],
                                                 self.router_s, self.adapter_s[j - 1], self.eta[:j],
                                                 self.routing_s, stats.struct, ws, ws_bytes, self.stream()),
                        "hero_routed_layer_hist")
                self.n_entries = j
                S_sel, z_sel = self.history_state(j, kv=pick(self.kv).contiguous())
            else:
                H.check(H.hero_routed_layer(self.dims, j, T, *args, self.state_s, self.ffn_s[j - 1],
                                            self.router_s, self.adapter_s[j - 1], self.eta[j - 1],
                                            self.routing_s, stats.struct, ws, ws_bytes, self.stream()),
                        "hero_routed_layer")
                S_sel, z_sel = pick(self.S), pick(self.zeta)
            torch.cuda.synchronize()
            after = (S_sel.float().cpu().numpy().astype(np.float64), z_sel.cpu().numpy().astype(np.float64),
                     pick(self.p_hist).cpu().numpy().astype(np.float64),
                     pick(self.m_hist).cpu().numpy().astype(np.float64))
            io.append(dict(hbar=download_f64(pick(hs[-1])), S=prev_state[0], zeta=prev_state[1],
                           p=prev_state[2], m=prev_state[3], stats=stats.host(), h=download_f64(pick(out)),
                           S1=after[0], zeta1=after[1], p1=after[2], m1=after[3]))
            prev_state = after
            hs.append(out)
            if len(hs) > 3:
                hs.pop(0)
        return io


class DeviceDecoder:
    """A full-decoder problem (synth workload with n_layers > 0) on the GPU: attention and FFN
    weights of every block, adapters of the routed ones, the router state and the ABI structs."""

    def __init__(self, prob: synth.Problem, device: str = "cuda:0", stats: bool = True):
        w = prob.w
        assert w.n_layers > 0 and w.dtype == "bf16"
        self.w = w
        self.device = device
        self.T = T = prob.hbar.shape[0]
        self.dims = dims_struct(w)
        self.adims = H.hero_attn_dims(w.n_heads, w.n_kv_heads, w.head_dim)
        self.h_in = upload(prob.hbar, device)
        self.h_out = torch.empty_like(self.h_in)
        self.router = {k: upload(v if k != "th1" else pad_th1(v, w), device) for k, v in prob.router.items()}
        self.router_s = H.hero_router_weights(**{k: self.router[k].data_ptr() for k in H.ROUTER_FIELDS})
        self.attn, self.attn_s, self.ffn, self.ffn_s = [], [], [], []
        for l in range(w.n_layers):
            a = {k: upload(v, device) for k, v in prob.attn[l].items()}
            self.attn.append(a)
            self.attn_s.append(H.hero_attn_weights(a["norm_w"].data_ptr(), a["w_qkv"].data_ptr(),
                                                   a["w_o"].data_ptr()))
            f = {k: upload(v, device) for k, v in prob.ffn[l].items()}
            self.ffn.append(f)
            self.ffn_s.append(H.hero_ffn_weights(f["norm_w"].data_ptr(), f["w_gate"].data_ptr(),
                                                 f["w_up"].data_ptr(), f["w_down"].data_ptr()))
        self.adapter = [{k: upload(v, device) for k, v in prob.adapter[j].items()} for j in range(w.L_R)]
        self.adapter_s = [H.hero_adapter_weights(a["w1"].data_ptr(), a["w2"].data_ptr()) for a in self.adapter]
        self.eta = [float(e) for e in prob.eta]
        self.inv_freq = [float(x) for x in prob.inv_freq]
        self.S = torch.zeros((T, w.d_m, w.d_m), dtype=torch.bfloat16 if w.state_dtype == "bf16" else torch.float32,
                             device=device)
        self.zeta = torch.zeros((T, w.d_m), dtype=torch.float32, device=device)
        self.p_hist = torch.ones(T, dtype=torch.float32, device=device)
        self.m_hist = torch.ones(T, dtype=torch.float32, device=device)
        self.state_s = H.hero_state(self.S.data_ptr(), self.zeta.data_ptr(), self.p_hist.data_ptr(),
                                    self.m_hist.data_ptr())
        self.beta = torch.from_numpy(prob.beta).to(device) if prob.beta is not None else None
        mode = H.HERO_MODE_BUDGET if w.mode == "budget" else H.HERO_MODE_THRESHOLD
        self.routing_s = H.hero_routing(mode, w.tau, w.budget,
                                        self.beta.data_ptr() if self.beta is not None else None, w.ablation)
        self.stats = [LayerStats(T, device) for _ in range(w.L_R)] if stats else None
        self.ws_bytes = H.hero_decoder_workspace_size(self.dims, self.adims, w.n_layers, w.batch, w.seq)
        self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device=device)

    def stream(self):
        return torch.cuda.current_stream(torch.device(self.device)).cuda_stream

    def run(self, check: bool = True) -> int:
        w = self.w
        st = H.hero_decoder_stack(self.dims, self.adims, w.n_layers, w.batch, w.seq, self.h_in, self.h_out,
                                  self.state_s, self.attn_s, self.ffn_s, self.router_s, self.adapter_s, self.eta,
                                  self.inv_freq, self.routing_s, [s.struct for s in self.stats] if self.stats else None,
                                  self.ws, self.ws_bytes, self.stream())
        if check:
            H.check(st, "hero_decoder_stack")
        return st

    def attention(self, layer: int, h=None, hbar=None) -> torch.Tensor:
        """One attention sub-block on h (default: the decoder input); returns hbar."""
        w = self.w
        h = self.h_in if h is None else h
        hbar = torch.empty_like(h) if hbar is None else hbar
        H.check(H.hero_attention_block(self.dims, self.adims, w.batch, w.seq, h, hbar, self.attn_s[layer],
                                       self.inv_freq, self.ws, self.ws_bytes, self.stream()),
                "hero_attention_block")
        return hbar

    def results(self) -> Dict[str, object]:
        torch.cuda.synchronize()
        out = dict(h=download_f64(self.h_out), S=self.S.float().cpu().numpy().astype(np.float64),
                   zeta=self.zeta.cpu().numpy().astype(np.float64),
                   p_hist=self.p_hist.cpu().numpy().astype(np.float64),
                   m_hist=self.m_hist.cpu().numpy().astype(np.float64))
        if self.stats:
            out["layers"] = [s.host() for s in self.stats]
        return out


class DeviceBackward:
    """The backward of one routed block on the GPU: the layer's input hbar, its frozen FFN (with
    the transposed copies the backward reads) and adapter, an upstream gradient, the gates and
    the branch lists, and the gradient buffers the ABI call fills."""

    def __init__(self, w: synth.Workload, hbar: synth.Tensor, ffn: Dict[str, synth.Tensor],
                 adapter: Dict[str, synth.Tensor], dh: synth.Tensor, gate: np.ndarray, use_ffn: np.ndarray,
                 dgate_in: Optional[np.ndarray] = None, device: str = "cuda:0", stream=None,
                 budget: Optional[float] = None):
        self.w = w
        self.T = T = hbar.shape[0]
        self.dims = dims_struct(w)
        self.hbar = upload(hbar, device)
        self.dh = upload(dh, device)
        self.ffn = {k: upload(v, device) for k, v in ffn.items()}
        self.ffn_s = H.hero_ffn_weights(self.ffn["norm_w"].data_ptr(), self.ffn["w_gate"].data_ptr(),
                                        self.ffn["w_up"].data_ptr(), self.ffn["w_down"].data_ptr())
        self.adapter = {k: upload(v, device) for k, v in adapter.items()}
        self.adapter_s = H.hero_adapter_weights(self.adapter["w1"].data_ptr(), self.adapter["w2"].data_ptr())
        wdt = self.ffn["w_down"].dtype
        self.w_down_t = torch.empty((w.d_ff, w.d), dtype=wdt, device=device)
        self.w_gate_up_t = torch.empty((w.d, 2 * w.d_ff), dtype=wdt, device=device)
        self.ffn_t = H.hero_ffn_backward_weights(self.w_down_t.data_ptr(), self.w_gate_up_t.data_ptr())
        self.device = device
        self._stream = stream
        H.check(H.hero_ffn_backward_weights_make(self.dims, self.ffn_s, self.w_down_t, self.w_gate_up_t,
                                                 self.stream()), "hero_ffn_backward_weights_make")
        self.gate = torch.from_numpy(np.ascontiguousarray(gate, dtype=np.float32)).to(device)
        use_ffn = np.asarray(use_ffn, dtype=bool)
        # the branch lists as the forward's stats hold them: ascending token indices
        idx_f = np.nonzero(use_ffn)[0].astype(np.int32)
        idx_a = np.nonzero(~use_ffn)[0].astype(np.int32)
        self.idx_ffn = torch.zeros(T, dtype=torch.int32, device=device)
        self.idx_ad = torch.zeros(T, dtype=torch.int32, device=device)
        self.idx_ffn[:len(idx_f)] = torch.from_numpy(idx_f).to(device)
        self.idx_ad[:len(idx_a)] = torch.from_numpy(idx_a).to(device)
        self.counts = torch.tensor([len(idx_f), len(idx_a), 0, 0], dtype=torch.int32, device=device)
        self.dgate_in = None if dgate_in is None else \
            torch.from_numpy(np.ascontiguousarray(dgate_in, dtype=np.float32)).to(device)
        # the forward's rule: in budget mode the branch sizes are known on the host
        self.routing_s = None if budget is None else H.hero_routing(H.HERO_MODE_BUDGET, 0.5, budget, None)
        self.dhbar = torch.empty_like(self.hbar)
        self.dgate = torch.empty(T, dtype=torch.float32, device=device)
        self.dlogit = torch.empty(T, dtype=torch.float32, device=device)
        self.dw1 = torch.empty((w.d_r, w.d), dtype=torch.float32, device=device)
        self.dw2 = torch.empty((w.d, w.d_r), dtype=torch.float32, device=device)
        self.grads_s = H.hero_block_grads(self.dhbar.data_ptr(), self.dgate.data_ptr(), self.dlogit.data_ptr(),
                                          self.dw1.data_ptr(), self.dw2.data_ptr())
        self.ws_bytes = H.hero_backward_workspace_size(self.dims, T)
        self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device=device)

    def stream(self):
        """The given stream, else torch's current one (so that graph capture sees the launches)."""
        if self._stream is not None:
            return self._stream
        return torch.cuda.current_stream(torch.device(self.device)).cuda_stream

    def run(self) -> None:
        H.check(H.hero_routed_block_backward(self.dims, self.T, self.hbar, self.dh, self.gate, self.idx_ffn,
                                             self.idx_ad, self.counts, self.routing_s, self.dgate_in, self.ffn_s,
                                             self.ffn_t, self.adapter_s, self.grads_s, self.ws, self.ws_bytes,
                                             self.stream()),
                "hero_routed_block_backward")

    def results(self) -> Dict[str, np.ndarray]:
        torch.cuda.synchronize()
        return dict(dhbar=download_f64(self.dhbar), dgate=self.dgate.cpu().numpy().astype(np.float64),
                    dlogit=self.dlogit.cpu().numpy().astype(np.float64),
                    dw1=self.dw1.cpu().numpy().astype(np.float64), dw2=self.dw2.cpu().numpy().astype(np.float64))


class DeviceRouterBackward:
    """The router's backward at routed layer j on the GPU, on a DeviceProblem's inputs (its hbar,
    hbar_{j-1}, hbar_{j-2}, router weights and the state entering the layer), given dL/dlogit and
    the carried state gradient; the fp32 gradient buffers start at zero.  With c_from_forward (j >= 2)
    the layer's forward runs once first, on a copy of the entering state, with hero_state.c_read set,
    and the backward is handed that memory read in place of reading S_{j-1} for it again."""

    def __init__(self, dp: "DeviceProblem", j: int, dlogit: np.ndarray, dS: np.ndarray, dzeta: np.ndarray,
                 dp_hist: np.ndarray, dm_hist: np.ndarray, c_from_forward: bool = False):
        w, dev, T = dp.w, dp.device, dp.T
        self.dp_, self.j, self.T, self.w = dp, j, T, w
        self.c_read = None
        self.state_s = dp.state_s
        if c_from_forward and j >= 2:
            self.c_read = torch.full((T, w.d_m), float("nan"), dtype=torch.float32, device=dev)
            S, z, p, m = (x.clone() for x in (dp.S, dp.zeta, dp.p_hist, dp.m_hist))
            st = H.hero_state(S.data_ptr(), z.data_ptr(), p.data_ptr(), m.data_ptr(), self.c_read.data_ptr())
            out = torch.empty_like(dp.h_out)
            H.check(H.hero_routed_layer(dp.dims, j, T, dp.hbar, dp.prev1, dp.prev2, out, st, dp.ffn_s[0],
                                        dp.router_s, dp.adapter_s[0], dp.eta[j - 1], dp.routing_s, None, dp.ws,
                                        dp.ws_bytes, dp.stream()), "hero_routed_layer")
            torch.cuda.synchronize()
            del S, z, p, m, out
            self.state_s = H.hero_state(dp.S.data_ptr(), dp.zeta.data_ptr(), dp.p_hist.data_ptr(),
                                        dp.m_hist.data_ptr(), self.c_read.data_ptr())
        f32 = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev)
        zeros = lambda *shape: torch.zeros(*shape, dtype=torch.float32, device=dev)
        self.dlogit = f32(dlogit)
        self.dS, self.dzeta, self.dpc, self.dmc = f32(dS), f32(dzeta), f32(dp_hist), f32(dm_hist)
        self.carry_s = H.hero_router_carry(self.dS.data_ptr(), self.dzeta.data_ptr(), self.dpc.data_ptr(),
                                           self.dmc.data_ptr())
        self.dh = [zeros(T, w.d) for _ in range(3)]
        self.grads = {k: zeros(*dp.router[k].shape) for k in H.ROUTER_FIELDS}
        self.grads_s = H.hero_router_grads(**{k: v.data_ptr() for k, v in self.grads.items()})
        self.deta = zeros(4)
        self.ws_bytes = H.hero_router_backward_workspace_size(dp.dims, T)
        self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device=dev)

    def run(self) -> None:
        dp, j = self.dp_, self.j
        H.check(H.hero_router_backward(dp.dims, j, self.T, dp.hbar, dp.prev1 if j >= 2 else None,
                                       dp.prev2 if j >= 3 else None, self.state_s, dp.router_s, dp.eta[j - 1],
                                       self.dlogit, self.carry_s, self.dh[0], self.dh[1] if j >= 2 else None,
                                       self.dh[2] if j >= 3 else None, self.grads_s, self.deta, self.ws,
                                       self.ws_bytes, dp.stream()), "hero_router_backward")

    def results(self) -> Dict[str, np.ndarray]:
        torch.cuda.synchronize()
        f64 = lambda t: t.cpu().numpy().astype(np.float64)
        g = {k: f64(v) for k, v in self.grads.items()}
        g["th1"] = g["th1"][:, :self.w.d_s + self.w.d_m + 1]
        return dict(dhbar=f64(self.dh[0]), dhbar1=f64(self.dh[1]), dhbar2=f64(self.dh[2]), grads=g,
                    deta=float(self.deta[0].item()), dS=f64(self.dS), dzeta=f64(self.dzeta), dp=f64(self.dpc),
                    dm=f64(self.dmc))
