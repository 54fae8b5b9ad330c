#!/usr/bin/env python3
"""Throughput of the HeRo routed FFN hot path on one MI355X.

A step is one hero_routed_layer call (router pre-pass, fused router tail with
the memory read-modify-write, branch decision and compaction, gathered SwiGLU
FFN, adapter, scatter) over the whole token batch of the workload, with every
input already resident in HBM.  Default workload: Llama-3.1-8B shape, one
routed layer (j = 17 of 32, synthesized incoming router state), bf16, 4096
prefill tokens, skip budget 26.87 %.

Prints one JSON line.  The dominant kernel (the FFN gate/up GEMM) is timed live
inside the timed region with HIP events recorded around its launches; a second,
untimed pass instruments every kernel for the per-kernel table.  The CPU
baseline times the float64 oracle on a bounded token sample of the same inputs.
"""
import argparse
import ctypes
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_F32_TFLOPS = 157.3     # MI355X fp32 vector / MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E


class HipEvents:
    """hipEvent_t handles through the HIP runtime already loaded by torch."""

    def __init__(self):
        self.hip = ctypes.CDLL("libamdhip64.so.7")
        self.hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.hip.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        self.hip.hipEventSynchronize.argtypes = [ctypes.c_void_p]

    def create(self, n):
        out = []
        for _ in range(n):
            e = ctypes.c_void_p()
            assert self.hip.hipEventCreate(ctypes.byref(e)) == 0
            out.append(e.value)
        return out

    def record(self, ev, stream):
        assert self.hip.hipEventRecord(ev, stream) == 0

    def elapsed_ms(self, a, b):
        f = ctypes.c_float()
        assert self.hip.hipEventSynchronize(b) == 0
        assert self.hip.hipEventElapsedTime(ctypes.byref(f), a, b) == 0
        return f.value

    def destroy(self, evs):
        for e in evs:
            self.hip.hipEventDestroy(e)


def kernel_work(w, n_f, n_a, T, j, memory="matrix"):
    """Algorithmic FLOPs and HBM bytes per launch of each kernel (bf16 I/O, fp32 or bf16 S).
    The memory pass moves S and zeta (read unless j = 1, written) in matrix form, or reads the
    j-1 stored (phi(k), v) pairs and writes one in depth-history form."""
    es = 2 if w.dtype == "bf16" else 4
    ss = 2 if w.state_dtype == "bf16" else 4
    d, dff, r, dm = w.d, w.d_ff, w.d_r, w.d_m
    npre = w.d_e + w.d_head
    hid_reads = 1 + (j >= 2) + (j >= 3)
    if memory == "history":
        state_rw = 4 * 2 * dm * ((j - 1) + 1)
    else:
        state_rw = (2 if j > 1 else 1) * (ss * dm * dm + 4 * dm)
    return {
        "rowstats": dict(flops=0, bytes=T * (hid_reads * d * es + d * es + 16)),
        "router_gemm": dict(flops=2 * d * npre * T, bytes=T * (d * es + 4 * npre)),
        "router_pre": dict(flops=0, bytes=T * (4 * npre + 16 + 8 + 4 * (4 * dm + w.d_head + 1))),
        "router_mem": dict(flops=0, bytes=T * (state_rw + 4 * 3 * dm + 4 * dm)),
        "router_post": dict(flops=0, bytes=T * (4 * (dm + dm + w.d_head + 1) + 8 * 2 + 8)),
        "select": dict(flops=0, bytes=T * (4 + 1 + 4)),
        "ffn_gate_up": dict(flops=4 * d * dff * n_f, bytes=n_f * (d * es + dff * es) + 2 * d * dff * es),
        "ffn_down": dict(flops=2 * d * dff * n_f, bytes=n_f * (dff * es + 2 * d * es) + d * dff * es),
        "adapter_down": dict(flops=2 * d * r * n_a, bytes=n_a * d * es + r * d * es),
        "adapter_up": dict(flops=2 * d * r * n_a, bytes=n_a * 2 * d * es + r * d * es),
    }


def describe(w, j):
    where = f"routed layer j={j} of {w.L_R}" if j > 0 else f"routed stack of {w.L_R} layers"
    return (f"{w.name}: d={w.d}, d_ff={w.d_ff}, adapter rank {w.d_r}, memory dim {w.d_m}, "
            f"T={w.T} tokens ({w.batch}x{w.seq}), {where}, "
            + (f"skip budget {w.budget}" if w.mode == "budget" else f"threshold tau={w.tau}"))


def cpu_baseline(prob, gpu_stats, j, target_s=12.0, max_tokens=None):
    """Time the float64 oracle on a growing token sample until it runs >= target_s."""
    import numpy as np
    from threadpoolctl import threadpool_info
    from oracle import hero_oracle as O
    from tests.oracle_inputs import adapter_of, dims_of, ffn_of, router_of

    w = prob.w
    T = prob.hbar.shape[0]
    max_tokens = T if max_tokens is None else min(T, max_tokens)
    dims, R = dims_of(w), router_of(prob)
    F, A = ffn_of(prob.ffn[0]), adapter_of(prob.adapter[0])
    hb = prob.hbar.f64
    hp1 = prob.hbar_prev1.f64 if prob.hbar_prev1 is not None else None
    hp2 = prob.hbar_prev2.f64 if prob.hbar_prev2 is not None else None
    lam = gpu_stats["lam"] if w.mode == "budget" else None

    def run(rows):
        st = O.State(prob.S[rows].astype("f8"), prob.zeta[rows].astype("f8"),
                     prob.p_hist[rows].astype("f8"), prob.m_hist[rows].astype("f8"))
        beta = None if prob.beta is None else prob.beta[rows].astype("f8")
        t0 = time.perf_counter()
        O.routed_layer(j, dims, hb[rows], None if hp1 is None else hp1[rows],
                       None if hp2 is None else hp2[rows], st, F, R, A, float(prob.eta[j - 1]),
                       mode=w.mode, budget=w.budget, tau=w.tau, beta=beta,
                       forced_ffn=gpu_stats["mask"][rows], lam_given=lam)
        return time.perf_counter() - t0

    n = 64
    while True:
        rows = np.linspace(0, T - 1, n).astype(np.int64)
        dt = run(rows)
        if dt >= target_s or n >= max_tokens:
            break
        n = min(max_tokens, max(2 * n, int(n * target_s / max(dt, 1e-3) * 1.1)))
    # the whole call took less than the target: repeat it (up to 8 runs in all) for a steadier rate
    reps = 1
    while dt < target_s and reps < 8:
        dt += run(rows)
        reps += 1
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    cpu_model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            cpu_model = next((l.split(":", 1)[1].strip() for l in f if l.startswith("model name")), cpu_model)
    except OSError:
        pass
    return {"value": n * reps / dt, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "nproc": os.cpu_count(), "omp_num_threads": os.environ.get("OMP_NUM_THREADS"), "cpu_model": cpu_model,
            "sample": f"{n} of {T} tokens of the same layer call (router, memory, branch; float64 numpy, "
                      f"branch decisions teacher-forced to the GPU's)" +
                      (f", run {reps} times" if reps > 1 else "") + f", {dt:.1f} s"}


# committed rocprofv3 FETCH_SIZE / WRITE_SIZE summaries, per workload
# a call of at most this many tokens is a decode step: timed as HIP-graph replays by default
DECODE_TOKENS = 256
COUNTERS_MD = {
    "llama31_8b_layer": os.path.join(ROOT, "profiles", "routed_layer_llama31_8b_hbm_counters.md"),
    "llama31_8b_stack": os.path.join(ROOT, "profiles", "routed_stack_llama31_8b_hbm_counters.md"),
}
GEMM_SOURCES = ("paper_2609_08189_amd/csrc/k_gemm.hip", "paper_2609_08189_amd/csrc/hero_device.h")


def gemm_source_hash():
    import hashlib
    h = hashlib.sha256()
    for f in GEMM_SOURCES:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def counted_traffic(kernel, workload):
    """HBM bytes per launch of `kernel` from the workload's committed rocprofv3 FETCH_SIZE /
    WRITE_SIZE summary (scaled by the copy calibration there), or None when there is none or the
    GEMM sources changed since it was taken."""
    try:
        text = open(COUNTERS_MD[workload]).read()
    except (KeyError, OSError):
        return None
    if f"`{gemm_source_hash()}`" not in text:
        return None
    for line in text.splitlines():
        cells = [c.strip() for c in line.strip().strip("|").split("|")]
        if len(cells) == 5 and cells[0] == kernel:
            return int(round((float(cells[3]) + float(cells[4])) * 1e6))
    return None


def _short(name):
    return name.replace("hero::(anonymous namespace)::", "").replace("void ", "")[:150].replace("|", "/")


def summarize_rocprof(root, window=None):
    """Markdown summary of rocprofv3 CSV files (kernel stats and/or counter collection) under root.

    Counter tables give the mean per dispatch of each kernel; for the plain device
    copy (the runtime's copyBuffer kernel) the largest dispatch is shown, which is
    the calibration copy of known size.  With window = (skip, count), the kernel trace
    also gives each kernel's mean duration over its dispatches skip .. skip+count-1 (in
    dispatch order): for a bench run with W warmup steps, (1 + W, K) selects exactly the
    K timed steps (one checked call precedes the warmup).
    """
    import csv
    import glob
    stats = sorted(glob.glob(os.path.join(root, "**", "*kernel_stats.csv"), recursive=True))
    for path in stats:
        print(f"### kernel stats ({os.path.relpath(path, root)})\n")
        print("| kernel | calls | total ms | avg us | min us | max us | % |")
        print("|---|---|---|---|---|---|---|")
        with open(path) as f:
            for r in csv.DictReader(f):
                print(f"| {_short(r['Name'])} | {r['Calls']} | {float(r['TotalDurationNs']) / 1e6:.3f} | "
                      f"{float(r['AverageNs']) / 1e3:.2f} | {float(r['MinNs']) / 1e3:.2f} | "
                      f"{float(r['MaxNs']) / 1e3:.2f} | {float(r['Percentage']):.2f} |")
        print()
    traces = sorted(glob.glob(os.path.join(root, "**", "*kernel_trace.csv"), recursive=True))
    if window is not None:
        skip, count = window
        for path in traces:
            per = {}
            with open(path) as f:
                for r in csv.DictReader(f):
                    per.setdefault(r["Kernel_Name"], []).append(
                        (int(r["Dispatch_Id"]), (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3))
            print(f"### dispatches {skip}..{skip + count - 1} of each kernel ({os.path.relpath(path, root)})\n")
            print("| kernel | dispatches | mean us | min us | max us |")
            print("|---|---|---|---|---|")
            for name, v in sorted(per.items(), key=lambda kv: -sum(d for _, d in kv[1])):
                sel = [d for _, d in sorted(v)][skip:skip + count]
                if sel:
                    print(f"| {_short(name)} | {len(sel)} | {sum(sel) / len(sel):.2f} | {min(sel):.2f} | "
                          f"{max(sel):.2f} |")
            print()
    counters = sorted(glob.glob(os.path.join(root, "**", "*counter_collection.csv"), recursive=True))
    for path in counters:
        agg, seq = {}, {}
        with open(path) as f:
            for n, r in enumerate(csv.DictReader(f)):
                key = (r["Kernel_Name"], r["Counter_Name"])
                agg.setdefault(key, []).append(float(r["Counter_Value"]))
                seq.setdefault(key, []).append((int(r.get("Dispatch_Id", n)), float(r["Counter_Value"])))
        print(f"### counters ({os.path.relpath(path, root)}), KiB per dispatch as reported\n")
        print("| kernel | counter | dispatches | mean | max |")
        print("|---|---|---|---|---|")
        for (k, c), v in sorted(agg.items()):
            print(f"| {_short(k)} | {c} | {len(v)} | {sum(v) / len(v):.1f} | {max(v):.1f} |")
        print()
        if window is not None:
            skip, count = window
            print(f"### counters over dispatches {skip}..{skip + count - 1} of each kernel "
                  f"({os.path.relpath(path, root)})\n")
            print("| kernel | counter | dispatches | mean | max |")
            print("|---|---|---|---|---|")
            for (k, c), v in sorted(seq.items()):
                sel = [x for _, x in sorted(v)][skip:skip + count]
                if sel:
                    print(f"| {_short(k)} | {c} | {len(sel)} | {sum(sel) / len(sel):.1f} | {max(sel):.1f} |")
            print()


_GRAPHS = []


def graphed(step):
    """The step captured once as a HIP graph (torch.cuda.graph around the library's launches, which
    go to torch's current stream); replays launch the whole call at once."""
    import torch
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()
    _GRAPHS.append(g)
    return g.replay


def step_stats(step_ms):
    """Median and 10th/90th percentiles of the per-step times inside the timed region."""
    n = len(step_ms)
    pick = lambda f: round(step_ms[min(n - 1, int(f * (n - 1) + 0.5))], 4)
    return {"median": pick(0.5), "p10": pick(0.1), "p90": pick(0.9), "n": n}


def ideal_fraction(works, ms_step, dtype, stack):
    """Ideal time of one step (every kernel at its own roof: max(FLOP / MFMA peak, bytes / HBM
    peak), summed) over the measured step time."""
    peak_f = (PEAK_BF16_TFLOPS if dtype == "bf16" else PEAK_F32_TFLOPS) * 1e12
    ideal = sum(max(k["flops"] / peak_f, k["bytes"] / (PEAK_HBM_GBS * 1e9)) for wk in works for k in wk.values())
    return {"ideal_ms": round(ideal * 1e3, 4), "measured_ms": round(ms_step, 4),
            "frac": round(ideal * 1e3 / ms_step, 4),
            "note": "sum over kernels of max(algorithmic FLOP / 2.5 PFLOP/s, algorithmic bytes / 8 TB/s)"}


def decoder_work(w, nfs, nas):
    """Algorithmic FLOPs / HBM bytes per step of each kernel of a full-decoder call."""
    T, d, dff, hd, B, S = w.T, w.d, w.d_ff, w.head_dim, w.batch, w.seq
    nh, nkv, r = w.n_heads, w.n_kv_heads, w.d_r
    n_dense = w.n_layers - w.L_R
    rows_ffn = n_dense * T + sum(nfs)
    rows_ad = sum(nas)
    pairs = B * nh * S * (S + 1) // 2                 # (query, visible key) pairs
    wk = {
        "attn_norm": dict(flops=0, bytes=w.n_layers * T * 4 * d),
        "attn_qkv": dict(flops=w.n_layers * 2 * T * d * (nh + 2 * nkv) * hd,
                         bytes=w.n_layers * 2 * ((nh + 2 * nkv) * hd * (d + T) + T * d)),
        "attn_core": dict(flops=w.n_layers * 4 * hd * pairs,
                          bytes=w.n_layers * 2 * B * S * hd * (2 * nh + 2 * nkv)),
        "attn_out": dict(flops=w.n_layers * 2 * T * nh * hd * d,
                         bytes=w.n_layers * 2 * (d * nh * hd + T * nh * hd + 2 * T * d)),
        "ffn_gate_up": dict(flops=4 * d * dff * rows_ffn,
                            bytes=sum(2 * (2 * d * dff + n * (d + dff)) for n in [T] * n_dense + nfs if n)),
        "ffn_down": dict(flops=2 * d * dff * rows_ffn,
                         bytes=sum(2 * (d * dff + n * (dff + 2 * d)) for n in [T] * n_dense + nfs if n)),
        "adapter_down": dict(flops=2 * d * r * rows_ad, bytes=2 * (rows_ad * d + sum(1 for n in nas if n) * r * d)),
        "adapter_up": dict(flops=2 * d * r * rows_ad, bytes=2 * (2 * rows_ad * d + sum(1 for n in nas if n) * r * d)),
    }
    return wk


def bench_decoder(args, w):
    """A step is one hero_decoder_stack call: every block's attention, the pretrained FFN of the
    first n_layers - L_R blocks and the routed layers of the rest, over all T tokens."""
    import torch
    from paper_2609_08189_amd import hero as H
    from paper_2609_08189_amd import synth
    from paper_2609_08189_amd.device import DeviceDecoder

    print(f"# preparing {w.name}: {w.n_layers} blocks, last {w.L_R} routed", file=sys.stderr, flush=True)
    prob = synth.make_problem(w, seed=args.seed)
    dd = DeviceDecoder(prob, device="cuda:0", stats=True)
    stream = dd.stream()
    ev = HipEvents()
    dd.run()
    torch.cuda.synchronize()
    layer_stats = [s.host() for s in dd.stats]
    nfs = [ls["n_ffn"] for ls in layer_stats]
    nas = [ls["n_ad"] for ls in layer_stats]
    dd.stats = None
    for _ in range(args.warmup):
        dd.run()
    torch.cuda.synchronize()
    K = args.steps
    n_dense = w.n_layers - w.L_R
    # launches per step of every kernel
    launches = {k: w.n_layers for k in ("attn_norm", "attn_qkv", "attn_core", "attn_out")}
    launches.update({k: w.L_R for k in ("router_gemm", "router_pre", "router_post", "select")})
    launches["router_mem"] = w.L_R if not (w.ablation & 12) else 0
    launches["rowstats"] = w.n_layers
    launches["ffn_gate_up"] = launches["ffn_down"] = n_dense + sum(1 for n in nfs if n)
    launches["adapter_down"] = launches["adapter_up"] = sum(1 for n in nas if n)
    # instrumented pass: every kernel's time per step, which names the dominant one
    per, handles = {}, {}
    for name, n in launches.items():
        if n:
            handles[name] = (ev.create(K * n), ev.create(K * n))
            H.hero_kernel_timer(H.HERO_K[name], *handles[name])
    for _ in range(K):
        dd.run()
    torch.cuda.synchronize()
    works = decoder_work(w, nfs, nas)
    for name, (a, b) in handles.items():
        H.hero_kernel_timer(H.HERO_K[name], [], [])
        ms = sum(ev.elapsed_ms(x, y) for x, y in zip(a, b)) / K         # per step
        n = launches[name]
        wk = works.get(name)
        per[name] = {"ms_per_step": round(ms, 3), "launches": n, "us": round(1000 * ms / n, 2),
                     "tflops": round(wk["flops"] / (ms * 1e-3) * 1e-12, 1) if wk and wk["flops"] else None,
                     "gbs": round(wk["bytes"] / (ms * 1e-3) * 1e-9, 1) if wk else None}
        ev.destroy(a + b)
    dom = max((k for k in per if k in works and works[k]["flops"]), key=lambda k: per[k]["ms_per_step"])
    # timed region, with the dominant kernel's launches bracketed on the call's stream (graph mode:
    # replays of the captured call; the kernel's time then comes from the instrumented pass)
    run = graphed(dd.run) if args.graph else dd.run
    n_dom = K * launches[dom]
    ks, ke = ev.create(n_dom), ev.create(n_dom)
    if not args.graph:
        H.hero_kernel_timer(H.HERO_K[dom], ks, ke)
    t_start, t_stop = ev.create(2)
    torch.cuda.synchronize()
    marks = ev.create(K - 1)
    ev.record(t_start, stream)
    for i in range(K):
        run()
        if i < K - 1:
            ev.record(marks[i], stream)
    ev.record(t_stop, stream)
    torch.cuda.synchronize()
    H.hero_kernel_timer(H.HERO_K[dom], [], [])
    ms_step = ev.elapsed_ms(t_start, t_stop) / K
    bounds = [t_start] + marks + [t_stop]
    step_ms = sorted(ev.elapsed_ms(a, b) for a, b in zip(bounds[:-1], bounds[1:]))
    dom_ms = per[dom]["ms_per_step"] if args.graph else sum(ev.elapsed_ms(a, b) for a, b in zip(ks, ke)) / K
    achieved = works[dom]["flops"] / (dom_ms * 1e-3) * 1e-12
    result = {
        "metric": "routed-FFN-stack tokens/sec at Llama-3.1-8B shape; % MFMA/HBM roofline",
        "value": round(w.T / (ms_step * 1e-3), 1), "unit": "tokens/s", "n_gpus": 1, "steps": K,
        "warmup": args.warmup, "ms_per_step": round(ms_step, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": w.dtype, "data": "synthetic",
        "config": {"workload": (f"{w.name}: full decoder, {w.n_layers} blocks of d={w.d}, d_ff={w.d_ff}, "
                                f"{w.n_heads}/{w.n_kv_heads} heads of {w.head_dim}, attention at every block, "
                                f"the last {w.L_R} routed (adapter rank {w.d_r}, memory dim {w.d_m}, "
                                f"skip budget {w.budget}), T={w.T} tokens ({w.batch}x{w.seq})"),
                   "global_batch": w.batch, "seq_len": w.seq, "tokens": w.T, "layers_per_step": w.n_layers,
                   "parallelism": "none", "n_ffn_routed": sum(nfs), "n_adapter": sum(nas),
                   "hip_graph": bool(args.graph)},
        "roofline": {"bound": "mfma", "achieved": round(achieved, 1), "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4), "traffic": None,
                     "kernel": dom, "avg_launch_us": round(1000 * dom_ms / launches[dom], 2),
                     "work_per_launch": f"{works[dom]['flops'] / 1e12:.2f} TFLOP per step over "
                                        f"{launches[dom]} launches"},
        "step_ms": step_stats(step_ms),
        "kernels": per,
    }
    print(json.dumps(result), flush=True)


BWD_KERNELS = ("bwd_norm", "bwd_ffn_e", "bwd_ffn_gate_up", "bwd_ffn_du", "bwd_adapter", "bwd_adapter_wgrad",
               "bwd_rows")


def backward_work(w, n_f, n_a):
    """Algorithmic FLOPs / HBM bytes of each kernel group of one routed-block backward call
    (storage dtype es; fp32 intermediates where the kernels keep them)."""
    T, d, dff, r = w.T, w.d, w.d_ff, w.d_r
    es = 2 if w.dtype == "bf16" else 4
    n_parts = dff // 32 if w.dtype == "bf16" else dff
    return {
        "bwd_norm": dict(flops=0, bytes=es * 2 * T * d),
        "bwd_ffn_e": dict(flops=2 * n_f * d * dff, bytes=es * (d * dff + n_f * d + n_f * dff)),
        "bwd_ffn_gate_up": dict(flops=4 * n_f * d * dff,
                                bytes=es * (2 * d * dff + n_f * d + n_f * dff + 2 * n_f * dff) + 4 * n_f * n_parts),
        "bwd_ffn_du": dict(flops=4 * n_f * d * dff, bytes=es * (2 * d * dff + 2 * n_f * dff) + 4 * n_f * d),
        "bwd_adapter": dict(flops=6 * n_a * d * r, bytes=es * (2 * n_a * d + 6 * d * r) + 4 * n_a * d),
        "bwd_adapter_wgrad": dict(flops=4 * n_a * d * r, bytes=es * 2 * n_a * d + 4 * 2 * d * r),
        "bwd_rows": dict(flops=0, bytes=es * (3 * T * d + d) + 4 * T * d),
    }


def cpu_baseline_backward(w, hbar, ffn, ad, dh, gate, use_ffn, target_s=12.0):
    """The oracle's block backward on a token sample of the same inputs (rows in their order)."""
    import numpy as np
    from oracle import hero_oracle as O
    from tests.oracle_inputs import adapter_of, dims_of, ffn_of
    dims, F, A = dims_of(w), ffn_of(ffn), adapter_of(ad)
    hb, dhf = hbar.f64, dh.f64
    g64 = gate.astype(np.float64)

    def run(n):
        t0 = time.perf_counter()
        O.routed_block_backward(hb[:n], g64[:n], use_ffn[:n], F, A, dims, dhf[:n])
        return time.perf_counter() - t0

    # grow the sample until it takes a quarter of the target; then repeat it up to the target
    n, t = 8, run(8)
    while t < target_s / 4 and n < w.T:
        n = min(w.T, 4 * n)
        t = run(n)
    reps, total = 1, t
    while total < target_s and reps < 8:
        total += run(n)
        reps += 1
    return {"value": round(reps * n / total, 2), "unit": "tokens/s",
            "cores": int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1)), "kind": "oracle",
            "sample": f"first {n} of {w.T} tokens ({int(use_ffn[:n].sum())} FFN, {int((~use_ffn[:n]).sum())} "
                      f"adapter), {reps} run(s), float64 numpy, {total:.1f} s; nproc {os.cpu_count()}"}


def bench_backward(args, w):
    """A step is one hero_routed_block_backward call over the workload's T tokens (frozen FFN with
    its transposed copies made once beforehand, adapter, upstream gradient, gates and branch lists
    resident in HBM)."""
    import numpy as np
    import torch
    from paper_2609_08189_amd import hero as H
    from paper_2609_08189_amd import synth
    from paper_2609_08189_amd.device import DeviceBackward

    if w.layer_j <= 0 or w.n_layers > 0:
        sys.exit("--backward times one routed block: use a single-layer workload")
    print(f"# preparing the backward of {describe(w, w.layer_j)}", file=sys.stderr, flush=True)
    hbar = synth.hidden(w, args.seed)
    ffn = synth.ffn_layer(w, w.layer_j - 1, args.seed)
    ad = synth.adapter_layer(w, w.layer_j - 1, args.seed)
    # the budget rule's branch sizes (floor(budget T + 1/2) adapter tokens) at random positions
    n_skip = int(math.floor(w.budget * w.T + 0.5)) if w.mode == "budget" else None
    dh, gate, use_ffn = synth.backward_inputs(w, args.seed, n_adapter=n_skip)
    n_f, n_a = int(use_ffn.sum()), int((~use_ffn).sum())
    db = DeviceBackward(w, hbar, ffn, ad, dh, gate, use_ffn, budget=w.budget if n_skip is not None else None)
    stream = db.stream()
    ev = HipEvents()
    db.run()
    for _ in range(args.warmup):
        db.run()
    torch.cuda.synchronize()
    K = args.steps
    works = backward_work(w, n_f, n_a)
    # instrumented pass: every kernel group's time per step
    per, handles = {}, {}
    for name in BWD_KERNELS:
        handles[name] = (ev.create(K), ev.create(K))
        H.hero_kernel_timer(H.HERO_K[name], *handles[name])
    for _ in range(K):
        db.run()
    torch.cuda.synchronize()
    for name, (a, b) in handles.items():
        H.hero_kernel_timer(H.HERO_K[name], [], [])
        us = 1000.0 * sum(ev.elapsed_ms(x, y) for x, y in zip(a, b)) / K
        wk = works[name]
        per[name] = {"us": round(us, 2), "tflops": round(wk["flops"] / us * 1e-6, 1) if wk["flops"] else None,
                     "gbs": round(wk["bytes"] / us * 1e-3, 1)}
        ev.destroy(a + b)
    dom = max((k for k in per if works[k]["flops"]), key=lambda k: per[k]["us"])
    run = graphed(db.run) if args.graph else db.run
    ks, ke = ev.create(K), ev.create(K)
    if not args.graph:
        H.hero_kernel_timer(H.HERO_K[dom], ks, ke)
    t_start, t_stop = ev.create(2)
    marks = ev.create(K - 1)
    torch.cuda.synchronize()
    ev.record(t_start, stream)
    for i in range(K):
        run()
        if i < K - 1:
            ev.record(marks[i], stream)
    ev.record(t_stop, stream)
    torch.cuda.synchronize()
    H.hero_kernel_timer(H.HERO_K[dom], [], [])
    ms_step = ev.elapsed_ms(t_start, t_stop) / K
    bounds = [t_start] + marks + [t_stop]
    step_ms = sorted(ev.elapsed_ms(a, b) for a, b in zip(bounds[:-1], bounds[1:]))
    dom_ms = per[dom]["us"] / 1000 if args.graph else sum(ev.elapsed_ms(a, b) for a, b in zip(ks, ke)) / K
    peak_f = PEAK_BF16_TFLOPS if w.dtype == "bf16" else PEAK_F32_TFLOPS
    achieved = works[dom]["flops"] / (dom_ms * 1e-3) * 1e-12
    result = {
        "metric": "routed-block backward tokens/sec at Llama-3.1-8B shape; % MFMA roofline",
        "value": round(w.T / (ms_step * 1e-3), 1), "unit": "tokens/s", "n_gpus": 1, "steps": K,
        "warmup": args.warmup, "ms_per_step": round(ms_step, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": w.dtype, "data": "synthetic",
        "config": {"workload": (f"backward of one routed block (eq:ffn_route through the gate scaling) at "
                                f"{describe(w, w.layer_j)}; upstream gradient N(0,1), gates U(0.02,0.98), "
                                f"the budget's adapter count at random positions"),
                   "global_batch": w.batch, "seq_len": w.seq, "tokens": w.T, "parallelism": "none",
                   "n_ffn": n_f, "n_adapter": n_a, "hip_graph": bool(args.graph)},
        "roofline": {"bound": "mfma", "achieved": round(achieved, 1), "peak": peak_f, "unit": "TFLOP/s",
                     "frac": round(achieved / peak_f, 4), "traffic": None, "kernel": dom,
                     "avg_launch_us": round(1000 * dom_ms, 2),
                     "work_per_launch": f"{works[dom]['flops'] // (n_f or 1) // (w.d * w.d_ff)}*d*d_ff FLOP per "
                                        f"FFN token x {n_f} FFN tokens = {works[dom]['flops'] / 1e9:.1f} GFLOP"},
        "step_ms": step_stats(step_ms),
        "whole_call": ideal_fraction([works], ms_step, w.dtype, False),
        "kernels": per,
    }
    if not args.no_cpu_baseline:
        print("# timing the CPU oracle on a token sample", file=sys.stderr, flush=True)
        result["cpu_baseline"] = cpu_baseline_backward(w, hbar, ffn, ad, dh, gate, use_ffn, args.cpu_target_s)
    print(json.dumps(result), flush=True)


RBWD_KERNELS = ("router_bwd_gemm", "router_bwd_token", "router_bwd_products", "router_bwd_rows")


def router_backward_work(w, j, c_given=False):
    """Algorithmic FLOPs and HBM bytes of hero_router_backward's kernel groups for T tokens at
    routed layer j (fp32 state; the token kernels stream S_{j-1} once and dL/dS in and out, and read
    the forward's memory read c when it is handed over)."""
    T, d, dm, es = w.T, w.d, w.d_m, (2 if w.dtype == "bf16" else 4)
    NP = w.d_e + w.d_head
    splits = 4 if w.dtype == "bf16" else 1
    d_x = w.d_s + dm + 1
    vec = d_x + 5 * dm + 3 * w.d_head + 2 + 2 * w.d_p + 8 + w.d_a + w.d_h + w.d_e
    small = 2 * T * (4 * dm * w.d_s + dm * dm + w.d_head * d_x + 2 * w.d_head + 6 * w.d_p + w.d_a * w.d_p
                     + w.d_h * w.d_e)
    n_prev = min(j - 1, 2)
    return {
        "router_bwd_gemm": dict(flops=2 * T * d * NP, bytes=T * d * es + NP * d * es + splits * T * NP * 4),
        "router_bwd_token": dict(flops=0, bytes=T * ((3 if j > 1 else 2) * dm * dm * 4 + (1 + n_prev) * d * es
                                                     + splits * NP * 4 + (2 * NP + vec + 8) * 4
                                                     + (dm * 4 if c_given and j > 1 else 0))),
        "router_bwd_products": dict(flops=4 * T * NP * d + small, bytes=(2 * NP + vec) * T * 4 + T * d * (es + 4)
                                    + 2 * T * d * 4),
        "router_bwd_rows": dict(flops=0, bytes=T * d * ((1 + n_prev) * es + 2 * (1 + n_prev) * 4)),
    }


def bench_router_backward(args, w):
    """A step is one hero_router_backward call at the workload's routed layer over its T tokens
    (post-attention states, router weights, the state entering the layer, dL/dlogit and a carried
    state gradient resident in HBM)."""
    import numpy as np
    import torch
    from paper_2609_08189_amd import hero as H
    from paper_2609_08189_amd import synth
    from paper_2609_08189_amd.device import DeviceProblem, DeviceRouterBackward

    j = w.layer_j
    if j <= 0 or w.n_layers > 0 or w.state_dtype != "f32":
        sys.exit("--router-backward times one routed layer's router with S in fp32")
    print(f"# preparing the router backward at {describe(w, j)}", file=sys.stderr, flush=True)
    prob = synth.make_problem(w, seed=args.seed, layer_j=j)
    rng = np.random.default_rng(args.seed + 77)
    T, dm = w.T, w.d_m
    dl = rng.standard_normal(T).astype(np.float32)
    dS = (0.05 * rng.standard_normal((T, dm, dm))).astype(np.float32)
    dz = (0.1 * rng.standard_normal((T, dm))).astype(np.float32)
    dph = rng.standard_normal(T).astype(np.float32)
    dmh = rng.standard_normal(T).astype(np.float32)
    dp = DeviceProblem(prob, stats=False)
    c_given = not args.reread_c
    rb = DeviceRouterBackward(dp, j, dl, dS, dz, dph, dmh, c_from_forward=c_given)
    stream = dp.stream()
    ev = HipEvents()
    for _ in range(1 + args.warmup):
        rb.run()
    torch.cuda.synchronize()
    K = args.steps
    works = router_backward_work(w, j, c_given)
    per, handles = {}, {}
    for name in RBWD_KERNELS:
        handles[name] = (ev.create(K), ev.create(K))
        H.hero_kernel_timer(H.HERO_K[name], *handles[name])
    for _ in range(K):
        rb.run()
    torch.cuda.synchronize()
    for name, (a, b) in handles.items():
        H.hero_kernel_timer(H.HERO_K[name], [], [])
        us = 1000.0 * sum(ev.elapsed_ms(x, y) for x, y in zip(a, b)) / K
        wk = works[name]
        per[name] = {"us": round(us, 2), "tflops": round(wk["flops"] / us * 1e-6, 1) if wk["flops"] else None,
                     "gbs": round(wk["bytes"] / us * 1e-3, 1)}
        ev.destroy(a + b)
    dom = max(per, key=lambda k: per[k]["us"])
    ks, ke = ev.create(K), ev.create(K)
    H.hero_kernel_timer(H.HERO_K[dom], ks, ke)
    t_start, t_stop = ev.create(2)
    marks = ev.create(K - 1)
    torch.cuda.synchronize()
    ev.record(t_start, stream)
    for i in range(K):
        rb.run()
        if i < K - 1:
            ev.record(marks[i], stream)
    ev.record(t_stop, stream)
    torch.cuda.synchronize()
    H.hero_kernel_timer(H.HERO_K[dom], [], [])
    ms_step = ev.elapsed_ms(t_start, t_stop) / K
    bounds = [t_start] + marks + [t_stop]
    step_ms = sorted(ev.elapsed_ms(a, b) for a, b in zip(bounds[:-1], bounds[1:]))
    dom_ms = sum(ev.elapsed_ms(a, b) for a, b in zip(ks, ke)) / K
    if dom == "router_bwd_products":      # fp32 products on the vector ALUs
        achieved, peak, unit, bound = works[dom]["flops"] / (dom_ms * 1e-3) * 1e-12, PEAK_F32_TFLOPS, "TFLOP/s", "alu"
        wpl = f"4 T (d_e + d_head) d FLOP (dW_hd, dpsi_1 and dP [W_hd; psi_1]) + the small weights' products"
    elif works[dom]["flops"]:
        achieved, peak, unit, bound = (works[dom]["flops"] / (dom_ms * 1e-3) * 1e-12,
                                       PEAK_BF16_TFLOPS if w.dtype == "bf16" else PEAK_F32_TFLOPS, "TFLOP/s", "mfma")
        wpl = "2 T d (d_e + d_head) FLOP"
    else:
        achieved, peak, unit, bound = works[dom]["bytes"] / (dom_ms * 1e-3) * 1e-9, PEAK_HBM_GBS, "GB/s", "hbm"
        wpl = "per token: S_{j-1} read, dL/dS read and written (4 d_m^2 B each), rows and vectors"
        if c_given:
            wpl += ", the forward's memory read c"
    result = {
        "metric": "router backward tokens/sec at Llama-3.1-8B shape; % roofline",
        "value": round(T / (ms_step * 1e-3), 1), "unit": "tokens/s", "n_gpus": 1, "steps": K,
        "warmup": args.warmup, "ms_per_step": round(ms_step, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": w.dtype, "data": "synthetic",
        "config": {"workload": (f"backward of the router (Sec. 3.2 in reverse) at {describe(w, j)}; dL/dlogit "
                                f"N(0,1), carried dL/dS N(0,0.05^2), dL/dzeta N(0,0.1^2), dL/dp, dL/dm N(0,1); "
                                + ("the forward's memory read c handed over" if c_given
                                   else "the memory read c recomputed from S_{j-1}")),
                   "global_batch": w.batch, "seq_len": w.seq, "tokens": T, "parallelism": "none"},
        "roofline": {"bound": bound, "achieved": round(achieved, 1), "peak": peak, "unit": unit,
                     "frac": round(achieved / peak, 4), "traffic": None, "kernel": dom,
                     "avg_launch_us": round(1000 * dom_ms, 2),
                     "work_per_launch": f"{wpl}: {works[dom]['flops'] / 1e9:.1f} GFLOP, {works[dom]['bytes'] / 1e6:.1f} MB"},
        "step_ms": step_stats(step_ms),
        "kernels": per,
    }
    if not args.no_cpu_baseline:
        print("# timing the CPU oracle on a token sample", file=sys.stderr, flush=True)
        result["cpu_baseline"] = cpu_baseline_router_backward(w, prob, j, dl, dS, dz, dph, dmh, args.cpu_target_s)
    print(json.dumps(result), flush=True)


def cpu_baseline_router_backward(w, prob, j, dl, dS, dz, dph, dmh, target_s=12.0):
    """The float64 oracle's router forward and router_layer_backward on the first n tokens, n
    growing until the call takes >= target_s or covers all T (then repeated, up to 8 runs)."""
    import numpy as np
    from threadpoolctl import threadpool_info
    from oracle import hero_oracle as O
    from tests.oracle_inputs import adapter_of, dims_of, ffn_of, router_of

    T = w.T
    dims, R = dims_of(w), router_of(prob)
    F, A = ffn_of(prob.ffn[0]), adapter_of(prob.adapter[0])
    eta = float(prob.eta[j - 1])

    def run(n):
        st = O.State(prob.S[:n].astype("f8"), prob.zeta[:n].astype("f8"), prob.p_hist[:n].astype("f8"),
                     prob.m_hist[:n].astype("f8"))
        h1 = prob.hbar_prev1.f64[:n] if j >= 2 else None
        h2 = prob.hbar_prev2.f64[:n] if j >= 3 else None
        t0 = time.perf_counter()
        fwd = O.routed_layer(j, dims, prob.hbar.f64[:n], h1, h2, st, F, R, A, eta, mode="threshold",
                             round_output=False, compute_rows=np.zeros(n, dtype=bool))
        O.router_layer_backward(j, dims, prob.hbar.f64[:n], h1, h2, st, fwd, R, dl[:n].astype("f8"),
                                dS[:n].astype("f8"), dz[:n].astype("f8"), dph[:n].astype("f8"),
                                dmh[:n].astype("f8"), O._zero_router(R))
        return time.perf_counter() - t0

    n = 64
    while True:
        dt = run(n)
        if dt >= target_s or n >= T:
            break
        n = min(T, max(2 * n, int(n * target_s / max(dt, 1e-3) * 1.1)))
    reps = 1
    while dt < target_s and reps < 8:
        dt += run(n)
        reps += 1
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    return {"value": n * reps / dt, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": f"the first {n} of {T} tokens (the router's forward and backward at this layer, float64 "
                      f"numpy)" + (f", run {reps} times" if reps > 1 else "") + f", {dt:.1f} s"}


# the paper's two Llama-3.1-8B operating points (Table 1: 26.87 % and 38.82 % skip)
PAPER_SKIPS = (0.2687, 0.3882)
# the router, compaction and memory kernels (timed and judged as one group against HBM)
ROUTER_GROUP = ("rowstats", "router_gemm", "router_pre", "router_mem", "router_post", "select")
BAND = 1e-3          # decision band on the gate around the layer's threshold


def measure_forward(w, dp, K, warmup, memory="matrix", graph=False, kernels=True):
    """Time K steps of the workload's call (a hero_routed_layer call at the workload's j, or one
    hero_routed_stack call) with every input resident in HBM.

    One checked call with the optional stats outputs comes first (realized branch sizes, masks,
    logits, lambda per layer); the timed steps run without them.  The dominant kernel (FFN gate/up)
    is bracketed live by HIP events on the call's stream.  With kernels=True a second, untimed pass
    instruments every kernel of the layer for the per-kernel table."""
    import torch
    from paper_2609_08189_amd import hero as H
    stack = w.layer_j <= 0
    j = w.layer_j
    L = w.L_R if stack else 1
    stream = dp.stream()
    ev = HipEvents()
    step = dp.run_stack if stack else (lambda: dp.run_layer(j))
    stats_saved = dp.stats
    step()
    torch.cuda.synchronize()
    layer_stats = [s.host() for s in dp.stats]
    nfs = [ls["n_ffn"] for ls in layer_stats]
    nas = [ls["n_ad"] for ls in layer_stats]
    dp.stats = None
    try:
        for _ in range(warmup):
            step()
        torch.cuda.synchronize()
        dom = "ffn_gate_up"
        n_dom = K * sum(1 for x in nfs if x > 0)   # launches of the dominant kernel in the timed steps
        run = graphed(step) if graph else step
        ks, ke = ev.create(n_dom), ev.create(n_dom)
        if not graph:
            H.hero_kernel_timer(H.HERO_K[dom], ks, ke)
        t_start, t_stop = ev.create(2)
        torch.cuda.synchronize()
        marks = ev.create(K - 1)            # step boundaries inside the timed region
        ev.record(t_start, stream)
        for i in range(K):
            run()
            if i < K - 1:
                ev.record(marks[i], stream)
        ev.record(t_stop, stream)
        torch.cuda.synchronize()
        H.hero_kernel_timer(H.HERO_K[dom], [], [])
        total_ms = ev.elapsed_ms(t_start, t_stop)
        bounds = [t_start] + marks + [t_stop]
        step_ms = sorted(ev.elapsed_ms(a, b) for a, b in zip(bounds[:-1], bounds[1:]))
        dom_ms_step = 0.0 if graph else sum(ev.elapsed_ms(a, b) for a, b in zip(ks, ke)) / K
        ev.destroy(ks + ke + [t_start, t_stop] + marks)
        ms_step = total_ms / K

        layers = list(range(1, L + 1)) if stack else [j]
        works = [kernel_work(w, nf, na, w.T, jj, memory) for nf, na, jj in zip(nfs, nas, layers)]
        if w.ablation & 12:            # no memory pass under the memory-less ablations
            for wk in works:
                wk["router_mem"] = dict(flops=0, bytes=0)
        per = {}
        if kernels or graph:
            names = [k for k in H.KERNELS[:H.HERO_K["adapter_up"] + 1]
                     if not (k == "router_mem" and w.ablation & 12)]
            handles = {}
            for name in names:
                a, b = ev.create(K * L), ev.create(K * L)
                handles[name] = (a, b)
                H.hero_kernel_timer(H.HERO_K[name], a, b)
            for _ in range(K):
                step()
            torch.cuda.synchronize()
            for name in names:
                H.hero_kernel_timer(H.HERO_K[name], [], [])
                a, b = handles[name]
                active = [i for i in range(L) if not ((name.startswith("ffn") and nfs[i] == 0) or
                                                       (name.startswith("adapter") and nas[i] == 0))]
                if active:
                    n_launch = K * len(active)
                    us = 1000.0 * sum(ev.elapsed_ms(x, y) for x, y in zip(a[:n_launch], b[:n_launch])) / n_launch
                    fl = sum(works[i][name]["flops"] for i in active) / len(active)
                    by = sum(works[i][name]["bytes"] for i in active) / len(active)
                    per[name] = {"us": round(us, 2), "tflops": round(fl / us * 1e-6, 1) if fl else None,
                                 "gbs": round(by / us * 1e-3, 1)}
                ev.destroy(a + b)
        if graph:
            dom_ms_step = per[dom]["us"] * sum(1 for x in nfs if x > 0) / 1000.0
    finally:
        dp.stats = stats_saved
    return dict(ms_step=ms_step, step_ms=step_ms, dom_ms_step=dom_ms_step, layer_stats=layer_stats,
                nfs=nfs, nas=nas, works=works, per=per, K=K, L=L, stack=stack, j=j)


def dominant_roofline(w, m, traffic=None):
    """Roofline of the FFN gate/up product: algorithmic work per step over its live-timed duration,
    against the tighter roof for the row count (MFMA at prefill sizes, HBM for decode batches)."""
    dom = "ffn_gate_up"
    nfs, K = m["nfs"], m["K"]
    dflops = sum(wk[dom]["flops"] for wk in m["works"])          # per step
    dbytes = sum(wk[dom]["bytes"] for wk in m["works"])
    peak_f = PEAK_BF16_TFLOPS if w.dtype == "bf16" else PEAK_F32_TFLOPS
    n_launch_step = max(1, sum(1 for x in nfs if x > 0))
    dom_ms = m["dom_ms_step"]
    hbm_bound = dbytes / (PEAK_HBM_GBS * 1e9) > dflops / (peak_f * 1e12)
    if hbm_bound:
        achieved, peak, unit = dbytes / (dom_ms * 1e-3) * 1e-9, PEAK_HBM_GBS, "GB/s"
        per_unit = "weights 2*d*d_ff*2 B per launch + (d + d_ff)*2 B per FFN token"
        total = f"{dbytes / n_launch_step / 1e6:.1f} MB"
    else:
        achieved, peak, unit = dflops / (dom_ms * 1e-3) * 1e-12, peak_f, "TFLOP/s"
        per_unit = "4*d*d_ff FLOP per FFN token"
        total = f"{dflops / n_launch_step / 1e9:.1f} GFLOP"
    nf_mean = sum(nfs) / n_launch_step
    return {"bound": "hbm" if hbm_bound else "mfma", "achieved": round(achieved, 1), "peak": peak,
            "unit": unit, "frac": round(achieved / peak, 4), "traffic": traffic,
            "kernel": dom, "avg_launch_us": round(dom_ms * 1e3 / n_launch_step, 2),
            "launches_per_step": n_launch_step,
            "work_per_launch": f"{per_unit} x {nf_mean:.0f} FFN tokens = {total}",
            "traffic_note": "HBM bytes read + written per launch (rocprofv3 FETCH_SIZE x2 + WRITE_SIZE x1, "
                            "calibrated on a 1 GiB copy) from profiles/, null if the GEMM sources changed "
                            "since or for workloads the counters were not taken on"}


def router_group(m):
    """The router, compaction and memory kernels as one group: algorithmic bytes of a mean layer
    over the group's summed mean launch times, against the HBM peak."""
    per, works = m["per"], m["works"]
    if not all(k in per for k in ROUTER_GROUP if k != "router_mem") or not per:
        return None
    names = [k for k in ROUTER_GROUP if k in per]
    us = sum(per[k]["us"] for k in names)
    by = sum(wk[k]["bytes"] for wk in works for k in names) / len(works)
    return {"kernels": names, "us": round(us, 2), "bytes": int(by), "gbs": round(by / us * 1e-3, 1),
            "frac_hbm": round(by / us * 1e-3 / PEAK_HBM_GBS, 4)}


def routing_report(w, layer_stats):
    """Realized skip per layer and the number of tokens whose gate lies within BAND of the layer's
    threshold (sigma(lambda_j) in budget mode, tau in threshold mode): decisions the rounding of
    the logit could flip."""
    import numpy as np
    skip, band, lam = [], [], []
    for ls in layer_stats:
        T = ls["n_ffn"] + ls["n_ad"]
        skip.append(round(ls["n_ad"] / max(T, 1), 5))
        g = 1.0 / (1.0 + np.exp(-ls["logit"].astype(np.float64)))
        thr = 1.0 / (1.0 + math.exp(-ls["lam"])) if w.mode == "budget" else w.tau
        band.append(int(np.sum(np.abs(g - thr) < BAND)))
        lam.append(round(ls["lam"], 6))
    out = {"mode": w.mode, "realized_skip_per_layer": skip,
           "realized_skip_mean": round(sum(skip) / len(skip), 5),
           "band_count_per_layer": band, "band_count_total": sum(band), "band": BAND}
    if w.mode == "budget":
        out["lambda_per_layer"] = lam
    return out


def cpu_baseline_stack(prob, layer_stats, n_tokens=256, target_s=12.0, single_tokens=16):
    """Time the float64 oracle on a token sample of the stack call: n_tokens spread evenly over the
    sequences go through all L_R layers, teacher-forced at each layer to the GPU's branch decision
    (and, in budget mode, given the GPU's lambda_j in place of the sample's own quantile).  Tokens are
    independent given these, so tokens/s of the sample is the oracle's rate on the whole call.  The
    weights' float64 decoding is data preparation and is not timed.  A one-thread figure runs
    single_tokens tokens through the first two layers with BLAS held to one thread, scaled to L_R
    layers."""
    import numpy as np
    from threadpoolctl import threadpool_info, threadpool_limits
    from oracle import hero_oracle as O
    from tests.oracle_inputs import adapter_of, dims_of, ffn_of, router_of

    w = prob.w
    T = prob.hbar.shape[0]
    dims, R = dims_of(w), router_of(prob)
    beta_all = None if prob.beta is None else prob.beta.astype("f8")

    def chain(rows, n_layers):
        h = prob.hbar.f64[rows]
        prev1 = prev2 = None
        st = O.State.initial(len(rows), w.d_m)
        beta = None if beta_all is None else beta_all[rows]
        dt = 0.0
        for jj in range(1, n_layers + 1):
            F, A = ffn_of(prob.ffn[jj - 1]), adapter_of(prob.adapter[jj - 1])
            ls = layer_stats[jj - 1]
            t0 = time.perf_counter()
            res = O.routed_layer(jj, dims, h, prev1, prev2, st, F, R, A, float(prob.eta[jj - 1]),
                                 mode=w.mode, budget=w.budget, tau=w.tau, beta=beta,
                                 forced_ffn=ls["mask"][rows],
                                 lam_given=ls["lam"] if w.mode == "budget" else None)
            dt += time.perf_counter() - t0
            prev2, prev1, h, st = prev1, h, res.h, res.state
        return dt

    rows = np.linspace(0, T - 1, min(n_tokens, T)).astype(np.int64)
    dt = chain(rows, w.L_R)
    reps = 1
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    with threadpool_limits(limits=1):
        srows = rows[:: max(1, len(rows) // single_tokens)][:single_tokens]
        n1 = min(2, w.L_R)
        dt1 = chain(srows, n1) * w.L_R / n1
    cpu_model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            cpu_model = next((l.split(":", 1)[1].strip() for l in f if l.startswith("model name")), cpu_model)
    except OSError:
        pass
    return {"value": round(len(rows) * reps / dt, 2), "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "nproc": os.cpu_count(), "omp_num_threads": os.environ.get("OMP_NUM_THREADS"), "cpu_model": cpu_model,
            "single_thread_value": round(len(srows) / dt1, 3),
            "sample": f"{len(rows)} of {T} tokens spread evenly over the {w.batch} sequences, through all "
                      f"{w.L_R} routed layers of the stack call (router, memory, branch; float64 numpy), each "
                      f"layer teacher-forced to the GPU's branch decisions" +
                      (" and lambda_j" if w.mode == "budget" else "") + f": {dt:.1f} s on {threads} BLAS threads; "
                      f"single thread: {len(srows)} tokens through layers 1-{n1}, scaled by {w.L_R}/{n1}"}


def other_skip_point(w, dp, budget, K, warmup):
    """The same call measured at another skip budget on the same device problem (the inputs do not
    depend on the budget; only the call's routing argument changes): tokens/s, the step time, branch
    sizes and the dominant kernel's roofline fraction."""
    saved_budget = dp.routing_s.budget
    dp.routing_s.budget = budget
    try:
        m = measure_forward(w.replace(budget=budget), dp, K, warmup, kernels=False)
    finally:
        dp.routing_s.budget = saved_budget
    roof = dominant_roofline(w.replace(budget=budget), m)
    return {"budget": budget, "value": round(w.T / (m["ms_step"] * 1e-3), 1), "unit": "tokens/s",
            "ms_per_step": round(m["ms_step"], 4), "steps": K, "n_ffn": sum(m["nfs"]),
            "n_adapter": sum(m["nas"]), "ffn_gate_up_us": roof["avg_launch_us"],
            "ffn_gate_up_frac": roof["frac"],
            "realized_skip_mean": routing_report(w, m["layer_stats"])["realized_skip_mean"]}


def layer_point(args, name="llama31_8b_layer"):
    """The single routed layer (Llama-3.1-8B shape, j = 17 of 32, T = 4096, 26.87 % skip) measured
    beside the stack: tokens/s, the gate/up roofline and the router group's HBM rate."""
    import torch
    from paper_2609_08189_amd import synth
    from paper_2609_08189_amd.device import DeviceProblem
    w = synth.WORKLOADS[name]
    print(f"# preparing {describe(w, w.layer_j)}", file=sys.stderr, flush=True)
    prob = synth.make_problem(w, seed=args.seed)
    dp = DeviceProblem(prob, device="cuda:0", stats=True)
    m = measure_forward(w, dp, args.steps, args.warmup)
    out = {"workload": describe(w, w.layer_j), "value": round(w.T / (m["ms_step"] * 1e-3), 1),
           "unit": "tokens/s", "ms_per_step": round(m["ms_step"], 4), "n_ffn": m["nfs"][0], "n_adapter": m["nas"][0],
           "roofline": dominant_roofline(w, m, counted_traffic("ffn_gate_up", name)),
           "router_group": router_group(m), "whole_call": ideal_fraction(m["works"], m["ms_step"], w.dtype, False),
           "kernels": m["per"]}
    del dp
    torch.cuda.empty_cache()
    return out


def bench_peaks(args):
    """The board's practical ceilings, measured live: the bf16 matrix-core loop of hero_peak_mfma
    (register operands, two waves per SIMD on all 256 CUs) with zero and with random operands, and a
    plain 1 GiB device-to-device copy (read + write).  The roofline fractions in the other lines use
    the published peaks (2.5 PFLOP/s, 8 TB/s); these say how much of them a kernel can reach here."""
    import torch
    from paper_2609_08189_amd import hero as H
    ev = HipEvents()
    stream = torch.cuda.current_stream().cuda_stream
    sink = torch.zeros(16, dtype=torch.float32, device="cuda:0")
    out = {"metric": "practical ceilings of the board", "n_gpus": 1}
    iters, wgs, reps = 20000, 256, 5
    for name, rnd, mi16 in (("mfma_bf16_zeros", False, False), ("mfma_bf16_random", True, False),
                            ("mfma16_bf16_zeros", False, True), ("mfma16_bf16_random", True, True)):
        H.hero_peak_mfma(rnd, iters, wgs, sink, stream, mi16)    # warm-up launch
        torch.cuda.synchronize()
        a, b = ev.create(2)
        ev.record(a, stream)
        flop = sum(H.hero_peak_mfma(rnd, iters, wgs, sink, stream, mi16) for _ in range(reps))
        ev.record(b, stream)
        ms = ev.elapsed_ms(a, b)
        ev.destroy([a, b])
        tf = flop / (ms * 1e-3) * 1e-12
        out[name] = {"tflops": round(tf, 1), "frac_of_2500": round(tf / PEAK_BF16_TFLOPS, 4),
                     "implied_clock_ghz": round(tf / PEAK_BF16_TFLOPS * 2.4, 3),
                     "launch_us": round(1000 * ms / reps, 1), "launches": reps}
    n = 1 << 30
    src = torch.empty(n, dtype=torch.uint8, device="cuda:0").fill_(1)
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    a, b = ev.create(2)
    ev.record(a, stream)
    for _ in range(reps):
        dst.copy_(src)
    ev.record(b, stream)
    ms = ev.elapsed_ms(a, b) / reps
    ev.destroy([a, b])
    gbs = 2 * n / (ms * 1e-3) * 1e-9
    out["device_copy_1gib"] = {"gbs_read_plus_write": round(gbs, 1), "frac_of_8000": round(gbs / PEAK_HBM_GBS, 4),
                               "copy_us": round(1000 * ms, 1), "launches": reps}
    del src, dst
    torch.cuda.empty_cache()

    # cold HBM reads: each launch reads a region the previous launches did not touch (regions
    # rotate through more than the 256 MB MALL holds)
    def cold_reads(region, nreg, visit):
        buf = torch.empty(nreg * region, dtype=torch.uint8, device="cuda:0").fill_(1)
        torch.cuda.synchronize()
        H.hero_peak_read(buf[:region], region, visit, sink, stream)
        torch.cuda.synchronize()
        a, b = ev.create(2)
        ev.record(a, stream)
        for r in range(2 * nreg):
            H.hero_peak_read(buf[((r + 1) % nreg) * region:], region, visit, sink, stream)
        ev.record(b, stream)
        us = 1000 * ev.elapsed_ms(a, b) / (2 * nreg)
        ev.destroy([a, b])
        del buf
        torch.cuda.empty_cache()
        return {"gbs": round(region / (us * 1e-6) * 1e-9, 1), "frac_of_8000": round(region / (us * 1e-6) * 1e-9 / PEAK_HBM_GBS, 4),
                "launch_us": round(us, 1), "bytes": region, "launches": 2 * nreg}
    out["hbm_read_contiguous"] = cold_reads(1 << 30, 4, 0)
    # a decode step's weight stream: 256 workgroups x 96 rows of 8 KiB, visit_bytes of each row per step
    rows_region = 256 * 96 * 8192
    for vb in (128, 256, 512):
        out[f"hbm_read_rows_{vb}B_visits"] = cold_reads(rows_region, 8, vb)

    # the vendor library (hipBLASLt through torch.matmul, bf16 in, fp32 accumulation, bf16 out) on
    # the plain, ungathered FFN shapes of the Llama-3.1-8B stack and layer workloads: the FFN rows of
    # one routed layer (T minus the budget's skipped tokens) by [W_g; W_u] (N = 2 d_ff) and by W_d
    from paper_2609_08189_amd import synth
    gen = torch.Generator(device="cuda:0").manual_seed(0)
    for wname in ("llama31_8b_stack", "llama31_8b_layer"):
        w = synth.WORKLOADS[wname]
        m = w.T - int(math.floor(w.budget * w.T + 0.5))
        for pname, n, k in (("gate_up", 2 * w.d_ff, w.d), ("down", w.d, w.d_ff)):
            x = torch.randn(m, k, device="cuda:0", generator=gen).to(torch.bfloat16)
            wt = (0.02 * torch.randn(n, k, device="cuda:0", generator=gen)).to(torch.bfloat16)
            y = x @ wt.t()
            torch.cuda.synchronize()
            a, b = ev.create(2)
            ev.record(a, stream)
            for _ in range(reps):
                y = x @ wt.t()
            ev.record(b, stream)
            us = 1000 * ev.elapsed_ms(a, b) / reps
            ev.destroy([a, b])
            tf = 2.0 * m * n * k / (us * 1e-6) * 1e-12
            out[f"vendor_gemm_{wname}_{pname}"] = {"m": m, "n": n, "k": k, "us": round(us, 1), "tflops": round(tf, 1),
                                                  "frac_of_2500": round(tf / PEAK_BF16_TFLOPS, 4), "launches": reps}
            del x, wt, y
            torch.cuda.empty_cache()
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="llama31_8b_stack")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--ablation", type=int, default=0,
                    help="router ablation bits (1 w/o Pos State, 2 w/o Aux State, 4 w/o MemRead, 8 w/o History)")
    ap.add_argument("--state", choices=("f32", "bf16"), default="f32",
                    help="storage of the router memory S between layers")
    ap.add_argument("--budget", type=float, default=None,
                    help="skip budget in place of the workload's own (budget-mode workloads)")
    ap.add_argument("--graph", action="store_true", default=None,
                    help="time replays of the call captured once as a HIP graph (kernel times then come "
                         "from the instrumented pass); the default for decode-sized calls (at most 256 tokens), "
                         "whose launch gaps are a visible share of the step")
    ap.add_argument("--eager", action="store_true",
                    help="time eager launches even for a decode-sized call")
    ap.add_argument("--untiled", action="store_true",
                    help="a decode-sized call reads the FFN weights row-major instead of the tiled copies "
                         "of hero_ffn_decode_weights_make")
    ap.add_argument("--backward", action="store_true",
                    help="time the backward of the routed block (training side) instead of the forward")
    ap.add_argument("--router-backward", action="store_true",
                    help="time the backward of the router at the workload's routed layer instead")
    ap.add_argument("--reread-c", action="store_true",
                    help="with --router-backward: recompute the memory read from S_{j-1} instead of taking "
                         "the forward's (hero_state.c_read)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-layer-point", action="store_true",
                    help="skip the single-layer measurement that accompanies the stack line")
    ap.add_argument("--cpu-target-s", type=float, default=12.0)
    ap.add_argument("--cpu-tokens", type=int, default=1024,
                    help="token sample of the stack call for the CPU oracle")
    ap.add_argument("--memory", choices=("matrix", "history"), default="matrix",
                    help="router memory as the matrix S (the paper's form) or in depth-history form")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="also run a plain device-to-device copy of this many MiB (HBM counter calibration)")
    ap.add_argument("--peaks", action="store_true",
                    help="measure the chip's practical ceilings instead (MFMA loops, device copy, cold HBM reads) and exit")
    ap.add_argument("--summarize", metavar="DIR",
                    help="print a summary of rocprofv3 CSV output found under DIR and exit (no GPU)")
    ap.add_argument("--window", type=int, nargs=2, metavar=("SKIP", "COUNT"),
                    help="with --summarize: per-kernel mean over dispatches SKIP..SKIP+COUNT-1")
    args = ap.parse_args()
    if args.summarize:
        summarize_rocprof(args.summarize, window=args.window)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only: the routed FFN path shards over tokens with no "
              f"communication in threshold mode, and runs on several GPUs are not implemented "
              f"(asked for --gpus {args.gpus}).", file=sys.stderr)
        sys.exit(2)
    if args.peaks:
        return bench_peaks(args)

    import torch
    from paper_2609_08189_amd import synth
    from paper_2609_08189_amd.device import DeviceProblem

    w = synth.WORKLOADS[args.workload]
    if args.graph is None:
        args.graph = w.T <= DECODE_TOKENS and not args.eager and w.n_layers == 0
    default_line = (args.budget is None and not args.ablation and args.state == "f32"
                    and args.memory == "matrix" and (not args.graph or w.T <= DECODE_TOKENS))
    if args.budget is not None:
        if w.mode != "budget" or not 0.0 <= args.budget <= 1.0:
            sys.exit("--budget needs a budget-mode workload and a fraction in [0, 1]")
        w = w.replace(budget=args.budget)
    if args.ablation:
        if not 0 < args.ablation <= 15:
            sys.exit("--ablation takes bits 1, 2, 4, 8")
        w = w.replace(ablation=args.ablation)
    if args.state == "bf16":
        if args.memory != "matrix":
            sys.exit("--state bf16 needs the matrix-form memory")
        w = w.replace(state_dtype="bf16")
    if args.backward:
        return bench_backward(args, w)
    if args.router_backward:
        return bench_router_backward(args, w)
    if w.n_layers > 0:
        return bench_decoder(args, w)
    stack = w.layer_j <= 0          # a stack workload: a step is one hero_routed_stack call
    j = w.layer_j
    print(f"# preparing {describe(w, j)}", file=sys.stderr, flush=True)
    prob = synth.make_problem(w, seed=args.seed)
    # a decode step streams every FFN weight once: it reads the copies in the streaming order
    tiled = w.dtype == "bf16" and w.T <= DECODE_TOKENS and not args.untiled
    dp = DeviceProblem(prob, device="cuda:0", stats=True, history=args.memory == "history", tiled=tiled)
    m = measure_forward(w, dp, args.steps, args.warmup, memory=args.memory, graph=args.graph)
    K, L, nfs, nas = m["K"], m["L"], m["nfs"], m["nas"]
    print(f"# timed {K} steps: {m['ms_step']:.4f} ms/step", file=sys.stderr, flush=True)
    result = {
        "metric": "routed-FFN-stack tokens/sec at Llama-3.1-8B shape; % MFMA/HBM roofline",
        "value": round(w.T / (m["ms_step"] * 1e-3), 1), "unit": "tokens/s", "n_gpus": 1, "steps": K,
        "warmup": args.warmup, "ms_per_step": round(m["ms_step"], 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": w.dtype, "data": "synthetic",
        "config": {"workload": describe(w, j) + ("" if args.state == "f32" else ", S stored in bf16") +
                               ("" if not args.ablation else f", router ablation bits {args.ablation}") +
                               ("" if args.memory == "matrix" else ", router memory in depth-history form"),
                   "memory": args.memory, "state": args.state, "global_batch": w.batch, "seq_len": w.seq,
                   "tokens": w.T, "layers_per_step": L, "parallelism": "none", "hip_graph": bool(args.graph),
                   "ffn_weights": "tiled" if tiled else "row-major",
                   "n_ffn": sum(nfs), "n_adapter": sum(nas)},
        "roofline": dominant_roofline(w, m, counted_traffic("ffn_gate_up", args.workload) if default_line else None),
        "router_group": router_group(m),
        "step_ms": step_stats(m["step_ms"]),
        "whole_call": ideal_fraction(m["works"], m["ms_step"], w.dtype, stack),
        "routing": routing_report(w, m["layer_stats"]),
        "kernels": m["per"],
    }
    # the paper's other Llama-3.1-8B operating point (Table 1: 26.87 % and 38.82 % skip), on the
    # same device problem
    others = [b for b in PAPER_SKIPS if abs(b - w.budget) > 1e-6]
    if w.mode == "budget" and default_line and args.workload.startswith("llama31_8b") and others:
        print(f"# timing the call at skip budget {others[0]}", file=sys.stderr, flush=True)
        result["other_skip"] = other_skip_point(w, dp, others[0], K, args.warmup)
    if not args.no_cpu_baseline:
        print("# timing the CPU oracle on a token sample", file=sys.stderr, flush=True)
        if stack:
            result["cpu_baseline"] = cpu_baseline_stack(prob, m["layer_stats"], args.cpu_tokens, args.cpu_target_s)
        else:
            result["cpu_baseline"] = cpu_baseline(prob, m["layer_stats"][0], j, target_s=args.cpu_target_s)
    if stack and default_line and args.workload == "llama31_8b_stack" and not args.no_layer_point:
        del dp
        torch.cuda.empty_cache()
        result["layer"] = layer_point(args)
    print(json.dumps(result), flush=True)
    if args.copy_calibration_mib > 0:
        n = args.copy_calibration_mib << 20
        src = torch.empty(n, dtype=torch.uint8, device="cuda:0").fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        print(f"# calibration copy: {n} bytes read, {n} bytes written", file=sys.stderr, flush=True)


if __name__ == "__main__":
    main()
