"""Host-side checks of bench.py that need no GPU: the --gpus contract, the rocprofv3 summary
parser, and the rule that roofline.traffic comes from committed counters only while the GEMM
sources they were taken with are unchanged."""
import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_exits_with_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr


def test_traffic_from_committed_counters(monkeypatch):
    import re
    text = open(bench.COUNTERS_MD["llama31_8b_layer"]).read()
    recorded = re.search(r"= `([0-9a-f]{64})`", text).group(1)
    # with the sources the counters were taken with, the gate/up row is reported
    monkeypatch.setattr(bench, "gemm_source_hash", lambda: recorded)
    t = bench.counted_traffic("ffn_gate_up", "llama31_8b_layer")
    assert t is not None and t > 260e6       # at least the algorithmic bytes of the launch
    assert bench.counted_traffic("no_such_kernel", "llama31_8b_layer") is None
    assert bench.counted_traffic("ffn_gate_up", "no_such_workload") is None
    # any other source hash makes the committed counters stale
    monkeypatch.setattr(bench, "gemm_source_hash", lambda: "0" * 64)
    assert bench.counted_traffic("ffn_gate_up", "llama31_8b_layer") is None


def test_default_workload_is_the_8b_stack():
    """The headline line times the metric's own configuration: the 32-layer Llama-3.1-8B routed
    stack over 16 x 2048 tokens at 38.82 % skip."""
    import argparse
    from paper_2609_08189_amd import synth
    src = open(os.path.join(ROOT, "bench.py")).read()
    assert 'ap.add_argument("--workload", default="llama31_8b_stack")' in src
    w = synth.WORKLOADS["llama31_8b_stack"]
    assert (w.d, w.d_ff, w.d_r, w.d_m, w.L_R, w.batch, w.seq, w.T) == (4096, 14336, 64, 128, 32, 16, 2048, 32768)
    assert w.mode == "budget" and w.budget == 0.3882 and w.layer_j == 0


def test_routing_report_band_and_skip():
    import numpy as np
    from paper_2609_08189_amd import synth
    w = synth.WORKLOADS["tiny_f32_stack"]
    lam = 0.25
    logit = np.array([lam - 1e-3, lam, lam + 1e-3, lam + 1.0, lam - 1.0, lam + 3.9e-3, lam + 4.1e-3],
                     dtype=np.float32)
    mask = logit >= lam
    ls = {"logit": logit, "lam": lam, "n_ffn": int(mask.sum()), "n_ad": int((~mask).sum())}
    r = bench.routing_report(w, [ls, ls])
    # sigma'(0.25) ~ 0.2461, so |dsigma| < 1e-3 <=> |dlogit| < ~4.06e-3
    assert r["band_count_per_layer"] == [4, 4] and r["band_count_total"] == 8
    assert r["realized_skip_per_layer"] == [round(2 / 7, 5)] * 2
    assert r["lambda_per_layer"] == [0.25, 0.25]


def test_cpu_baseline_stack_follows_the_gpu_decisions():
    """The stack's oracle baseline runs a token sample through every layer, forced at each layer to
    the given decisions; it reports the multi-thread and the one-thread rate."""
    import numpy as np
    from paper_2609_08189_amd import synth
    from oracle import hero_oracle as O
    from tests.oracle_inputs import adapter_of, dims_of, ffn_of, router_of
    w = synth.WORKLOADS["tiny_f32_stack"]
    prob = synth.make_problem(w, seed=2)
    ref = O.routed_stack(dims_of(w), prob.hbar.f64, [ffn_of(l) for l in prob.ffn], router_of(prob),
                         [adapter_of(l) for l in prob.adapter], prob.eta.astype("f8"),
                         mode=w.mode, budget=w.budget)
    stats = [{"mask": L.use_ffn, "lam": L.lam} for L in ref.layers]
    r = bench.cpu_baseline_stack(prob, stats, n_tokens=32, single_tokens=4)
    assert r["kind"] == "oracle" and r["value"] > 0 and r["single_thread_value"] > 0
    assert r["sample"].startswith(f"32 of {w.T} tokens") and f"all {w.L_R} routed layers" in r["sample"]


def test_summarize_reads_rocprof_csv(tmp_path, capsys):
    d = tmp_path / "prof"
    d.mkdir()
    (d / "x_kernel_stats.csv").write_text(
        '"Name","Calls","TotalDurationNs","AverageNs","Percentage","MinNs","MaxNs","StdDev"\n'
        '"void hero::(anonymous namespace)::k(int)",3,3000,1000,100.0,900,1100,0\n')
    (d / "x_counter_collection.csv").write_text(
        '"Kernel_Name","Counter_Name","Counter_Value"\n"k(int)","FETCH_SIZE",10\n"k(int)","FETCH_SIZE",30\n')
    (d / "x_kernel_trace.csv").write_text(
        '"Kernel_Name","Dispatch_Id","Start_Timestamp","End_Timestamp"\n'
        '"k(int)",1,0,1000\n"k(int)",2,5000,7000\n"k(int)",3,9000,12000\n"j(int)",4,0,500\n')
    bench.summarize_rocprof(str(d), window=(1, 2))
    out = capsys.readouterr().out
    assert "| k(int) | 3 | 0.003 | 1.00 | 0.90 | 1.10 | 100.00 |" in out
    assert "| k(int) | FETCH_SIZE | 2 | 20.0 | 30.0 |" in out
    assert "| k(int) | 2 | 2.50 | 2.00 | 3.00 |" in out      # dispatches 2 and 3 of k
    assert "| j(int) |" not in out.split("dispatches 1..2")[1].split("###")[0]   # j has one dispatch


def test_backward_work_counts():
    """The backward's algorithmic work: e (2 d d_ff), the gate/up recompute and du (4 d d_ff each)
    per FFN token; 6 d r + 4 d r per adapter token; every kernel group has bytes."""
    from paper_2609_08189_amd import synth
    w = synth.WORKLOADS["llama31_8b_layer"]
    n_f, n_a = 2995, 1101
    wk = bench.backward_work(w, n_f, n_a)
    assert set(wk) == set(bench.BWD_KERNELS)
    dd = w.d * w.d_ff
    assert wk["bwd_ffn_e"]["flops"] == 2 * dd * n_f
    assert wk["bwd_ffn_gate_up"]["flops"] == wk["bwd_ffn_du"]["flops"] == 4 * dd * n_f
    assert wk["bwd_adapter"]["flops"] + wk["bwd_adapter_wgrad"]["flops"] == 10 * w.d * w.d_r * n_a
    # the weights dominate the FFN products' bytes: W_d^T once, W_g and W_u (or their transposes) twice
    assert wk["bwd_ffn_e"]["bytes"] >= 2 * dd and wk["bwd_ffn_du"]["bytes"] >= 4 * dd
    assert all(v["bytes"] > 0 for v in wk.values())


def test_graph_flag_and_backward_flag_parse():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--help"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 0 and "--graph" in r.stdout and "--backward" in r.stdout


def test_both_paper_skip_points_are_reported():
    """The default stack workload runs at one of the paper's two Llama-3.1-8B operating points
    (Table 1: 26.87 % and 38.82 % skip); the bench line adds the other as `other_skip`."""
    from paper_2609_08189_amd import synth
    assert bench.PAPER_SKIPS == (0.2687, 0.3882)
    for name, other in (("llama31_8b_stack", 0.2687), ("llama31_8b_layer", 0.3882)):
        w = synth.WORKLOADS[name]
        assert w.mode == "budget" and w.budget in bench.PAPER_SKIPS
        assert [b for b in bench.PAPER_SKIPS if abs(b - w.budget) > 1e-6] == [other]


def test_cpu_baseline_repeats_a_short_whole_call():
    """On a call shorter than the time target the oracle baseline covers every token and repeats
    the whole call (at most 8 runs); the rate is tokens x runs over the summed time."""
    from paper_2609_08189_amd import synth
    from oracle import hero_oracle as O
    from tests.oracle_inputs import adapter_of, dims_of, ffn_of, router_of
    w = synth.WORKLOADS["tiny_f32_stack"].replace(layer_j=3)
    prob = synth.make_problem(w, seed=1, layer_j=3)
    st = O.State(prob.S.astype("f8"), prob.zeta.astype("f8"), prob.p_hist.astype("f8"),
                 prob.m_hist.astype("f8"))
    ref = O.routed_layer(3, dims_of(w), prob.hbar.f64, prob.hbar_prev1.f64, prob.hbar_prev2.f64, st,
                         ffn_of(prob.ffn[0]), router_of(prob), adapter_of(prob.adapter[0]),
                         float(prob.eta[2]), mode=w.mode, budget=w.budget)
    r = bench.cpu_baseline(prob, {"mask": ref.use_ffn, "lam": ref.lam}, 3, target_s=30.0)
    assert r["kind"] == "oracle" and r["value"] > 0
    assert r["sample"].startswith(f"{w.T} of {w.T} tokens") and "run 8 times" in r["sample"]


def test_router_backward_work_counts():
    """The router backward's algorithmic work at the Llama-3.1-8B layer: the recomputed
    pre-activations 2 T d (d_e + d_head) FLOP; the products 4 T (d_e + d_head) d FLOP plus the small
    weights'; the token pass streams S_{j-1} once and dL/dS in and out (3 x 64 KiB per token)."""
    from paper_2609_08189_amd import synth
    w = synth.WORKLOADS["llama31_8b_layer"]
    wk = bench.router_backward_work(w, w.layer_j)
    assert set(wk) == set(bench.RBWD_KERNELS)
    assert wk["router_bwd_gemm"]["flops"] == 2 * 4096 * 4096 * 512
    assert 4 * 4096 * 512 * 4096 < wk["router_bwd_products"]["flops"] < 1.1 * 4 * 4096 * 512 * 4096
    assert wk["router_bwd_token"]["bytes"] > 4096 * 3 * 128 * 128 * 4
    assert bench.router_backward_work(w, 1)["router_bwd_token"]["bytes"] < wk["router_bwd_token"]["bytes"]
