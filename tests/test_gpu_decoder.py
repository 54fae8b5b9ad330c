"""GPU parity of the full decoder through the C ABI: the attention sub-block
(hero_attention_block) against the oracle's Llama attention, and hero_decoder_stack (attention
at every block, the pretrained FFN at the first blocks, routing at the last L_R) against the
oracle decoder."""
import numpy as np
import pytest

from oracle import hero_oracle as O
from paper_2609_08189_amd import synth
from tests.oracle_inputs import adims_of, attn_of, dims_of
from tests.parity import TOL, check_decoder, row_rel_err

pytestmark = pytest.mark.gpu

SMALL = synth.Workload("decoder_small", "bf16", d=512, d_ff=1408, d_r=64, L_R=2, d_m=64, T=600,
                       mode="budget", budget=0.3, batch=2, seq=300, n_layers=4, n_heads=4,
                       n_kv_heads=2, head_dim=128, rope_theta=10000.0)


def _attention(w, layer=0, seed=0, rows=None):
    import torch
    from paper_2609_08189_amd.device import DeviceDecoder, download_f64
    print(f"case {w.name} batch={w.batch} seq={w.seq} d={w.d} heads={w.n_heads}/{w.n_kv_heads} "
          f"layer={layer} seed={seed}", flush=True)
    prob = synth.make_problem(w, seed=seed)
    dd = DeviceDecoder(prob, stats=False)
    hbar = dd.attention(layer)
    got = download_f64(hbar)
    A = attn_of(prob.attn[layer], w, prob.inv_freq)
    ref = O.attention_block(prob.hbar.f64, A, adims_of(w), w.batch, w.seq, dims_of(w), rows=rows)
    sel = np.arange(w.T) if rows is None else np.asarray(rows)
    err = row_rel_err(got[sel], ref[sel])
    moved = np.abs(ref[sel] - prob.hbar.f64[sel]).max()
    print(f"  hbar err {err:.2e} (attention moved h by up to {moved:.2f})", flush=True)
    assert np.isfinite(got).all()
    assert err <= TOL["bf16"], err
    del dd
    torch.cuda.empty_cache()
    return err


@pytest.mark.parametrize("batch,seq,nh,nkv", [(2, 300, 4, 2), (3, 1, 4, 2), (1, 128, 4, 4), (2, 129, 4, 1),
                                              (1, 64, 8, 2), (2, 257, 2, 2)])
def test_attention_block(batch, seq, nh, nkv):
    w = SMALL.replace(batch=batch, seq=seq, T=batch * seq, n_heads=nh, n_kv_heads=nkv)
    _attention(w, layer=1, seed=batch + seq)


def test_attention_block_llama31_8b_full_shape():
    """Llama-3.1-8B attention (32 query / 8 key-value heads of 128, rotary base 5e5), 2 x 2048
    tokens, in the launch configuration the decoder uses; 24 sampled rows, including the first
    and last positions of both sequences."""
    w = synth.WORKLOADS["llama31_8b_decoder"]
    rng = np.random.default_rng(3)
    rows = np.unique(np.concatenate([[0, w.seq - 1, w.seq, w.T - 1],
                                     rng.choice(w.T, size=20, replace=False)]))
    _attention(w, layer=5, seed=0, rows=rows)


@pytest.mark.parametrize("budget", [0.3, 0.75])
def test_decoder_stack(budget):
    """4 blocks (2 with the pretrained FFN, then 2 routed), 2 x 300 tokens."""
    import torch
    from paper_2609_08189_amd.device import DeviceDecoder
    w = SMALL.replace(budget=budget)
    print(f"case {w.name} n_layers={w.n_layers} L_R={w.L_R} budget={budget}", flush=True)
    prob = synth.make_problem(w, seed=11)
    dd = DeviceDecoder(prob)
    dd.run()
    report = {}
    check_decoder(prob, dd.results(), report=report)
    print("  errors:", report, flush=True)
    del dd
    torch.cuda.empty_cache()


def test_decoder_all_blocks_routed_threshold():
    """Every block routed (n_layers = L_R = 3), threshold mode."""
    import torch
    from paper_2609_08189_amd.device import DeviceDecoder
    w = SMALL.replace(n_layers=3, L_R=3, mode="threshold", tau=0.5, batch=1, seq=200, T=200)
    print(f"case {w.name} all routed, threshold", flush=True)
    prob = synth.make_problem(w, seed=12)
    dd = DeviceDecoder(prob)
    dd.run()
    report = {}
    check_decoder(prob, dd.results(), report=report)
    print("  errors:", report, flush=True)
    del dd
    torch.cuda.empty_cache()
