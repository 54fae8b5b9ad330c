"""High-contrast parity cases (test helper).

With the default synthetic weights (std 0.02) the gates of an untrained router sit near 1/2 and
both branch outputs are small next to hbar, so a wrong branch scale barely moves h.  These cases
make such mistakes visible: FFN weights of std 0.05 and adapter weights of std 0.2 give branch
outputs several times larger than hbar, and a per-token logit bias U(-3, 3) spreads the gates over
about (0.05, 0.95).  `mutant_errors` measures, with the oracle alone, how far three plausible
kernel mistakes would move h under the contract's metric: a half-scale adapter output, a quarter
of the adapter's K range dropped, and the two branch scales swapped (g <-> 1 - g)."""
import numpy as np

from oracle import hero_oracle as O
from paper_2609_08189_amd import synth
from tests.oracle_inputs import adapter_of, dims_of, ffn_of
from tests.parity import row_rel_err

# the Llama shapes scaled down to keep the oracle quick, at token counts whose FFN products take
# the launch configurations the benchmark times: 256-row tiles at 8192 tokens (as the 8B stack's
# ~20k FFN rows do) and the persistent 192-row gate/up kernel at 4096 tokens (as the 8B layer does)
CONTRAST = synth.Workload("contrast", "bf16", d=1024, d_ff=3584, d_r=64, L_R=32, d_m=128, T=8192,
                          mode="budget", budget=0.3882, layer_j=17, bias="spread", batch=4, seq=2048,
                          ffn_std=0.05, adapter_std=0.2)


def sample_rows(mask, n_each, seed):
    rng = np.random.default_rng(seed)
    rows = np.zeros(mask.shape[0], bool)
    f, a = np.nonzero(mask)[0], np.nonzero(~mask)[0]
    rows[rng.choice(f, min(n_each, f.size), replace=False)] = True
    rows[rng.choice(a, min(n_each, a.size), replace=False)] = True
    return rows


def mutant_errors(prob, ref, rows):
    """Row-relative error (the contract metric) that each planted mistake would leave in h on the
    sampled rows, against the correct oracle output `ref` (a LayerResult on the same rows)."""
    w = prob.w
    dims = dims_of(w)
    sel = np.nonzero(rows)[0]
    hbar = prob.hbar.f64[sel]
    F, A = ffn_of(prob.ffn[0]), adapter_of(prob.adapter[0])
    use_ffn = ref.use_ffn[sel]
    g = ref.gate[sel]
    u = O.ffn_input(hbar, F, dims)
    ffn_out = np.where(use_ffn[:, None], O.frozen_ffn(u, F), np.nan)
    ad_out = np.where(use_ffn[:, None], np.nan, O.adapter(u, A))
    good = O.round_io(O.routed_output(hbar, g, use_ffn, ffn_out, ad_out), dims.io_dtype)
    assert row_rel_err(good, ref.h[sel]) == 0.0      # the pieces reassemble the oracle's rows
    half = O.routed_output(hbar, g, use_ffn, ffn_out, 0.5 * ad_out)
    w1 = A.w1.copy()
    w1[:, : w.d // 4] = 0.0
    ad_cut = np.where(use_ffn[:, None], np.nan, O.adapter(u, O.AdapterParams(w1=w1, w2=A.w2)))
    cut = O.routed_output(hbar, g, use_ffn, ffn_out, ad_cut)
    swap = O.routed_output(hbar, 1.0 - g, use_ffn, ffn_out, ad_out)
    ad, ff = ~use_ffn, use_ffn
    return {"adapter_half_scale": row_rel_err(half[ad], good[ad]),
            "adapter_k_quarter_dropped": row_rel_err(cut[ad], good[ad]),
            "gate_swap_adapter_rows": row_rel_err(swap[ad], good[ad]),
            "gate_swap_ffn_rows": row_rel_err(swap[ff], good[ff])}
