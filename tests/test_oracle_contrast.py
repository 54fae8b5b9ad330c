"""The high-contrast parity workload discriminates branch-scale mistakes (CPU, oracle only):
each planted mistake moves h by at least five times the bf16 tolerance on the sampled rows."""
import numpy as np
import pytest

from paper_2609_08189_amd import synth
from tests.contrast import CONTRAST, mutant_errors, sample_rows
from tests.parity import TOL, oracle_layer


@pytest.mark.parametrize("d_r", [32, 128])
def test_contrast_margins_on_the_oracle(d_r):
    w = CONTRAST.replace(d_r=d_r, T=1024, batch=1, seq=1024)
    prob = synth.make_problem(w, seed=3)
    ref = oracle_layer(prob, w.layer_j)
    # the bias spreads the gates of both branches well away from 1/2
    g = ref.gate
    assert g.min() < 0.1 and g.max() > 0.9
    rows = sample_rows(ref.own_ffn, 24, seed=0)
    ref_rows = oracle_layer(prob, w.layer_j, forced_ffn=ref.own_ffn, rows=rows)
    errs = mutant_errors(prob, ref_rows, rows)
    print(errs)
    assert min(errs.values()) >= 5 * TOL["bf16"], errs
