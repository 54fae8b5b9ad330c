"""GPU parity of hero_routed_layer against the CPU oracle over a seeded random sweep of the shapes
the library accepts: model and FFN widths, adapter ranks (register-tiled and wide), memory widths,
the router's sub-network widths (d_h + d_a = d_s, d_e, d_p, d_head), layer index, token count
(ragged, down to one), budget or threshold routing, and S stored in fp32 or bf16.

The cases are drawn once on the host from a fixed seed, so the list is the same on every run; each
is printed before it runs."""
import numpy as np
import pytest

from paper_2609_08189_amd import synth
from tests.test_gpu_layer import _run


def _cases(n_bf16=10, n_f32=4, seed=20260):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n_bf16 + n_f32):
        bf16 = i < n_bf16
        if bf16:
            d = int(rng.choice([256, 512, 768, 1024, 1280]))
            d_ff = 128 * int(rng.integers(2, 25))
            d_r = int(rng.choice([32, 64, 96, 128, 256, 384]))
            d_e = int(rng.choice([64, 128, 192, 256]))
            d_head = int(rng.choice([x for x in (64, 128, 192, 256) if (d_e + x) % 128 == 0]))
            d_s = 8 * int(rng.integers(1, 17))
        else:
            d = int(rng.choice([128, 256, 384]))
            d_ff = int(rng.integers(40, 700))
            d_r = int(rng.integers(4, 80))
            d_e = int(rng.integers(8, 257))
            d_head = int(rng.integers(8, 257))
            d_s = int(rng.integers(2, 129))
        d_h = int(rng.integers(1, d_s))
        d_m = int(rng.choice([32, 64, 128, 256]))
        L_R = int(rng.integers(2, 13))
        j = int(rng.integers(1, L_R + 1))
        T = int(rng.integers(1, 1201)) if i % 3 else int(rng.integers(1, 40))
        if i in (n_bf16 - 1, n_bf16 + n_f32 - 1):
            T = 1                                   # one token per dtype
        mode = "budget" if rng.uniform() < 0.6 else "threshold"
        state = "bf16" if (d_m >= 64 and rng.uniform() < 0.3) else "f32"
        w = synth.Workload(f"sweep{i}", "bf16" if bf16 else "f32", d=d, d_ff=d_ff, d_r=d_r, L_R=L_R, d_m=d_m,
                           T=T, mode=mode, budget=float(rng.uniform()) if mode == "budget" else 0.0,
                           tau=float(rng.choice([0.45, 0.5, 0.55])), d_s=d_s, d_h=d_h, d_a=d_s - d_h, d_e=d_e,
                           d_p=int(rng.integers(4, 129)), d_head=d_head, state_dtype=state)
        out.append((w, j, int(rng.integers(0, 1 << 16))))
    return out


CASES = _cases()


def test_sweep_cases_are_valid_shapes():
    """Every drawn case passes the library's host checks (no GPU work), and the sweep reaches
    both dtypes, both routing modes, both state storages, wide adapter ranks and one-token calls."""
    from paper_2609_08189_amd import hero as H
    from paper_2609_08189_amd.device import dims_struct
    for w, j, _ in CASES:
        assert H.hero_workspace_size(dims_struct(w), w.T, False) > 0, w
        assert 1 <= j <= w.L_R
    assert {w.dtype for w, _, _ in CASES} == {"bf16", "f32"}
    assert {w.mode for w, _, _ in CASES} == {"budget", "threshold"}
    assert {w.state_dtype for w, _, _ in CASES} == {"f32", "bf16"}
    assert any(w.d_r > 128 for w, _, _ in CASES if w.dtype == "bf16")
    assert {w.dtype for w, _, _ in CASES if w.T == 1} == {"bf16", "f32"}


@pytest.mark.gpu
@pytest.mark.parametrize("k", range(len(CASES)))
def test_layer_sweep(k):
    w, j, seed = CASES[k]
    print(f"sweep case {k}: d_s={w.d_s} d_h={w.d_h} d_e={w.d_e} d_p={w.d_p} d_head={w.d_head} "
          f"d_r={w.d_r} L_R={w.L_R} state={w.state_dtype} budget={w.budget:.3f} tau={w.tau}", flush=True)
    _run(w, j, seed=seed)


def _bwd_cases(n_bf16=7, n_f32=3, seed=20261):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n_bf16 + n_f32):
        bf16 = i < n_bf16
        if bf16:
            d = int(rng.choice([256, 512, 768, 1024, 1280]))
            d_ff = 128 * int(rng.integers(2, 25))
            d_r = int(rng.choice([32, 64, 96, 128, 256, 384]))
        else:
            d = int(rng.choice([128, 256, 384]))
            d_ff = int(rng.integers(40, 700))
            d_r = int(rng.integers(4, 80))
        T = 1 if i in (0, n_bf16) else int(rng.integers(2, 1500))
        w = synth.Workload(f"bwd_sweep{i}", "bf16" if bf16 else "f32", d=d, d_ff=d_ff, d_r=d_r, L_R=4,
                           d_m=64, T=T, mode="budget", budget=float(rng.uniform()))
        out.append((w, int(rng.integers(0, 1 << 16)), bool(rng.uniform() < 0.5), bool(rng.uniform() < 0.5)))
    return out


BWD_CASES = _bwd_cases()


def test_backward_sweep_cases_are_valid_shapes():
    from paper_2609_08189_amd import hero as H
    from paper_2609_08189_amd.device import dims_struct
    import ctypes
    for w, _, _, _ in BWD_CASES:
        out = ctypes.c_size_t(0)
        assert H.lib().hero_backward_workspace_size(ctypes.byref(dims_struct(w)), w.T,
                                                    ctypes.byref(out)) == H.HERO_OK, w
    assert {w.dtype for w, *_ in BWD_CASES} == {"bf16", "f32"}
    assert any(bm for *_, bm in BWD_CASES) and not all(bm for *_, bm in BWD_CASES)


@pytest.mark.gpu
@pytest.mark.parametrize("k", range(len(BWD_CASES)))
def test_block_backward_sweep(k):
    from tests.test_gpu_backward import _run_small
    w, seed, gin, bm = BWD_CASES[k]
    print(f"backward sweep case {k}", flush=True)
    _run_small(w, seed, dgate_in=gin, budget_mode=bm)


def _rbwd_cases(n_bf16=6, n_f32=4, seed=20262):
    """Router backward over drawn router shapes (sub-network widths, memory width, layer index,
    token count), fp32 state storage (the only one the backward accepts)."""
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n_bf16 + n_f32):
        bf16 = i < n_bf16
        if bf16:
            d = int(rng.choice([256, 512, 768, 1024]))
            d_e = int(rng.choice([64, 128, 192, 256]))
            d_head = int(rng.choice([x for x in (64, 128, 192, 256) if (d_e + x) % 128 == 0]))
            d_s = 8 * int(rng.integers(1, 17))
        else:
            d = int(rng.choice([128, 256, 384]))
            d_e = int(rng.integers(8, 257))
            d_head = int(rng.integers(8, 257))
            d_s = int(rng.integers(2, 129))
        d_h = int(rng.integers(1, d_s))
        d_m = (32, 64, 128, 256)[i % 4]
        L_R = int(rng.integers(2, 13))
        j = int(rng.integers(1, L_R + 1)) if i % 2 else int(rng.integers(2, L_R + 1))
        T = int(rng.integers(1, 600 if d_m < 256 else 160))
        w = synth.Workload(f"rbwd_sweep{i}", "bf16" if bf16 else "f32", d=d, d_ff=256, d_r=32, L_R=L_R, d_m=d_m,
                           T=T, mode="budget", budget=float(rng.uniform()), d_s=d_s, d_h=d_h, d_a=d_s - d_h,
                           d_e=d_e, d_p=int(rng.integers(4, 129)), d_head=d_head)
        out.append((w, j, int(rng.integers(0, 1 << 16))))
    return out


RBWD_CASES = _rbwd_cases()


def test_router_backward_sweep_cases_are_valid_shapes():
    import ctypes
    from paper_2609_08189_amd import hero as H
    from paper_2609_08189_amd.device import dims_struct
    for w, j, _ in RBWD_CASES:
        out = ctypes.c_size_t(0)
        assert H.lib().hero_router_backward_workspace_size(ctypes.byref(dims_struct(w)), w.T,
                                                           ctypes.byref(out)) == H.HERO_OK, w
        assert 1 <= j <= w.L_R
    assert {w.dtype for w, _, _ in RBWD_CASES} == {"bf16", "f32"}
    assert {w.d_m for w, _, _ in RBWD_CASES} >= {32, 64, 128}
    assert sum(j >= 3 for _, j, _ in RBWD_CASES) >= 4


@pytest.mark.gpu
@pytest.mark.parametrize("k", range(len(RBWD_CASES)))
def test_router_backward_sweep(k):
    from tests.test_gpu_router_backward import _run as _run_rbwd
    w, j, seed = RBWD_CASES[k]
    print(f"router backward sweep case {k}: d_s={w.d_s} d_h={w.d_h} d_e={w.d_e} d_p={w.d_p} "
          f"d_head={w.d_head} L_R={w.L_R}", flush=True)
    _run_rbwd(w, j, seed=seed)
