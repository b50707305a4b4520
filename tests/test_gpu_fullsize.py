"""GPU parity at the full workload sizes, in the launch configuration the
benchmark times.  Saliency, protected selection and every mask row are
compared in full; attention outputs on sampled query blocks (all protected
blocks of one head, the ragged tail block, the first block and random ones),
which the oracle evaluates one by one, plus finiteness of the whole output."""
import numpy as np
import pytest

import synth
from sa_parity import compare_layer, gpu_layer

pytestmark = pytest.mark.gpu

FULL = ["ovi_bf16", "ltx_bf16", "long_cfg_bf16"]


def sample_rows(g, w, n_random=16, seed=0):
    rng = np.random.default_rng(seed)
    rows = {(0, 0, int(r)) for r in np.nonzero(g["prot_flag"][0])[0]}
    for b in range(w.B):
        rows.add((b, w.H - 1, w.n_b - 1))
        rows.add((b, 0, 0))
    for _ in range(n_random):
        rows.add((int(rng.integers(w.B)), int(rng.integers(w.H)),
                  int(rng.integers(w.n_b))))
    return sorted(rows)


@pytest.mark.parametrize("name", FULL)
def test_fullsize_layer_parity(name):
    w = synth.WORKLOADS[name]
    print(f"case {name}: B={w.B} H={w.H} L_v={w.L_v} L_a={w.L_a} n_b={w.n_b} "
          f"k_keep={w.k_keep} k_prot={w.k_prot}", flush=True)
    x = synth.make_inputs(w)
    g = gpu_layer(x, w, w.k_keep, w.k_prot)
    print(f"{name}: gpu done", flush=True)
    rows = sample_rows(g, w)
    rep = compare_layer(x, w, g, w.k_keep, w.k_prot, rows=rows)
    print(name, rep, flush=True)


def test_sweep_cell_parity():
    """One cell of the density sweep away from the default budgets (10 %
    density, 10 % protection, seed 1), at the full Ovi-like size."""
    w = [s for s in synth.sweep_workloads()
         if s.name == "ovi_sweep_k10_p10_s1"][0]
    x = synth.make_inputs(w)
    g = gpu_layer(x, w, w.k_keep, w.k_prot)
    rep = compare_layer(x, w, g, w.k_keep, w.k_prot, rows=sample_rows(g, w, 8))
    print(w.name, rep, flush=True)
