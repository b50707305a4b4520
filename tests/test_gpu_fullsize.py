"""GPU parity at the full workload sizes, in the launch configuration the
benchmark times.  Saliency, protected selection and every mask row are
compared in full.  Attention: every row of O and lse of the Ovi-like layer;
at the LTX-like and long-clip sizes sampled query blocks (all protected
blocks of one head, the ragged tail block, the first block and random ones),
which the oracle evaluates one by one, plus finiteness of the whole output."""
import pytest

import synth
from sa_parity import compare_layer, gpu_layer, sample_rows

pytestmark = pytest.mark.gpu

FULL = ["ovi_bf16", "ltx_bf16", "long_cfg_bf16"]


@pytest.mark.parametrize("name", FULL)
def test_fullsize_layer_parity(name):
    w = synth.WORKLOADS[name]
    print(f"case {name}: B={w.B} H={w.H} L_v={w.L_v} L_a={w.L_a} n_b={w.n_b} "
          f"k_keep={w.k_keep} k_prot={w.k_prot}", flush=True)
    x = synth.make_inputs(w)
    g = gpu_layer(x, w, w.k_keep, w.k_prot)
    print(f"{name}: gpu done", flush=True)
    rows = None if name == "ovi_bf16" else sample_rows(g, w)
    rep = compare_layer(x, w, g, w.k_keep, w.k_prot, rows=rows)
    print(name, rep, flush=True)
