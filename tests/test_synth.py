"""Workload shapes, integer budgets and input rounding.  CPU only."""
import json
import os

import numpy as np

import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_budgets_match_hand_derived_table():
    g = json.load(open(os.path.join(GOLDEN, "budgets.json")))
    for name, row in g["workloads"].items():
        w = synth.WORKLOADS[name]
        assert (w.L_v, w.n_b, w.tail, w.k_keep, w.k_prot) == (
            row["L_v"], row["n_b"], row["tail"], row["k_keep"], row["k_prot"])
        pairs = (w.n_b - w.k_prot) * w.k_keep + w.k_prot * w.n_b
        assert pairs == row["computed_pairs_blocks"]
        assert w.n_b ** 2 == row["all_pairs_blocks"]
    hz = g["ceil_hazard"]
    assert hz["ratio"] * hz["n"] > hz["expected"]          # the hazard exists
    assert synth.budget(hz["ratio"], hz["n"]) == hz["expected"]
    sw = g["sweep_ovi_shape"]
    for dens, k in sw["k_keep"].items():
        assert synth.budget(float(dens), sw["n_b"]) == k
    for rho, k in sw["k_prot"].items():
        assert synth.budget(float(rho), sw["n_b"]) == k
    assert len(synth.sweep_workloads()) == 36


def test_bf16_rounding_is_nearest_even():
    vals = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -9,
                     -1.0 - 2 ** -8, 3.0e-3, 1.0 + 2 ** -8 + 2 ** -20],
                    dtype=np.float32)
    r = synth.round_to_bf16(vals)
    expect = [1.0, 1.0, 1.0 + 2 ** -6, 1.0, -1.0, None, 1.0 + 2 ** -7]
    for got, e in zip(r, expect):
        if e is not None:
            assert got == np.float32(e)
    # every result is exact in bf16 and within half a bf16 ulp
    bits = r.view(np.uint32)
    assert np.all(bits & 0xFFFF == 0)
    assert np.all(np.abs(r - vals) <= np.abs(vals) * 2 ** -8)


def test_inputs_are_seeded_and_exact_in_device_dtype():
    w = synth.WORKLOADS["tiny_f32"]
    a, b = synth.make_inputs(w), synth.make_inputs(w)
    for k in ("q_v", "k_v", "v_v", "q_a", "k_a"):
        assert np.array_equal(a[k], b[k])
        assert a[k].dtype == np.float32
    c = synth.make_inputs(w, seed=1)
    assert not np.array_equal(a["q_v"], c["q_v"])
    small = w.with_(name="t", dtype="bf16", frames=2)
    x = synth.make_inputs(small)
    assert np.all(x["q_v"].view(np.uint32) & 0xFFFF == 0)
    bits = synth.bf16_bits(x["q_v"])
    back = (bits.astype(np.uint32) << 16).view(np.float32)
    assert np.array_equal(back, x["q_v"])


def test_planted_regions():
    w = synth.WORKLOADS["tiny_f32"]
    x = synth.make_inputs(w)
    per_block = x["planted"][0].reshape(w.n_b, w.block)
    assert np.all(per_block.all(1) | ~per_block.any(1))     # whole blocks
    assert per_block.all(1).sum() == w.n_plant
    ltx = synth.WORKLOADS["ltx_bf16"].with_(H=1, frames=3)
    rng_mask = synth._planted_tokens(ltx, np.random.default_rng(0))
    assert rng_mask.sum() == 16 * 3
