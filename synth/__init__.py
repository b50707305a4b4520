"""Seeded synthetic inputs shaped like the video and audio branches of a joint
audio-video diffusion transformer layer.

This module is shared by the tests, the benchmark and the oracle checks.  It
holds no arithmetic of the method itself: it only draws Q/K/V tensors, plants a
correlated region, rounds to the device dtype and states the integer budgets
(block count, keep count, protected count) that both the GPU path and the
oracle receive as plain integers.

The paper's own activations (Ovi, LTX-2.3) are not available; these tensors
stand in for them with the token counts of a 21-frame 30x52 latent (Ovi-like),
a 24-frame 32x64 latent (LTX-like) and a 21-frame 45x80 latent with a CFG batch
of two (long clip), and audio lengths of 512 or 1024 tokens.

Recipe (per workload, per seed; numpy PCG64 via ``default_rng(seed)``):

1. planted region: per batch item, either ``n_plant`` distinct full video
   blocks drawn with ``rng.choice(n_full_blocks, n_plant, replace=False)``, or
   (``moving_patch``) a 4x4 patch per latent frame that moves one row and two
   columns per frame from a random start ``(r0, c0)``;
2. shared vectors ``u[b, h, :] ~ N(0, 1)^d`` (float32);
3. ``Q_v, K_v, V_v, Q_a, K_a`` in that order, each filled slab by slab
   (b, h) with ``standard_normal((L, d), float32)``;
4. the tiny fp32 workload multiplies Q/K/V by ``1/sqrt(d)`` at this point;
5. plant: ``0.5 * u[b, h]`` is added to every row of ``Q_a`` and ``K_a`` and
   to the planted rows of ``Q_v`` and ``K_v``;
6. bf16 workloads are rounded to bf16 (round to nearest even) here, so the
   float32 arrays returned hold values that are exact in the device dtype and
   the device tensors and the oracle's float64 copies hold the same numbers.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, replace
from typing import Dict

import numpy as np

__all__ = [
    "Workload", "WORKLOADS", "budget", "make_inputs", "bf16_bits",
    "round_to_bf16", "sweep_workloads",
]


def budget(ratio: float, n: int) -> int:
    """Integer budget ceil(ratio * n) taken in a form that does not overshoot
    on binary rounding (0.07 * 100 evaluates to 7.000000000000001)."""
    return int(math.ceil(round(ratio * n, 9)))


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    H: int
    d: int
    frames: int
    rows: int
    cols: int
    L_a: int
    dtype: str          # "f32" or "bf16": the device storage type of Q/K/V/O
    block: int
    density: float      # sparse keep ratio kappa of non-protected query blocks
    rho: float          # protected ratio of blocks (ignored if k_prot_fixed set)
    plant: str          # "blocks" or "moving_patch"
    n_plant: int        # planted blocks per batch item ("blocks" only)
    prescale: bool      # multiply Q/K/V by 1/sqrt(d) before planting
    k_prot_fixed: int = -1
    seed: int = 0
    block_a: int = 64   # audio branch: tokens per block of its sparse pattern
    rho_a: float = 0.05  # audio branch: protected token ratio

    @property
    def L_v(self) -> int:
        return self.frames * self.rows * self.cols

    @property
    def n_b(self) -> int:
        return -(-self.L_v // self.block)

    @property
    def tail(self) -> int:
        """Length of the last video block (== block when L_v divides)."""
        return self.L_v - (self.n_b - 1) * self.block

    @property
    def k_keep(self) -> int:
        return budget(self.density, self.n_b)

    @property
    def k_prot(self) -> int:
        if self.k_prot_fixed >= 0:
            return self.k_prot_fixed
        return budget(self.rho, self.n_b)

    @property
    def n_b_a(self) -> int:
        return -(-self.L_a // self.block_a)

    @property
    def k_keep_a(self) -> int:
        """Audio key blocks kept per non-protected audio query block (the
        video keep ratio over the audio blocks)."""
        return budget(self.density, self.n_b_a)

    @property
    def k_tok_a(self) -> int:
        return budget(self.rho_a, self.L_a)

    @property
    def scale(self) -> float:
        """Softmax scale 1/sqrt(d), rounded to float32 so that the device
        and the oracle use the very same number."""
        return float(np.float32(1.0 / math.sqrt(self.d)))

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


WORKLOADS: Dict[str, Workload] = {
    "tiny_f32": Workload(
        name="tiny_f32", B=1, H=2, d=64, frames=8, rows=8, cols=16, L_a=128,
        dtype="f32", block=64, density=0.25, rho=0.0, plant="blocks",
        n_plant=4, prescale=True, k_prot_fixed=2),
    "ovi_bf16": Workload(
        name="ovi_bf16", B=1, H=24, d=128, frames=21, rows=30, cols=52,
        L_a=512, dtype="bf16", block=128, density=0.25, rho=0.05,
        plant="blocks", n_plant=16, prescale=False),
    "ltx_bf16": Workload(
        name="ltx_bf16", B=1, H=32, d=128, frames=24, rows=32, cols=64,
        L_a=1024, dtype="bf16", block=128, density=0.20, rho=0.05,
        plant="moving_patch", n_plant=0, prescale=False),
    "long_cfg_bf16": Workload(
        name="long_cfg_bf16", B=2, H=24, d=128, frames=21, rows=45, cols=80,
        L_a=1024, dtype="bf16", block=128, density=0.15, rho=0.05,
        plant="blocks", n_plant=37, prescale=False),
}


def sweep_workloads():
    """Density x protection sweep at the Ovi-like shape, seeds 0-2."""
    base = WORKLOADS["ovi_bf16"]
    out = []
    for density in (0.10, 0.25, 0.50, 1.00):
        for rho in (0.0, 0.05, 0.10):
            for seed in (0, 1, 2):
                out.append(base.with_(
                    name=f"ovi_sweep_k{int(round(density*100))}_p{int(round(rho*100))}_s{seed}",
                    density=density, rho=rho, seed=seed))
    return out


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bf16 (ties to even), returned as
    float32.  Inputs are finite."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = u + (np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1)))
    r &= np.uint32(0xFFFF0000)
    return r.view(np.float32)


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """Upper 16 bits of float32 values that are already exact bf16."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    return (u >> np.uint32(16)).astype(np.uint16)


def _planted_tokens(w: Workload, rng: np.random.Generator) -> np.ndarray:
    mask = np.zeros((w.B, w.L_v), dtype=bool)
    if w.plant == "blocks":
        n_full = w.L_v // w.block
        for b in range(w.B):
            if w.n_plant == 0:
                continue
            blocks = rng.choice(n_full, w.n_plant, replace=False)
            for c in blocks:
                mask[b, c * w.block:(c + 1) * w.block] = True
    elif w.plant == "moving_patch":
        for b in range(w.B):
            r0 = int(rng.integers(w.rows - 3))
            c0 = int(rng.integers(w.cols - 3))
            for f in range(w.frames):
                r = (r0 + f) % (w.rows - 3)
                c = (c0 + 2 * f) % (w.cols - 3)
                for dr in range(4):
                    base = f * w.rows * w.cols + (r + dr) * w.cols + c
                    mask[b, base:base + 4] = True
    else:
        raise ValueError(f"unknown plant kind {w.plant!r}")
    return mask


def make_inputs(w: Workload, seed: int | None = None, with_v: bool = True):
    """Draw the layer inputs of workload ``w``.

    Returns a dict with float32 arrays ``q_v, k_v, v_v`` of shape
    [B, H, L_v, d] and ``q_a, k_a`` of shape [B, H, L_a, d] (values exact in
    ``w.dtype``), the boolean ``planted`` [B, L_v] token mask and ``u``.
    """
    seed = w.seed if seed is None else seed
    rng = np.random.default_rng(seed)
    planted = _planted_tokens(w, rng)
    u = rng.standard_normal((w.B, w.H, w.d), dtype=np.float32)
    out = {"planted": planted, "u": u}
    names = [("q_v", w.L_v), ("k_v", w.L_v), ("v_v", w.L_v),
             ("q_a", w.L_a), ("k_a", w.L_a)]
    for name, L in names:
        arr = np.empty((w.B, w.H, L, w.d), dtype=np.float32)
        for b in range(w.B):
            for h in range(w.H):
                rng.standard_normal(dtype=np.float32, out=arr[b, h])
        if name == "v_v" and not with_v:
            arr = None
        out[name] = arr
    s = np.float32(1.0 / math.sqrt(w.d))
    for name in ("q_v", "k_v", "v_v", "q_a", "k_a"):
        if w.prescale and out[name] is not None:
            out[name] *= s
    half_u = np.float32(0.5) * u
    for b in range(w.B):
        rows = np.nonzero(planted[b])[0]
        for h in range(w.H):
            out["q_a"][b, h] += half_u[b, h]
            out["k_a"][b, h] += half_u[b, h]
            out["q_v"][b, h, rows] += half_u[b, h]
            out["k_v"][b, h, rows] += half_u[b, h]
    if w.dtype == "bf16":
        for name in ("q_v", "k_v", "v_v", "q_a", "k_a"):
            if out[name] is not None:
                out[name] = round_to_bf16(out[name]).reshape(out[name].shape)
    elif w.dtype != "f32":
        raise ValueError(f"unknown dtype {w.dtype!r}")
    return out


def make_audio_values(w: Workload, seed: int | None = None) -> np.ndarray:
    """V^a [B, H, L_a, d] for the audio branch's self-attention, standard
    normal from its own generator (seeded with (seed, 1)) so that the draws
    of ``make_inputs`` do not change; scaled and rounded like the other
    inputs of ``w``."""
    seed = w.seed if seed is None else seed
    rng = np.random.default_rng([seed, 1])
    arr = np.empty((w.B, w.H, w.L_a, w.d), dtype=np.float32)
    for b in range(w.B):
        for h in range(w.H):
            rng.standard_normal(dtype=np.float32, out=arr[b, h])
    if w.prescale:
        arr *= np.float32(1.0 / math.sqrt(w.d))
    if w.dtype == "bf16":
        arr = round_to_bf16(arr).reshape(arr.shape)
    return arr
