"""Seeded synthetic inputs for the INT4 attention path (no method arithmetic here).

The paper measures on Wan2.2 and HunyuanVideo attention activations (Sec. 5.1);
neither the models nor their prompts are available, so every input is drawn
from a seeded generator with the shapes of those workloads and the outlier
structure the paper reports for 3D-RoPE video DiTs (Sec. 3.1: outliers sit in
the RoPE segments, concentrated in the low-frequency pairs, at the same
channels of Q and K).

Arrays are bf16 *bit patterns* (uint16), layout [B, H, N, D], produced by
round-to-nearest-even from binary32 draws.  Both the CPU oracle and the GPU
library consume these same bits.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

D = 128


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    H: int
    T: int
    Hg: int
    W: int
    split: tuple = (44, 42, 42)
    theta: float = 10000.0
    seed: int = 0
    dist: str = "lowfreq"          # "c1" | "lowfreq" | "student_lowfreq"
    desc: str = ""

    @property
    def N(self) -> int:
        return self.T * self.Hg * self.W

    @property
    def shape(self) -> tuple:
        return (self.B, self.H, self.N, D)

    def ops(self) -> float:
        """Effective attention operation count 4*B*H*N^2*d."""
        return 4.0 * self.B * self.H * float(self.N) ** 2 * D


WORKLOADS = {
    "c1": Workload("c1", 1, 2, 4, 16, 16, seed=1, dist="c1",
                   desc="tiny oracle case, grid 4x16x16, 8 outlier channels x20"),
    "c2": Workload("c2", 1, 12, 21, 30, 52, seed=2, dist="lowfreq",
                   desc="Wan2.2-480P-like layer, grid 21x30x52 (N=32760), 12 heads"),
    "c3": Workload("c3", 1, 40, 21, 45, 80, seed=3, dist="lowfreq",
                   desc="large layer, grid 21x45x80 (N=75600), 40 heads"),
    "c4": Workload("c4", 1, 24, 33, 45, 80, split=(16, 56, 56), theta=256.0, seed=4, dist="student_lowfreq",
                   desc="HunyuanVideo-like split 16/56/56 theta=256, grid 33x45x80 (N=118800)"),
}

# Mixed-precision schedule (40 DiT blocks x 10 denoising steps at c2's shape).
SCHEDULE = dict(steps=10, blocks=40, fallback_steps=(0, 1), mask_frac=0.15, mask_seed=5, input_sets=3)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round-to-nearest-even binary32 -> bf16 bit patterns (uint16)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    t = np.right_shift(u, 16)
    np.bitwise_and(t, np.uint32(1), out=t)
    t += np.uint32(0x7FFF)
    t += u
    np.right_shift(t, 16, out=t)
    r = t.astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        r[nan] = (np.right_shift(u[nan], 16) | 0x40).astype(np.uint16)
    return r


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def lowfreq_pairs(split) -> list:
    """Indices of the two lowest-frequency channel pairs of each RoPE segment
    (the last pairs of each segment, whose angle advances slowest)."""
    pairs, first = [], 0
    for Da in split:
        npair = Da // 2
        pairs += [first + npair - 2, first + npair - 1]
        first += npair
    return pairs


def outlier_plan(w: Workload, rng: np.random.Generator):
    """Per head: list of (channel pair, multiplier), shared by Q and K."""
    plans = []
    for _ in range(w.B * w.H):
        if w.dist == "c1":
            pairs = sorted(rng.choice(D // 2, size=4, replace=False).tolist())
            plans.append([(p, 20.0) for p in pairs])
        else:
            pairs = lowfreq_pairs(w.split)
            mult = rng.uniform(10.0, 30.0, size=len(pairs))
            plans.append(list(zip(pairs, mult.tolist())))
    return plans


def _draw(w: Workload, rng: np.random.Generator, heavy: bool) -> np.ndarray:
    shape = (w.B * w.H, w.N, D)
    if heavy:
        return rng.standard_t(3.0, size=shape).astype(np.float32)
    return rng.standard_normal(size=shape, dtype=np.float32)


def make_inputs(w: Workload, seed: int | None = None):
    """Return (q, k, v) bf16 bits [B, H, N, D] for workload ``w``."""
    ss = np.random.SeedSequence(w.seed if seed is None else seed)
    sq, sk, sv, so = [np.random.default_rng(s) for s in ss.spawn(4)]
    heavy = w.dist == "student_lowfreq"
    plans = outlier_plan(w, so)
    out = []
    for rng, is_qk in ((sq, True), (sk, True), (sv, False)):
        x = _draw(w, rng, heavy and is_qk)
        if is_qk:
            for bh, plan in enumerate(plans):
                for p, m in plan:
                    x[bh, :, 2 * p:2 * p + 2] *= np.float32(m)
        out.append(f32_to_bf16_bits(x).reshape(w.shape))
    return tuple(out)


def schedule_mask(seed: int = SCHEDULE["mask_seed"], steps: int = SCHEDULE["steps"], blocks: int = SCHEDULE["blocks"],
                  fallback_steps=SCHEDULE["fallback_steps"], mask_frac: float = SCHEDULE["mask_frac"]) -> np.ndarray:
    """bool [steps, blocks]: True where the BF16 fallback runs (first steps plus
    a seeded set of accuracy-sensitive blocks)."""
    rng = np.random.default_rng(seed)
    nmask = int(round(mask_frac * blocks))
    blk = np.zeros(blocks, bool)
    blk[rng.choice(blocks, size=nmask, replace=False)] = True
    m = np.repeat(blk[None, :], steps, axis=0)
    for s in fallback_steps:
        m[s, :] = True
    return m


def small_workload(name: str, T: int, Hg: int, W: int, H: int = 1, split=(44, 42, 42), theta=10000.0,
                   seed: int = 11, dist: str = "lowfreq", B: int = 1) -> Workload:
    """Ad-hoc small geometry for parity cases (ragged N, few heads, batch)."""
    return Workload(name, B, H, T, Hg, W, split=tuple(split), theta=theta, seed=seed, dist=dist)
