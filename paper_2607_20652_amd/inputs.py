"""Seeded synthetic inputs for the DPB workloads.

This module holds no arithmetic of the method: it only names the workload
shapes and draws random activations / upstream gradients from fixed seeds, so
that the HIP path and the CPU oracle see the identical bits.

The paper measures on residual-stream activations of GPT-2-style models
trained on FineWeb-Edu (§3); those activations are not available, so these
seeded draws stand in for them, with the shapes of the workloads below.

Recipe (per workload with index c; the pt_* workloads use the per-level
shapes of the paper's Table 6, with d = 1024 or 2048 and Delta = 256):
  * x  ~ N(0, 1) drawn as float32 by NumPy PCG64(seed 1000 + c), row-major, then
    rounded to bfloat16 (round-to-nearest-even) for bf16 workloads;
  * the gpt2 workload scales round(0.05 T) tokens by 4 (exact in bf16), chosen
    by the first entries of a PCG64(seed 2000 + c) permutation of the T tokens;
  * upstream gradients g ~ N(0, 1) from PCG64(seed 3000 + c), same rounding;
  * the "dyadic" tiny variant draws integers in [-8, 8] (PCG64 seed 4000 + c),
    so every product and sum in the path is exact in fp32.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np
import torch


@dataclass(frozen=True)
class Workload:
    name: str
    index: int          # seed offset c
    d: int              # residual width
    n: int              # dictionary bits: N = 2^n features
    levels: int         # hierarchy levels, level 0 included
    branching: int      # children scored per active parent
    beam: int           # active features per level below the last
    k: int              # active features on the last level
    tokens: int         # T
    dtype: str          # "f32" or "bf16" activations
    # explicit per-level hierarchy (n_l, K_l), when it is not the even spacing
    # of the configuration terms (the paper's own Table 6 shapes)
    level_bits: tuple | None = None
    active: tuple | None = None

    def hierarchy(self):
        """(level_bits, branching per level with [0] = 0, active) when explicit, else None."""
        if self.level_bits is None:
            return None
        return list(self.level_bits), [0] + [self.branching] * (self.levels - 1), list(self.active)

    def plan_kwargs(self) -> dict:
        """Keyword arguments of the binding's Plan for this workload's hierarchy."""
        h = self.hierarchy()
        if h is None:
            return dict(n_bits=self.n, levels=self.levels, branching=self.branching, beam=self.beam, k=self.k)
        return dict(level_bits=h[0], branchings=h[1], active=h[2])


WORKLOADS = {
    "tiny": Workload("tiny", 0, 64, 12, 3, 16, 4, 8, 256, "f32"),
    "gpt2": Workload("gpt2", 1, 768, 16, 4, 16, 8, 32, 8192, "bf16"),
    "wide": Workload("wide", 2, 768, 20, 5, 16, 8, 64, 65536, "bf16"),
    "very_wide": Workload("very_wide", 3, 1024, 24, 6, 16, 16, 64, 16384, "bf16"),
    "train": Workload("train", 4, 768, 20, 5, 16, 8, 64, 65536, "bf16"),
    # Table 6 (App. G) hierarchies: 256 children scored per active parent
    "pt_small_2l": Workload("pt_small_2l", 5, 1024, 15, 2, 256, 16, 32, 16384, "bf16", (10, 15), (16, 32)),
    "pt_large_2l": Workload("pt_large_2l", 6, 2048, 15, 2, 256, 16, 32, 16384, "bf16", (11, 15), (16, 32)),
    "pt_small_3l": Workload("pt_small_3l", 7, 1024, 17, 3, 256, 16, 64, 16384, "bf16", (10, 15, 17), (16, 32, 64)),
}


def workload(name: str) -> Workload:
    return WORKLOADS[name]


def _round(a: np.ndarray, dtype: str) -> torch.Tensor:
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    if dtype == "bf16":
        return t.to(torch.bfloat16)
    return t


def activations(name: str, tokens: int | None = None) -> torch.Tensor:
    """x [T, d] on the CPU (float32 or bfloat16)."""
    w = WORKLOADS[name]
    T = w.tokens if tokens is None else tokens
    rng = np.random.Generator(np.random.PCG64(1000 + w.index))
    x = rng.standard_normal((T, w.d), dtype=np.float32)
    if name == "gpt2":
        perm = np.random.Generator(np.random.PCG64(2000 + w.index)).permutation(T)
        x[perm[: int(round(0.05 * T))]] *= 4.0
    return _round(x, w.dtype)


def upstream_grad(name: str, tokens: int | None = None) -> torch.Tensor:
    """g [T, d] on the CPU, same dtype as the activations."""
    w = WORKLOADS[name]
    T = w.tokens if tokens is None else tokens
    rng = np.random.Generator(np.random.PCG64(3000 + w.index))
    return _round(rng.standard_normal((T, w.d), dtype=np.float32), w.dtype)


def dyadic(d: int, tokens: int, seed: int = 4000) -> torch.Tensor:
    """Small integers in [-8, 8] as float32: every path result is exact."""
    rng = np.random.Generator(np.random.PCG64(seed))
    return torch.from_numpy(rng.integers(-8, 9, size=(tokens, d)).astype(np.float32))


def normal(shape, seed: int, dtype: str = "f32") -> torch.Tensor:
    """Generic seeded N(0, 1) draw for ad-hoc test shapes."""
    rng = np.random.Generator(np.random.PCG64(seed))
    return _round(rng.standard_normal(shape, dtype=np.float32), dtype)
