"""Seeded synthetic Q/K/V shaped like the paper's attention workloads.

This module only draws random inputs; it holds none of the approximation's
arithmetic, so both the kernels' tests and the float64 checker can take their
inputs from it.

Shapes follow the paper's model settings (head dim 64 for every model,
12 heads for RoBERTa-base at 512 and 4096 tokens, Tab. 8); the paper's own
inputs come from pretrained models that are not available, so every value
here is synthetic.

Generation recipe (all in float64, then rounded once to the compute dtype):

* ``iid``:   Q, K, V ~ N(0, 1) i.i.d., each scaled by 1/sqrt(d).
* ``ar1``:   Q and K are independent AR(1) sequences along the token axis,
             ``x_0 ~ N(0, s2/(1-rho^2))``, ``x_t = rho*x_{t-1} + e_t``,
             ``e_t ~ N(0, s2)`` per feature; V ~ N(0, 1) i.i.d.
* ``hub``:   Q, K, V ~ N(0, 1) i.i.d.; then, per sequence, a direction
             ``u = 4 g/|g|`` (g ~ N(0, I_d)) shared by all heads is added to
             K at ``round(0.05 n)`` token positions drawn without replacement.

Draw order: Q, K, V (standard normals in C order over [B, H, n, d]), then the
hub directions and positions. The generator is numpy's PCG64 seeded with
``SEED_BASE + workload index``.
"""
from __future__ import annotations

import dataclasses
import numpy as np
from scipy.signal import lfilter

SEED_BASE = 220710284


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    index: int          # 1-based position in WORKLOADS; the seed offset
    B: int
    H: int
    n: int
    d: int
    dtype: str          # "f32" or "bf16"
    budget: int         # selected 32x32 blocks per block-row
    kind: str           # "iid", "ar1" or "hub"
    rho: float = 0.0
    s2: float = 1.0
    block: int = 32

    @property
    def nb(self) -> int:
        return self.n // self.block

    @property
    def seed(self) -> int:
        return SEED_BASE + self.index


WORKLOADS = {
    w.name: w for w in [
        # one head, i.i.d. inputs: the small case the checker runs in full
        Workload("tiny-512", 1, B=1, H=1, n=512, d=64, dtype="f32", budget=4, kind="iid"),
        # RoBERTa-base encoder layer at 512 tokens (12 heads, head dim 64)
        Workload("base-512", 2, B=32, H=12, n=512, d=64, dtype="bf16", budget=8, kind="ar1", rho=0.9, s2=1.0),
        # small long-sequence classifier layer with heavy key columns
        Workload("small-4096", 3, B=16, H=2, n=4096, d=32, dtype="f32", budget=8, kind="hub"),
        # RoBERTa-base encoder layer at 4096 tokens: the throughput workload
        Workload("base-4096", 4, B=8, H=12, n=4096, d=64, dtype="bf16", budget=16, kind="ar1", rho=0.95, s2=1.0),
        # 32k-token sequence, 16 heads of dim 128
        Workload("long-32768", 5, B=1, H=16, n=32768, d=128, dtype="bf16", budget=32, kind="ar1", rho=0.98, s2=0.5),
    ]
}

BENCH_WORKLOAD = "base-4096"


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round float64 values to the nearest bfloat16 (ties to even), returned
    as float32 (every bfloat16 value is exactly a float32).

    Rounds straight from float64 so there is no double rounding through
    float32. Values must be finite and inside float32's normal range.
    """
    x = np.ascontiguousarray(x, dtype=np.float64)
    bits = x.view(np.uint64)
    # bfloat16 keeps 7 of float64's 52 fraction bits: drop the low 45.
    lsb = (bits >> np.uint64(45)) & np.uint64(1)
    rounded = (bits + np.uint64((1 << 44) - 1) + lsb) & ~np.uint64((1 << 45) - 1)
    out = rounded.view(np.float64).astype(np.float32)
    return out


def bf16_bits(x32: np.ndarray) -> np.ndarray:
    """uint16 bit patterns of float32 values that are exact bfloat16 values."""
    u = np.ascontiguousarray(x32, dtype=np.float32).view(np.uint32)
    if np.any(u & np.uint32(0xFFFF)):
        raise ValueError("values are not exactly representable in bfloat16")
    return (u >> np.uint32(16)).astype(np.uint16)


def _ar1(rng: np.random.Generator, shape, rho: float, s2: float) -> np.ndarray:
    e = rng.standard_normal(shape) * np.sqrt(s2)
    e[:, :, 0, :] /= np.sqrt(1.0 - rho * rho)      # stationary start
    return lfilter([1.0], [1.0, -rho], e, axis=2)


def make_qkv(w: Workload, B=None, H=None, n=None, meta=None):
    """Draw (q, k, v) for workload ``w`` as float32 arrays [B, H, n, d] whose
    values are exactly representable in ``w.dtype``. B, H, n may be overridden
    to draw smaller instances with the same recipe. If ``meta`` is a dict, the
    hub directions and positions of a ``hub`` workload are stored in it."""
    B = w.B if B is None else B
    H = w.H if H is None else H
    n = w.n if n is None else n
    d = w.d
    shape = (B, H, n, d)
    rng = np.random.Generator(np.random.PCG64(w.seed))
    if w.kind == "iid":
        s = 1.0 / np.sqrt(d)
        q = rng.standard_normal(shape) * s
        k = rng.standard_normal(shape) * s
        v = rng.standard_normal(shape) * s
    elif w.kind == "ar1":
        q = _ar1(rng, shape, w.rho, w.s2)
        k = _ar1(rng, shape, w.rho, w.s2)
        v = rng.standard_normal(shape)
    elif w.kind == "hub":
        q = rng.standard_normal(shape)
        k = rng.standard_normal(shape)
        v = rng.standard_normal(shape)
        n_hub = int(round(0.05 * n))
        for b in range(B):
            g = rng.standard_normal(d)
            u = 4.0 * g / np.linalg.norm(g)
            pos = rng.choice(n, size=n_hub, replace=False)
            k[b, :, pos, :] += u
            if meta is not None:
                meta.setdefault("hubs", []).append((u, np.sort(pos)))
    else:
        raise ValueError(f"unknown input kind {w.kind!r}")
    cast = round_to_bf16 if w.dtype == "bf16" else (lambda a: a.astype(np.float32))
    return cast(q), cast(k), cast(v)


def random_qkv(seed: int, B: int, H: int, n: int, d: int, dtype: str = "f32", scale: float = 1.0):
    """Plain i.i.d. N(0, scale^2) inputs for edge-case tests."""
    rng = np.random.Generator(np.random.PCG64(seed))
    shape = (B, H, n, d)
    arrs = [rng.standard_normal(shape) * scale for _ in range(3)]
    cast = round_to_bf16 if dtype == "bf16" else (lambda a: a.astype(np.float32))
    return tuple(cast(a) for a in arrs)

# Three-resolution settings R = {coarse_block, 32, 1} per workload:
# (coarse_block, first-level budget per coarse block-row). The second-level
# budget is the workload's own; first-level budgets leave at least twice as
# many candidate 32-blocks as that budget.
MULTILEVEL = {
    "tiny-512": (64, 3),
    "base-512": (64, 8),
    "small-4096": (128, 4),
    "base-4096": (128, 8),
    "long-32768": (256, 8),
}

# Four resolutions R = {s_0, s_1, 32, 1} per workload: (scales, budgets per level).
LEVELS = {
    "tiny-512": ((256, 64, 32), (1, 3, 4)),
    "base-512": ((256, 64, 32), (2, 6, 8)),
    "small-4096": ((1024, 128, 32), (2, 6, 8)),
    "base-4096": ((512, 128, 32), (3, 8, 16)),
    "long-32768": ((2048, 256, 32), (4, 12, 32)),
}
