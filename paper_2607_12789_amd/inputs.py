"""Seeded synthetic inputs for the AVQ-Attention forward pass.

This module only draws random tensors; it holds none of the method's
arithmetic. The same tensors feed the HIP path and the fp64 oracle.

Workload recipe (one generator, NumPy PCG64, fp64 draws, fixed draw order):

1. Parent codebook ``Cp[H, M0, d] ~ N(0, I)``.
2. Child offsets ``eps[H, M0, Ch, d] ~ sigma_c * N(0, I)``, centred over the
   children of each parent so that the parent is the mean of its children
   (the parent-child constraint of Sec. 4.1; the App. A projection with equal
   masses). ``Cc = Cp[:, :, None] + eps``.
3. Keys, per ``(b, h)`` in row-major order: pick one child component per key
   (uniformly, or from Dirichlet(alpha) weights over the ``M0*Ch`` children
   drawn per ``(b, h)``), then ``K = Cc[h, comp] + sigma_k * N(0, I)``.
4. Queries ``Q = (q_scale / sqrt(d)) * N(0, I)``.
5. Values ``V ~ N(0, 1)``.
6. Every tensor is rounded to the storage dtype (fp64 -> fp32 -> bf16, each
   step round-to-nearest-even). Both sides receive the same rounded tensors.

A flat codebook (``Ch = 0``) skips step 2 (``Cc`` is ``[H, M0, 0, d]``) and
draws the key components over the parents in step 3.

The paper's own workloads (keys of trained ViT-B / DPT-L models, Sec. 5)
are not available; these Gaussian-mixture keys stand in for them.
"""
from __future__ import annotations

import dataclasses
import math
from dataclasses import dataclass
from typing import Optional

import numpy as np
import torch


@dataclass(frozen=True)
class Workload:
    """Shape, method hyper-parameters and generator knobs of one workload."""

    name: str
    B: int
    H: int
    N: int
    d: int
    M0: int
    Ch: int
    P: int
    block_q: int
    dtype: str = "bf16"  # "f32" or "bf16"
    sigma_c: float = 0.1
    sigma_k: float = 0.05
    q_scale: float = 2.0  # queries are N(0, I) * q_scale / sqrt(d)
    dirichlet_alpha: Optional[float] = None  # None: uniform child choice
    seed: int = 0

    @property
    def Mtot(self) -> int:
        return self.M0 * (1 + self.Ch)

    @property
    def n_tiles(self) -> int:
        return (self.N + self.block_q - 1) // self.block_q

    @property
    def torch_dtype(self) -> torch.dtype:
        return {"f32": torch.float32, "bf16": torch.bfloat16}[self.dtype]

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)

    def describe(self) -> str:
        unit = "children" if self.Ch > 0 else "parents (flat codebook)"
        mix = (f"uniform {unit}" if self.dirichlet_alpha is None
               else f"Dirichlet({self.dirichlet_alpha}) {unit}")
        return (f"B={self.B} H={self.H} N={self.N} d={self.d} {self.dtype} "
                f"M0={self.M0} Ch={self.Ch} P={self.P} Bq={self.block_q}; "
                f"keys: {mix}, sigma_c={self.sigma_c}, sigma_k={self.sigma_k}; "
                f"Q scale {self.q_scale}/sqrt(d); seed {self.seed}")


# The five evaluation workloads: sizes, codebook shape, P and query block as
# stated for this path; the first one is small enough for the oracle to run in
# seconds, the fourth (N=16384) is the throughput workload.
WORKLOADS = {
    "c1": Workload("c1", B=1, H=1, N=1024, d=64, M0=32, Ch=4, P=4, block_q=64,
                   dtype="f32"),
    "c2": Workload("c2", B=4, H=8, N=4096, d=64, M0=128, Ch=4, P=16, block_q=128),
    "c3": Workload("c3", B=8, H=12, N=4096, d=64, M0=256, Ch=8, P=32, block_q=128,
                   dirichlet_alpha=0.5),
    "c4": Workload("c4", B=2, H=16, N=16384, d=128, M0=256, Ch=8, P=32, block_q=128,
                   q_scale=6.0),
    "c5": Workload("c5", B=1, H=16, N=65536, d=128, M0=512, Ch=8, P=64, block_q=256,
                   dirichlet_alpha=0.3),
}

# The sequence-length sweep of the scaling analysis (Sec. 5, scaling table):
# B=4, H=12, d=64, N in {1k, 4k, 16k, 64k}; flat codebooks of M = 256 and 512
# codewords (P = 0) and tree codebooks M0/P/Ch = 64/8/8, 64/16/8, 128/8/8,
# 128/16/8. The query block is not given there; 128 is used throughout.
SCALING_N = (1024, 4096, 16384, 65536)
SCALING_CODEBOOKS = (("vq256", 256, 0, 0), ("vq512", 512, 0, 0), ("avq64/8/8", 64, 8, 8),
                     ("avq64/16/8", 64, 8, 16), ("avq128/8/8", 128, 8, 8),
                     ("avq128/16/8", 128, 8, 16))


def scaling_workloads(ns=SCALING_N):
    """The sweep's workloads, codebook-major (name, M0, Ch, P per codebook)."""
    return [Workload(f"{name}@N={n}", B=4, H=12, N=n, d=64, M0=M0, Ch=Ch, P=P, block_q=128)
            for name, M0, Ch, P in SCALING_CODEBOOKS for n in ns]


def _round(x: np.ndarray, dtype: str) -> torch.Tensor:
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float64)).to(torch.float32)
    if dtype == "bf16":
        t = t.to(torch.bfloat16)
    elif dtype != "f32":
        raise ValueError(f"unknown dtype {dtype}")
    return t.contiguous()


def generate(w: Workload) -> dict:
    """Draw ``Q, K, V, Cp, Cc`` for workload ``w`` as CPU tensors of ``w.dtype``.

    Shapes: ``Q, K, V: [B, H, N, d]``, ``Cp: [H, M0, d]``, ``Cc: [H, M0, Ch, d]``.
    """
    rng = np.random.default_rng(w.seed)
    B, H, N, d, M0, Ch = w.B, w.H, w.N, w.d, w.M0, w.Ch
    cp = rng.standard_normal((H, M0, d))
    if Ch > 0:
        eps = w.sigma_c * rng.standard_normal((H, M0, Ch, d))
        eps -= eps.mean(axis=2, keepdims=True)
        cc = cp[:, :, None, :] + eps
        comps = cc.reshape(H, M0 * Ch, d)
    else:  # flat codebook: keys around the parents
        cc = np.zeros((H, M0, 0, d))
        comps = cp
    n_comp = comps.shape[1]
    k = np.empty((B, H, N, d))
    for b in range(B):
        for h in range(H):
            if w.dirichlet_alpha is None:
                comp = rng.integers(0, n_comp, size=N)
            else:
                pi = rng.dirichlet(np.full(n_comp, w.dirichlet_alpha))
                comp = rng.choice(n_comp, size=N, p=pi)
            k[b, h] = comps[h, comp] + w.sigma_k * rng.standard_normal((N, d))
    q = (w.q_scale / math.sqrt(d)) * rng.standard_normal((B, H, N, d))
    v = rng.standard_normal((B, H, N, d))
    return {
        "Q": _round(q, w.dtype),
        "K": _round(k, w.dtype),
        "V": _round(v, w.dtype),
        "Cp": _round(cp, w.dtype),
        "Cc": _round(cc, w.dtype),
    }


def dyadic_exact(B: int, H: int, N: int, d: int, M0: int, Ch: int, seed: int = 0,
                 dtype: str = "bf16") -> dict:
    """Inputs on a coarse dyadic grid, exact in bf16, fp32 and fp64.

    Parents have entries ``k/4`` with ``|k| <= 8``; each parent's child offsets
    are ``+-1/8`` patterns that sum to zero over the children exactly, so the
    parent-child constraint holds exactly after rounding. Keys are children or
    parents plus ``+-1/16`` noise; queries are multiples of ``1/16`` in
    ``[-1/2, 1/2]``; values are multiples of ``1/8`` in ``[-2, 2]``. With few
    significant bits every dot product and squared distance is exact in fp32,
    so exact ties stay exact ties on both sides.
    """
    if Ch % 2 != 0:
        raise ValueError("dyadic_exact needs an even number of children")
    rng = np.random.default_rng(seed)
    cp = rng.integers(-8, 9, size=(H, M0, d)) / 4.0
    half = rng.choice([-1.0, 1.0], size=(H, M0, Ch // 2, d)) / 8.0
    eps = np.concatenate([half, -half], axis=2)
    cc = cp[:, :, None, :] + eps
    cand = np.concatenate([cc.reshape(H, M0 * Ch, d), cp], axis=1)
    k = np.empty((B, H, N, d))
    for b in range(B):
        for h in range(H):
            comp = rng.integers(0, cand.shape[1], size=N)
            k[b, h] = cand[h, comp] + rng.integers(-1, 2, size=(N, d)) / 16.0
    q = rng.integers(-8, 9, size=(B, H, N, d)) / 16.0
    v = rng.integers(-16, 17, size=(B, H, N, d)) / 8.0
    return {"Q": _round(q, dtype), "K": _round(k, dtype), "V": _round(v, dtype),
            "Cp": _round(cp, dtype), "Cc": _round(cc, dtype)}


def spatial(w: Workload, width: int, height: int, regions: int = 48,
            comps_per_region: int = 4) -> dict:
    """Tokens on a width x height grid (token y*width + x, N = width*height)
    whose keys and queries depend on where they lie, the 2-D structure of
    image tokens that makes per-tile refinement adaptive (Sec. 4,
    Fig. per-tile adaptivity).

    Draw order (one PCG64 generator, fp64): the codebook as in ``generate``;
    then per head: ``regions`` seed cells uniform on the grid (each token
    belongs to the region of its nearest seed, lowest seed on ties) and, per
    region, ``comps_per_region`` mixture components (children, or parents for a
    flat codebook) uniform without replacement; then per (batch, head): each
    token's component uniform over its region's, key = component +
    sigma_k N(0, I); query = (q_scale / d) * component + (1 / sqrt(d)) N(0, I),
    so that a query attends mostly to keys of its own component; values
    N(0, 1). Rounding as in ``generate``.
    """
    N = width * height
    if w.N != N:
        raise ValueError(f"workload N={w.N} but the grid has {N} tokens")
    rng = np.random.default_rng(w.seed)
    B, H, d, M0, Ch = w.B, w.H, w.d, w.M0, w.Ch
    cp = rng.standard_normal((H, M0, d))
    if Ch > 0:
        eps = w.sigma_c * rng.standard_normal((H, M0, Ch, d))
        eps -= eps.mean(axis=2, keepdims=True)
        cc = cp[:, :, None, :] + eps
        comps = cc.reshape(H, M0 * Ch, d)
    else:
        cc = np.zeros((H, M0, 0, d))
        comps = cp
    n_comp = comps.shape[1]
    ys, xs = np.divmod(np.arange(N), width)
    region = np.empty((H, N), np.int64)
    members = np.empty((H, regions, comps_per_region), np.int64)
    for h in range(H):
        seeds = rng.integers(0, N, size=regions)
        sy, sx = np.divmod(seeds, width)
        d2 = (ys[:, None] - sy[None, :]) ** 2 + (xs[:, None] - sx[None, :]) ** 2
        region[h] = np.argmin(d2, axis=1)
        for r in range(regions):
            members[h, r] = rng.choice(n_comp, size=comps_per_region, replace=False)
    k = np.empty((B, H, N, d))
    q = np.empty((B, H, N, d))
    for b in range(B):
        for h in range(H):
            pick = rng.integers(0, comps_per_region, size=N)
            comp = members[h, region[h], pick]
            k[b, h] = comps[h, comp] + w.sigma_k * rng.standard_normal((N, d))
            q[b, h] = (w.q_scale / d) * comps[h, comp] + rng.standard_normal((N, d)) / math.sqrt(d)
    v = rng.standard_normal((B, H, N, d))
    return {
        "Q": _round(q, w.dtype),
        "K": _round(k, w.dtype),
        "V": _round(v, w.dtype),
        "Cp": _round(cp, w.dtype),
        "Cc": _round(cc, w.dtype),
    }
