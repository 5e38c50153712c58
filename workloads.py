"""Seeded synthetic workloads for k-MIP attention.

This module only draws random inputs and rounds them to bfloat16.  It holds
none of the attention arithmetic: both the CPU oracle and the GPU path take
the arrays it returns, so that the two sides see bit-identical inputs.

The paper's efficiency study samples Q, K and V from a standard normal
distribution (Appendix H.2, "Objective 1: Computational efficiency"); its
real workloads are superpixel graphs (LRGB), city road networks with Fourier
position encodings (Appendix H.4, City-Networks) and point clouds with xyz
inputs (Appendix H.5, point cloud datasets).  None of those datasets is available here, so each
configuration below is a synthetic stand-in with the same shapes and value
structure:

  c1  single graph, N=2048, H=1, d=32, k=16, i.i.d. N(0,1); forward only
  c2  128 graphs with n_g ~ U{100..450} (block-diagonal batch), H=3, d=32,
      k=16, i.i.d. N(0,1)
  c3  single graph, N=100,000, H=4, d=32, k=32; random Fourier features of
      2-D positions plus N(0, 0.1^2) noise, projected by random matrices
  c4  single graph, N=500,000, H=4, d=16, k=32; random projection of xyz
      uniform in the unit cube plus N(0, 0.05^2) noise, projected again
  c5  single graph, N=262,144, H=1, d=64, k=128; Q and K from a Gaussian
      mixture with 64 centres and sigma 0.1 (many near-tied scores)

Draw order is fixed: structure -> Q -> K -> V -> dOut, from one
``numpy.random.default_rng(seed)`` (PCG64) stream.  Every float32 draw is
rounded to bfloat16 by round-to-nearest-even.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Optional

import numpy as np

__all__ = [
    "Workload", "bf16_round", "bf16_to_f32", "bf16_to_f64", "make", "iid",
    "CONFIGS",
]


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (nearest, ties to even); return raw uint16 bits."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    # NaN stays NaN (quiet); inputs here are always finite.
    lsb = (u >> 16) & 1
    r = (u + 0x7FFF + lsb) >> 16
    return r.astype(np.uint16)


def bf16_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of raw bfloat16 bits to float32."""
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


def bf16_to_f64(b: np.ndarray) -> np.ndarray:
    """Exact widening of raw bfloat16 bits to float64."""
    return bf16_to_f32(b).astype(np.float64)


@dataclass
class Workload:
    """One seeded input set.  Tensors are raw bf16 bits, shape [N, H, d], node-major."""

    name: str
    N: int
    H: int
    d: int
    k: int
    scale: float
    offsets: Optional[np.ndarray]  # int32 [G+1] or None for a single graph
    q: np.ndarray
    kk: np.ndarray
    v: np.ndarray
    dout: Optional[np.ndarray]
    backward: bool = True
    notes: str = ""
    meta: dict = field(default_factory=dict)

    @property
    def num_graphs(self) -> int:
        return 1 if self.offsets is None else len(self.offsets) - 1

    def graph_sizes(self) -> np.ndarray:
        if self.offsets is None:
            return np.array([self.N], dtype=np.int64)
        return np.diff(self.offsets.astype(np.int64))

    def score_pairs(self) -> int:
        """Number of (query, key) score pairs per head summed over graphs (sum of n_g^2)."""
        n = self.graph_sizes()
        return int((n * n).sum())


def _normal(rng, shape, std=1.0):
    return (rng.standard_normal(shape, dtype=np.float32) * np.float32(std)).astype(np.float32)


def iid(N: int, H: int, d: int, k: int, seed: int = 0, sizes=None,
        scale: Optional[float] = None, backward: bool = True, std: float = 1.0,
        name: str = "iid", dv: Optional[int] = None) -> Workload:
    """Q, K, V, dOut i.i.d. N(0, std^2) rounded to bf16.

    ``sizes`` (list of graph sizes) gives a block-diagonal batch; None means one graph.
    ``dv`` is the width of V and dOut (default d).
    """
    rng = np.random.default_rng(seed)
    offsets = None
    if sizes is not None:
        sizes = np.asarray(sizes, dtype=np.int64)
        assert int(sizes.sum()) == N
        offsets = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    dv = d if dv is None else dv
    q = bf16_round(_normal(rng, (N, H, d), std))
    kk = bf16_round(_normal(rng, (N, H, d), std))
    v = bf16_round(_normal(rng, (N, H, dv)))
    dout = bf16_round(_normal(rng, (N, H, dv))) if backward else None
    return Workload(name, N, H, d, k, scale if scale is not None else 1.0 / math.sqrt(d),
                    offsets, q, kk, v, dout, backward)


def _c1(seed: int, n: Optional[int]) -> Workload:
    N = n or 2048
    w = iid(N, 1, 32, 16, seed=seed, backward=False, name="c1")
    w.notes = "single graph, i.i.d. N(0,1) Q/K/V, forward only"
    return w


def _c2(seed: int, n: Optional[int]) -> Workload:
    rng = np.random.default_rng(seed)
    G = n or 128
    sizes = rng.integers(100, 451, size=G).astype(np.int64)
    N = int(sizes.sum())
    offsets = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    H, d = 3, 32
    q = bf16_round(_normal(rng, (N, H, d)))
    kk = bf16_round(_normal(rng, (N, H, d)))
    v = bf16_round(_normal(rng, (N, H, d)))
    dout = bf16_round(_normal(rng, (N, H, d)))
    return Workload("c2", N, H, d, 16, 1.0 / math.sqrt(d), offsets, q, kk, v, dout, True,
                    notes=f"{G} graphs, n_g ~ U{{100..450}}, block-diagonal")


def _c3(seed: int, n: Optional[int], heads: Optional[int] = None, k: Optional[int] = None,
        d: Optional[int] = None) -> Workload:
    rng = np.random.default_rng(seed)
    N = n or 100_000
    H, d, F = heads or 4, d or 32, 32
    pos = rng.random((N, 2), dtype=np.float32)
    omega = _normal(rng, (2, F // 2), 8.0)
    phase = (rng.random(F // 2, dtype=np.float32) * np.float32(2 * math.pi)).astype(np.float32)
    ang = (np.float32(2 * math.pi) * (pos @ omega) + phase).astype(np.float32)
    X = np.concatenate([np.cos(ang), np.sin(ang)], axis=1).astype(np.float32)
    X += _normal(rng, (N, F), 0.1)
    ws = [_normal(rng, (F, H * d), 1.0 / math.sqrt(F)) for _ in range(3)]
    q = bf16_round((X @ ws[0]).reshape(N, H, d))
    kk = bf16_round((X @ ws[1]).reshape(N, H, d))
    v = bf16_round((X @ ws[2]).reshape(N, H, d))
    dout = bf16_round(_normal(rng, (N, H, d)))
    return Workload("c3", N, H, d, k or 32, 1.0 / math.sqrt(d), None, q, kk, v, dout, True,
                    notes="2-D positions, random Fourier features + N(0,0.1^2), random projections")


def _c4(seed: int, n: Optional[int], heads: Optional[int] = None, k: Optional[int] = None,
        d: Optional[int] = None) -> Workload:
    rng = np.random.default_rng(seed)
    N = n or 500_000
    H, d, F = heads or 4, d or 16, 64
    xyz = rng.random((N, 3), dtype=np.float32)
    P = _normal(rng, (3, F))
    X = (xyz @ P).astype(np.float32) + _normal(rng, (N, F), 0.05)
    ws = [_normal(rng, (F, H * d), 1.0 / math.sqrt(F)) for _ in range(3)]
    q = bf16_round((X @ ws[0]).reshape(N, H, d))
    kk = bf16_round((X @ ws[1]).reshape(N, H, d))
    v = bf16_round((X @ ws[2]).reshape(N, H, d))
    dout = bf16_round(_normal(rng, (N, H, d)))
    return Workload("c4", N, H, d, k or 32, 1.0 / math.sqrt(d), None, q, kk, v, dout, True,
                    notes="xyz ~ U[0,1]^3 projected + N(0,0.05^2), random projections")


def _c5(seed: int, n: Optional[int]) -> Workload:
    rng = np.random.default_rng(seed)
    N = n or 262_144
    H, d, C = 1, 64, 64
    mu = _normal(rng, (C, d))
    cq = rng.integers(0, C, size=N)
    ck = rng.integers(0, C, size=N)
    q = bf16_round((mu[cq] + _normal(rng, (N, d), 0.1)).reshape(N, H, d))
    kk = bf16_round((mu[ck] + _normal(rng, (N, d), 0.1)).reshape(N, H, d))
    v = bf16_round(_normal(rng, (N, H, d)))
    dout = bf16_round(_normal(rng, (N, H, d)))
    return Workload("c5", N, H, d, 128, 1.0 / math.sqrt(d), None, q, kk, v, dout, True,
                    notes="Gaussian mixture, 64 centres, sigma 0.1, shared by Q and K")


CONFIGS = {1: _c1, 2: _c2, 3: _c3, 4: _c4, 5: _c5}


def make(config: int, seed: int = 0, n: Optional[int] = None, heads: Optional[int] = None,
         k: Optional[int] = None, d: Optional[int] = None) -> Workload:
    """Build workload ``config`` (1..5).  ``n`` changes N (c2: the number of
    graphs); ``heads``, ``k`` and ``d`` change H, k and the head width of the
    projected-feature workloads c3 and c4 (the features are drawn first, so
    they do not depend on H or d; the projections do)."""
    if heads is not None or k is not None or d is not None:
        if config not in (3, 4):
            raise ValueError("heads, k and d apply to configs 3 and 4")
        return CONFIGS[config](seed, n, heads, k, d)
    return CONFIGS[config](seed, n)
