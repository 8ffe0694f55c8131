"""Seeded synthetic chunk representations for the route-maintenance workloads.

This module only draws inputs.  It holds none of the routing arithmetic, and it
is the one piece of code that both the GPU path's tests/benchmark and the
oracle's tests use.

Recipe (the draw order is part of the definition; ``numpy.random.default_rng``
with PCG64):

1. per key head g, ``C`` cluster centres ``mu[g] ~ N(0, I_d)``;
2. a cluster id per key chunk, uniform over ``C``;
3. a cluster id per query chunk, uniform over ``C`` (a query head uses the
   centres of the key head it reads, so queries have same-cluster keys);
4. ``K0 = (mu[z] + 0.3 eps) / sqrt(d)`` with ``eps ~ N(0, I_d)``;
5. ``Q0`` likewise;
6. near-tie workloads only: 25 % of the key chunks of each head (without
   replacement) become duplicates, each paired with a source key of the same
   cluster (any non-duplicate key if its cluster has none);
7. per layer l >= 1: ``Q <- sqrt(1 - rho^2) Q + rho xi`` and then the same for
   ``K``, with ``xi ~ N(0, 1/d)`` per element;
8. near-tie workloads, at every layer after the drift step:
   ``K[dup] = K[src] + 1e-3 eta`` with ``eta ~ N(0, I_d)``.

Query-dependent route budgets (``route_budgets``) come from a stream of their
own, ``default_rng([seed, 7])``: each row draws one of a few widths (buckets)
uniformly.

bf16 workloads round the binary32 draw to bf16 with round-to-nearest-even; the
GPU reads those bits and the oracle reads the same values widened exactly to
binary32.
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace
from typing import Iterator, Tuple

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    n_heads: int
    n_kv_heads: int
    n_layers: int
    anchor_every: int          # anchors at layers 0, a, 2a, ... (0: layer 0 only)
    n: int                     # n_q = n_k chunks
    d: int
    dtype: str                 # "f32" or "bf16"
    k: int
    m: int
    r: int
    clusters: int
    rho: float                 # drift coefficient of the AR(1) step
    causal: bool = False
    near_ties: bool = False
    seed: int = 0
    gamma: float = 0.0
    n_keys: int = 0            # key chunks n_k when it differs from n_q = n (0: n_k = n)
    n_sink: int = 0            # mandatory sink sentinels
    n_recent: int = 0          # mandatory recent sentinels
    min_reuse: int = 0         # minimum reuse horizon (layers)
    extra: dict = field(default_factory=dict, compare=False)

    @property
    def rows(self) -> int:
        return self.n_heads * self.n

    @property
    def nk(self) -> int:
        return self.n_keys or self.n

    def is_anchor(self, layer: int) -> bool:
        if layer == 0:
            return True
        return self.anchor_every > 0 and layer % self.anchor_every == 0

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


def preset(name: str, **kw) -> Workload:
    """Named workloads: tiny, drift, scale, gqa, longctx, ablation, stride."""
    if name == "tiny":
        w = Workload("tiny", 1, 1, 4, 0, 128, 64, "f32", 8, 4, 4, 16, 0.3)
    elif name == "drift":
        w = Workload("drift", 8, 8, 16, 8, 256, 128, "f32", 16, 8, 8, 16, 0.3)
    elif name == "scale":
        w = Workload("scale", 32, 32, 32, 8, 1024, 128, "bf16", 32, 16, 16, 64, 0.3)
    elif name == "gqa":
        w = Workload("gqa", 32, 8, 32, 8, 512, 128, "bf16", 32, 16, 16, 64, 0.3, causal=True)
    elif name == "longctx":
        w = Workload("longctx", 32, 32, 32, 8, 4096, 128, "bf16", 64, 32, 32, 64, 0.6,
                     causal=True, near_ties=True)
    elif name == "ablation":
        # the sentinel-ablation shape (Sec. 5.2, Table 3): 256 query rows, 256
        # key chunks, d = 64, top-12, 24 layers with one anchor; sentinel
        # widths vary per study point
        w = Workload("ablation", 1, 1, 24, 0, 256, 64, "f32", 12, 12, 12, 16, 0.05)
    elif name == "stride":
        # the cross-layer drift shape (Sec. 5.1, Table 2): 384 query rows, 192
        # key chunks, top-12 with 24 near-miss and 12 random sentinels, 32
        # layers with one anchor
        w = Workload("stride", 1, 1, 32, 0, 384, 64, "f32", 12, 24, 12, 16, 0.2, n_keys=192)
    else:
        raise KeyError(name)
    return w.with_(**kw) if kw else w


def route_budgets(w: Workload, widths=None) -> np.ndarray:
    """Per-row route widths k_i (int32 [rows], head-major like the rows): one
    of ``widths`` per row, uniformly; by default the four buckets k/4, k/2,
    3k/4 and k (at least 1)."""
    if widths is None:
        widths = sorted({max(1, (w.k * q) // 4) for q in (1, 2, 3, 4)})
    widths = np.asarray(widths, dtype=np.int32)
    if widths.min() < 1 or widths.max() > w.k:
        raise ValueError("route widths must lie in [1, k]")
    rng = np.random.default_rng([w.seed, 7])
    return widths[rng.integers(0, len(widths), size=w.rows)].astype(np.int32)


def bf16_round(x: np.ndarray) -> np.ndarray:
    """binary32 -> bf16 bit patterns (uint16), round to nearest, ties to even."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    b = (b + 0x7FFF + ((b >> 16) & 1)) >> 16
    return b.astype(np.uint16)


def bf16_widen(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns -> binary32 values (exact)."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


class Generator:
    """Streams the layers of a workload: ``for l, Qf, Kf, Qdev, Kdev in Generator(w)``.

    ``Qf``/``Kf`` are binary32 values (bf16-exact for bf16 workloads);
    ``Qdev``/``Kdev`` are what the device reads (binary32, or uint16 bf16 bits).
    """

    def __init__(self, w: Workload):
        self.w = w

    def __iter__(self) -> Iterator[Tuple[int, np.ndarray, np.ndarray, np.ndarray, np.ndarray]]:
        w = self.w
        d = w.d
        rng = np.random.default_rng(w.seed)
        mu = rng.standard_normal((w.n_kv_heads, w.clusters, d))
        nk = w.nk
        zk = rng.integers(0, w.clusters, size=(w.n_kv_heads, nk))
        zq = rng.integers(0, w.clusters, size=(w.n_heads, w.n))
        group = w.n_heads // w.n_kv_heads
        K = np.empty((w.n_kv_heads, nk, d), dtype=np.float64)
        for g in range(w.n_kv_heads):
            K[g] = mu[g][zk[g]]
        K += 0.3 * rng.standard_normal(K.shape)
        K /= np.sqrt(d)
        Q = np.empty((w.n_heads, w.n, d), dtype=np.float64)
        for h in range(w.n_heads):
            Q[h] = mu[h // group][zq[h]]
        Q += 0.3 * rng.standard_normal(Q.shape)
        Q /= np.sqrt(d)
        dups = None
        if w.near_ties:
            dups = []
            n_dup = nk // 4
            for g in range(w.n_kv_heads):
                dup = np.sort(rng.permutation(nk)[:n_dup])
                is_dup = np.zeros(nk, dtype=bool)
                is_dup[dup] = True
                src = np.empty(n_dup, dtype=np.int64)
                for t, j in enumerate(dup):
                    same = np.flatnonzero((zk[g] == zk[g][j]) & ~is_dup)
                    pool = same if len(same) else np.flatnonzero(~is_dup)
                    src[t] = pool[rng.integers(0, len(pool))]
                dups.append((dup, src))
        a = np.sqrt(1.0 - w.rho * w.rho)
        for layer in range(w.n_layers):
            if layer > 0:
                Q *= a
                Q += (w.rho / np.sqrt(d)) * rng.standard_normal(Q.shape)
                K *= a
                K += (w.rho / np.sqrt(d)) * rng.standard_normal(K.shape)
            if dups is not None:
                for g, (dup, src) in enumerate(dups):
                    K[g, dup] = K[g, src] + 1e-3 * rng.standard_normal((len(dup), d))
            Q32 = Q.astype(np.float32)
            K32 = K.astype(np.float32)
            if w.dtype == "bf16":
                Qb, Kb = bf16_round(Q32), bf16_round(K32)
                yield layer, bf16_widen(Qb), bf16_widen(Kb), Qb, Kb
            elif w.dtype == "f32":
                yield layer, Q32, K32, Q32, K32
            else:
                raise ValueError(w.dtype)


def layers(w: Workload):
    """Materialise every layer: list of (Qf, Kf, Qdev, Kdev)."""
    return [(Qf, Kf, Qd, Kd) for _, Qf, Kf, Qd, Kd in Generator(w)]
