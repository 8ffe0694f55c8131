"""RouteRelay reference oracle (arXiv 2609.07306) -- TEST INFRASTRUCTURE.

A thin ctypes wrapper over ``rr_oracle.c``: plain, slow, single-threaded C that
computes in binary64 what the route-maintenance path computes (full routing,
Sec. 2.1 Eq. (1)-(2); the route ledger, Sec. 3.1; candidate rescoring and the
trigger, Sec. 3.2 Eq. (5)-(8)).  Only the test-suite, the smoke check and the
benchmark's CPU-baseline leg may import this package.  It imports nothing from
the product package, and the product package imports nothing from here.

Inputs are binary32 numpy arrays: ``Q`` is [H_q, n_q, d] and ``K`` is
[H_kv, n_k, d].  For bf16 workloads the caller passes the bf16 values widened
exactly to binary32 (the same bits the GPU reads).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass, field

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "rr_oracle.c")
_LIB = os.path.join(_HERE, "librr_oracle.so")


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (C99, -O2, no fast-math)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp"
        subprocess.check_call(
            ["gcc", "-std=c99", "-O2", "-fno-fast-math", "-ffp-contract=off", "-shared",
             "-fPIC", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


class _Problem(ctypes.Structure):
    _fields_ = [
        ("n_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
        ("n_q", ctypes.c_int32), ("n_k", ctypes.c_int32), ("d", ctypes.c_int32),
        ("k", ctypes.c_int32), ("m", ctypes.c_int32), ("r", ctypes.c_int32),
        ("causal", ctypes.c_int32), ("pad_", ctypes.c_int32),
        ("gamma", ctypes.c_double), ("seed", ctypes.c_uint64),
        ("n_sink", ctypes.c_int32), ("n_recent", ctypes.c_int32),
        ("min_reuse", ctypes.c_int32), ("pad2_", ctypes.c_int32),
        ("gamma_rows", ctypes.c_void_p), ("k_rows", ctypes.c_void_p),
    ]


@dataclass(frozen=True)
class Problem:
    """Shape and rule parameters of one routing problem."""
    n_heads: int
    n_kv_heads: int
    n_q: int
    n_k: int
    d: int
    k: int
    m: int = 0
    r: int = 0
    causal: bool = False
    gamma: float = 0.0
    seed: int = 0
    n_sink: int = 0        # mandatory sentinels: the first n_sink chunks ...
    n_recent: int = 0      # ... and the n_recent most recent valid chunks (Sec. 3.1, item 3)
    min_reuse: int = 0     # hysteresis: rows (re)built at layer b keep their route through b + min_reuse
    gamma_rows: object = field(default=None, compare=False)  # per-row guard margins (binary64 [rows]) or None
    k_rows: object = field(default=None, compare=False)      # per-row route widths (int32 [rows], 1..k) or None

    @property
    def rows(self) -> int:
        return self.n_heads * self.n_q

    @property
    def sent_width(self) -> int:
        """Sentinel slots per row: near-miss, random, then mandatory."""
        return self.m + self.r + self.n_sink + self.n_recent

    def n_valid(self, i: int) -> int:
        return min(i + 1, self.n_k) if self.causal else self.n_k

    def k_of(self, row: int) -> int:
        """The route width of a row (k_i, or k)."""
        return int(self.k_rows[row]) if self.k_rows is not None else self.k

    def _c(self) -> _Problem:
        g = None
        if self.gamma_rows is not None:
            g = np.ascontiguousarray(self.gamma_rows, dtype=np.float64)
            if g.shape != (self.rows,):
                raise ValueError("gamma_rows must have one entry per row")
            object.__setattr__(self, "_keep", g)  # (kept alive while the struct is in use)
        kr = None
        if self.k_rows is not None:
            kr = np.ascontiguousarray(self.k_rows, dtype=np.int32)
            if kr.shape != (self.rows,) or kr.min() < 1 or kr.max() > self.k:
                raise ValueError("k_rows must hold one width in [1, k] per row")
            object.__setattr__(self, "_keep_k", kr)
        return _Problem(self.n_heads, self.n_kv_heads, self.n_q, self.n_k, self.d, self.k,
                        self.m, self.r, int(self.causal), 0, float(self.gamma),
                        int(self.seed) & 0xFFFFFFFFFFFFFFFF, int(self.n_sink), int(self.n_recent),
                        int(self.min_reuse), 0, None if g is None else g.ctypes.data,
                        None if kr is None else kr.ctypes.data)


_lib = None


def _load():
    global _lib
    if _lib is None:
        lib = ctypes.CDLL(build())
        P = ctypes.POINTER(_Problem)
        vp = ctypes.c_void_p
        i32, i64, u64 = ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64
        lib.orc_splitmix64.argtypes = [u64]
        lib.orc_splitmix64.restype = u64
        lib.orc_probe_hash.argtypes = [u64, u64, u64, u64, u64]
        lib.orc_probe_hash.restype = u64
        lib.orc_random_sentinels.argtypes = [P, i32, i64, i32, vp, i32, vp, i32, vp]
        lib.orc_full_route.argtypes = [P, vp, vp, vp, i64, vp, vp, vp]
        lib.orc_route_bounds.argtypes = [P, vp, vp, vp, i64, vp]
        lib.orc_anchor.argtypes = [P, i32, vp, vp, vp, i64, vp, vp, vp, vp, vp, vp]
        lib.orc_relay.argtypes = [P, i32, vp, vp, vp, i64, vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                  vp, vp]
        for f in ("orc_random_sentinels", "orc_full_route", "orc_route_bounds", "orc_anchor",
                  "orc_relay"):
            getattr(lib, f).restype = ctypes.c_int
        _lib = lib
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _check_inputs(p: Problem, Q, K):
    Q = np.ascontiguousarray(Q, dtype=np.float32)
    K = np.ascontiguousarray(K, dtype=np.float32)
    if Q.shape != (p.n_heads, p.n_q, p.d):
        raise ValueError(f"Q shape {Q.shape} != {(p.n_heads, p.n_q, p.d)}")
    if K.shape != (p.n_kv_heads, p.n_k, p.d):
        raise ValueError(f"K shape {K.shape} != {(p.n_kv_heads, p.n_k, p.d)}")
    if p.n_heads % p.n_kv_heads:
        raise ValueError("n_heads must be a multiple of n_kv_heads")
    if p.causal and p.n_q != p.n_k:
        raise ValueError("the causal chunk mask needs n_q == n_k")
    return Q, K


def _rows_arg(rows):
    if rows is None:
        return None, 0
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    return rows, len(rows)


def _rc(code):
    if code != 0:
        raise MemoryError(f"oracle call failed with code {code}")


# ------------------------------------------------------------------ hashing

def splitmix64(z: int) -> int:
    """splitmix64 output function (increment, then two xor-shift-multiply rounds)."""
    return int(_load().orc_splitmix64(z & 0xFFFFFFFFFFFFFFFF))


def probe_hash(seed: int, layer: int, row: int, slot: int, attempt: int) -> int:
    """Counter hash of one random probe, chained over (seed, layer, row, slot, attempt)."""
    return int(_load().orc_probe_hash(seed & 0xFFFFFFFFFFFFFFFF, layer, row, slot, attempt))


def random_sentinels(p: Problem, layer: int, row: int, n_valid: int, R, N):
    """Random sentinels of one row, given its selected set R and near-miss set N."""
    R = np.ascontiguousarray([x for x in R if x >= 0], dtype=np.int32)
    N = np.ascontiguousarray([x for x in N if x >= 0], dtype=np.int32)
    out = np.empty(p.r, dtype=np.int32)
    _rc(_load().orc_random_sentinels(ctypes.byref(p._c()), layer, row, n_valid, _ptr(R), len(R),
                                     _ptr(N), len(N), _ptr(out)))
    return out


# ------------------------------------------------------------------ routing

def full_route(p: Problem, Q, K, rows=None, with_scores: bool = False):
    """Eq. (1)-(2) for every row (or the listed rows).

    Returns ``routes`` [rows, k] int32 (sorted by id, -1 padded), the total
    score-pair count and, if asked, the binary64 scores of the route slots.
    """
    Q, K = _check_inputs(p, Q, K)
    rows, n = _rows_arg(rows)
    routes = np.full((p.rows, p.k), -1, dtype=np.int32)
    scores = np.full((p.rows, p.k), np.nan) if with_scores else None
    pairs = np.zeros(1, dtype=np.int64)
    _rc(_load().orc_full_route(ctypes.byref(p._c()), _ptr(Q), _ptr(K), _ptr(rows), n,
                               _ptr(routes), _ptr(scores), _ptr(pairs)))
    if with_scores:
        return routes, int(pairs[0]), scores
    return routes, int(pairs[0])


def route_bounds(p: Problem, Q, K, rows=None):
    """Per row: scores at ranks k, k+1, k+m, k+m+1 and their sum_t |q_t k_t|.

    Returns an array [n_rows, 8] (NaN where the rank does not exist).
    """
    Q, K = _check_inputs(p, Q, K)
    rows, n = _rows_arg(rows)
    out = np.empty((n if rows is not None else p.rows, 8), dtype=np.float64)
    _rc(_load().orc_route_bounds(ctypes.byref(p._c()), _ptr(Q), _ptr(K), _ptr(rows), n,
                                 _ptr(out)))
    return out


def new_ledger(p: Problem):
    """An empty ledger in the layout of Sec. 4.1: routes, sentinels, build layer, age."""
    return {
        "routes": np.full((p.rows, p.k), -1, dtype=np.int32),
        "sent": np.full((p.rows, p.sent_width), -1, dtype=np.int32),
        "build": np.full(p.rows, -1, dtype=np.int32),
        "age": np.zeros(p.rows, dtype=np.int32),
    }


def anchor(p: Problem, layer: int, Q, K, ledger, rows=None):
    """Anchor layer: rebuild the ledger of every (listed) row.  Returns (mask, pairs)."""
    Q, K = _check_inputs(p, Q, K)
    rows, n = _rows_arg(rows)
    mask = np.zeros(p.rows, dtype=np.uint8)
    pairs = np.zeros(1, dtype=np.int64)
    _rc(_load().orc_anchor(ctypes.byref(p._c()), layer, _ptr(Q), _ptr(K), _ptr(rows), n,
                           _ptr(ledger["routes"]), _ptr(ledger["sent"]), _ptr(ledger["build"]),
                           _ptr(ledger["age"]), _ptr(mask), _ptr(pairs)))
    return mask, int(pairs[0])


def relay(p: Problem, layer: int, Q, K, ledger, rows=None):
    """Relay layer: rescore, trigger and refresh.  Updates ``ledger`` in place.

    Returns a dict with ``mask`` [rows] uint8, ``pairs``, per-row
    ``row_pairs`` (int64: |A_i| plus n_i when rerouted; -1 on rows not
    relayed), and per-row ``alpha``/``beta`` (binary64) plus
    ``alpha_abs``/``beta_abs``.
    """
    Q, K = _check_inputs(p, Q, K)
    rows, n = _rows_arg(rows)
    row_pairs = np.full(p.rows, -1, dtype=np.int64)
    mask = np.zeros(p.rows, dtype=np.uint8)
    a = np.full(p.rows, np.nan)
    b = np.full(p.rows, np.nan)
    aa = np.full(p.rows, np.nan)
    ba = np.full(p.rows, np.nan)
    pairs = np.zeros(1, dtype=np.int64)
    _rc(_load().orc_relay(ctypes.byref(p._c()), layer, _ptr(Q), _ptr(K), _ptr(rows), n,
                          _ptr(ledger["routes"]), _ptr(ledger["sent"]), _ptr(ledger["build"]),
                          _ptr(ledger["age"]), _ptr(mask), _ptr(a), _ptr(b), _ptr(aa), _ptr(ba),
                          _ptr(pairs), _ptr(row_pairs)))
    return {"mask": mask, "pairs": int(pairs[0]), "row_pairs": row_pairs, "alpha": a, "beta": b,
            "alpha_abs": aa, "beta_abs": ba}


def recall(routes, exact) -> float:
    """Fraction of the exact per-layer top-k chunk ids present in ``routes``."""
    hit = tot = 0
    for a, b in zip(np.asarray(routes), np.asarray(exact)):
        e = set(int(x) for x in b if x >= 0)
        hit += len(e & set(int(x) for x in a if x >= 0))
        tot += len(e)
    return hit / tot if tot else 1.0
