"""Oracle of the steps either side of route maintenance -- TEST INFRASTRUCTURE.

Plain numpy in binary64, written from the paper's description, for the test
suite, the smoke check and the benchmark's CPU baseline only:

* chunk pooling (Sec. 2.1: the router forms one representation per chunk of
  tokens): the mean of the chunk's token vectors;
* token expansion (Sec. 2.1: selected chunks are expanded into token indices):
  chunk j covers tokens j*C .. min((j+1)*C, n_tokens) - 1;
* sparse attention over the expanded tokens (Sec. 2.2 Eq. (3)): a query token
  attends, with one softmax, to the tokens of its chunk's routed chunks,
  scaled by 1/sqrt(d), keys after the query excluded when causal.

Readings (the paper leaves them to the router and the attention backend):
chunks are consecutive runs of C tokens, the last one possibly shorter; every
query token of chunk i uses chunk i's route; route slots holding -1 (or an id
outside the chunk range) contribute nothing; a query with no admissible key
gets a zero output.  Inputs are binary32 arrays (bf16 inputs widened exactly).
"""
from __future__ import annotations

import math

import numpy as np


def n_chunks(n_tokens: int, chunk: int) -> int:
    return -(-n_tokens // chunk)


def pool_chunks(X: np.ndarray, chunk: int) -> np.ndarray:
    """[H, n_tokens, d] -> [H, ceil(n_tokens / chunk), d]: each chunk's mean
    token vector, in binary64."""
    H, n, d = X.shape
    nc = n_chunks(n, chunk)
    out = np.zeros((H, nc, d), np.float64)
    for j in range(nc):
        lo, hi = j * chunk, min((j + 1) * chunk, n)
        out[:, j] = X[:, lo:hi].astype(np.float64).sum(axis=1) / (hi - lo)
    return out


def expand_tokens(routes: np.ndarray, chunk: int, n_tokens: int) -> np.ndarray:
    """[rows, k] chunk ids -> [rows, k*chunk] token ids: route slot s fills
    columns s*chunk .. s*chunk + chunk - 1 with its chunk's tokens ascending,
    -1 past the last token or for an empty (or out-of-range) slot."""
    rows, k = routes.shape
    nc = n_chunks(n_tokens, chunk)
    out = np.full((rows, k * chunk), -1, np.int32)
    for r in range(rows):
        for s in range(k):
            j = int(routes[r, s])
            if j < 0 or j >= nc:
                continue
            for t in range(chunk):
                u = j * chunk + t
                if u < n_tokens:
                    out[r, s * chunk + t] = u
    return out


def sparse_attention(Q, K, V, routes, chunk, causal, scale=None, rows=None):
    """Eq. (3) over the expanded tokens.

    Q [H, n, d], K and V [H_kv, n, d]; query head h reads key head
    h // (H // H_kv).  routes [H * n_chunks, k] (row = h * n_chunks + i).
    rows: optional iterable of (h, t) query tokens; returns [len(rows), d]
    for those, else the whole [H, n, d] output.  binary64."""
    H, n, d = Q.shape
    Hkv = K.shape[0]
    group = H // Hkv
    nc = n_chunks(n, chunk)
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    routes = np.asarray(routes)

    def one(h, t):
        i = t // chunk
        # the tokens of the row's admissible route slots, slot by slot
        parts = [np.arange(j * chunk, min((j + 1) * chunk, n)) for j in routes[h * nc + i].tolist() if 0 <= j < nc]
        u = np.concatenate(parts) if parts else np.zeros(0, np.int64)
        if causal:
            u = u[u <= t]
        if len(u) == 0:
            return np.zeros(d)
        g = h // group
        q = Q[h, t].astype(np.float64)
        s = (K[g, u].astype(np.float64) @ q) * scale
        p = np.exp(s - s.max())
        return (p / p.sum()) @ V[g, u].astype(np.float64)

    if rows is not None:
        return np.stack([one(h, t) for h, t in rows]) if len(rows) else np.zeros((0, d))
    out = np.zeros((H, n, d))
    for h in range(H):
        for t in range(n):
            out[h, t] = one(h, t)
    return out

