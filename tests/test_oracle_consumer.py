"""Pins of the consumer-side oracle (chunk pooling, token expansion, sparse
attention over the expanded tokens; Sec. 2.1 and Sec. 2.2 Eq. (3)) against
library routines and hand cases."""
import math

import numpy as np
import pytest
import torch

from oracle import consumer as oc


def _rand(rng, *shape):
    return rng.standard_normal(shape).astype(np.float32)


def test_pool_divisible_equals_reshape_mean():
    rng = np.random.default_rng(1)
    X = _rand(rng, 3, 48, 16)
    np.testing.assert_allclose(oc.pool_chunks(X, 8), X.astype(np.float64).reshape(3, 6, 8, 16).mean(2),
                               rtol=0, atol=1e-15)


def test_pool_ragged_tail_and_constant_chunks():
    rng = np.random.default_rng(2)
    X = _rand(rng, 2, 21, 4)
    X[:, 0:5] = X[:, 0:1]  # a chunk of identical vectors
    P = oc.pool_chunks(X, 5)
    assert P.shape == (2, 5, 4)
    np.testing.assert_array_equal(P[:, 0], X[:, 0].astype(np.float64))
    # the last chunk holds the single token 20
    np.testing.assert_array_equal(P[:, 4], X[:, 20].astype(np.float64))
    np.testing.assert_allclose(P[:, 3], X[:, 15:20].astype(np.float64).mean(1), rtol=0, atol=1e-15)


def test_expand_tokens_hand_case():
    routes = np.array([[2, -1, 0], [1, 9, -1]], np.int32)
    got = oc.expand_tokens(routes, 3, 8)
    assert got.tolist() == [[6, 7, -1, -1, -1, -1, 0, 1, 2], [3, 4, 5, -1, -1, -1, -1, -1, -1]]


def _sdpa(Q, K, V, causal):
    group = Q.shape[0] // K.shape[0]
    q = torch.from_numpy(Q.astype(np.float64))
    k = torch.from_numpy(K.astype(np.float64)).repeat_interleave(group, 0)
    v = torch.from_numpy(V.astype(np.float64)).repeat_interleave(group, 0)
    return torch.nn.functional.scaled_dot_product_attention(q, k, v, is_causal=causal).numpy()


@pytest.mark.parametrize("n,chunk", [(40, 8), (37, 8), (33, 16)])
def test_every_chunk_routed_is_dense_attention(n, chunk):
    rng = np.random.default_rng(n)
    H, Hkv, d = 4, 2, 16
    Q, K, V = _rand(rng, H, n, d), _rand(rng, Hkv, n, d), _rand(rng, Hkv, n, d)
    nc = oc.n_chunks(n, chunk)
    routes = np.tile(rng.permutation(nc).astype(np.int32), (H * nc, 1))
    np.testing.assert_allclose(oc.sparse_attention(Q, K, V, routes, chunk, False), _sdpa(Q, K, V, False),
                               rtol=0, atol=1e-12)


@pytest.mark.parametrize("n,chunk", [(40, 8), (37, 8)])
def test_causal_prefix_routes_are_causal_attention(n, chunk):
    rng = np.random.default_rng(100 + n)
    H, Hkv, d = 2, 1, 8
    Q, K, V = _rand(rng, H, n, d), _rand(rng, Hkv, n, d), _rand(rng, Hkv, n, d)
    nc = oc.n_chunks(n, chunk)
    routes = np.full((H * nc, nc), -1, np.int32)
    for h in range(H):
        for i in range(nc):
            routes[h * nc + i, : i + 1] = rng.permutation(i + 1)
    np.testing.assert_allclose(oc.sparse_attention(Q, K, V, routes, chunk, True), _sdpa(Q, K, V, True),
                               rtol=0, atol=1e-12)


def test_sparse_routes_match_masked_dense_attention():
    """A sparse route equals dense attention with the unrouted keys masked
    out (torch's boolean-mask form)."""
    rng = np.random.default_rng(7)
    H, n, d, chunk, k = 2, 48, 8, 4, 3
    Q, K, V = _rand(rng, H, n, d), _rand(rng, H, n, d), _rand(rng, H, n, d)
    nc = n // chunk
    routes = np.stack([rng.choice(nc, k, replace=False) for _ in range(H * nc)]).astype(np.int32)
    for causal in (False, True):
        allow = np.zeros((H, n, n), bool)
        for h in range(H):
            for t in range(n):
                for j in routes[h * nc + t // chunk]:
                    allow[h, t, j * chunk:(j + 1) * chunk] = True
        if causal:
            allow &= np.tril(np.ones((n, n), bool))[None]
        has = allow.any(2)
        q, kk, v = (torch.from_numpy(x.astype(np.float64)) for x in (Q, K, V))
        ref = torch.nn.functional.scaled_dot_product_attention(
            q, kk, v, attn_mask=torch.from_numpy(allow | ~has[:, :, None])).numpy()
        ref[~has] = 0.0
        np.testing.assert_allclose(oc.sparse_attention(Q, K, V, routes, chunk, causal), ref, rtol=0, atol=1e-12)


def test_invariances_and_degenerate_cases():
    rng = np.random.default_rng(3)
    H, n, d, chunk = 1, 24, 8, 4
    Q, K, V = _rand(rng, H, n, d), _rand(rng, H, n, d), _rand(rng, H, n, d)
    nc = n // chunk
    routes = np.stack([rng.choice(nc, 2, replace=False) for _ in range(nc)]).astype(np.int32)
    base = oc.sparse_attention(Q, K, V, routes, chunk, False)
    # slot order, empty and out-of-range slots change nothing
    padded = np.concatenate([routes[:, ::-1], np.full((nc, 1), -1, np.int32), np.full((nc, 1), nc + 5, np.int32)], 1)
    np.testing.assert_allclose(oc.sparse_attention(Q, K, V, padded, chunk, False), base, rtol=0, atol=1e-15)
    # a common shift of every key (exact in binary64) shifts each query's
    # scores uniformly
    np.testing.assert_allclose(oc.sparse_attention(Q, K.astype(np.float64) + _rand(rng, 1, 1, d), V, routes, chunk, False), base,
                               rtol=0, atol=1e-12)
    # one token per chunk and one routed chunk: the output is that token's value
    one = np.arange(n, dtype=np.int32)[::-1].reshape(n, 1).copy()
    out = oc.sparse_attention(Q, K, V, one, 1, False)
    np.testing.assert_array_equal(out[0], V[0, ::-1].astype(np.float64))
    # no admissible key: zero output
    none = np.full((nc, 2), -1, np.int32)
    assert not oc.sparse_attention(Q, K, V, none, chunk, True).any()
    # sampled rows equal the corresponding entries of the whole output
    rows = [(0, 0), (0, 13), (0, 23)]
    np.testing.assert_array_equal(oc.sparse_attention(Q, K, V, routes, chunk, False, rows=rows),
                                  base[0, [0, 13, 23]])
    # the scale: doubling it equals doubling the queries
    np.testing.assert_allclose(oc.sparse_attention(Q, K, V, routes, chunk, False, scale=2 / math.sqrt(d)),
                               oc.sparse_attention(2 * Q, K, V, routes, chunk, False), rtol=0, atol=1e-12)
