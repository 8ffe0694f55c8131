"""Pins of the oracle's full routing (Sec. 2.1, Eq. (1)-(2)) and ledger build
(Sec. 3.1) against definitions that do not go through the oracle's code:
exact rational brute force over all subsets, and numpy's stable lexsort."""
import itertools
from fractions import Fraction

import numpy as np
import pytest

import oracle
from oracle import Problem


def exact_scores(q, K):
    """Exact rational dot products of binary32 inputs."""
    qf = [Fraction(float(x)) for x in q]
    return [sum(a * Fraction(float(b)) for a, b in zip(qf, krow)) for krow in K]


def better(sa, a, sb, b):
    return sa > sb or (sa == sb and a < b)


def brute_topset(scores, ids, size):
    """The unique subset of ``ids`` of the given size whose every member ranks
    above every non-member (found by enumeration)."""
    found = []
    for S in itertools.combinations(ids, size):
        rest = [j for j in ids if j not in S]
        if all(better(scores[a], a, scores[b], b) for a in S for b in rest):
            found.append(sorted(S))
    assert len(found) == 1, found
    return found[0]


def tiny_inputs(rng, p, quantised):
    if quantised:
        # quarter-integers: many exactly equal scores, exercising the id tie-break
        Q = rng.integers(-2, 3, size=(p.n_heads, p.n_q, p.d)).astype(np.float32) / 4
        K = rng.integers(-2, 3, size=(p.n_kv_heads, p.n_k, p.d)).astype(np.float32) / 4
    else:
        Q = rng.standard_normal((p.n_heads, p.n_q, p.d)).astype(np.float32)
        K = rng.standard_normal((p.n_kv_heads, p.n_k, p.d)).astype(np.float32)
    return Q, K


@pytest.mark.parametrize("quantised", [True, False])
@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("k,m", [(1, 0), (2, 2), (3, 1), (4, 3), (8, 0)])
def test_anchor_matches_bruteforce(quantised, causal, k, m):
    rng = np.random.default_rng(100 + 10 * k + m + (7 if causal else 0) + (3 if quantised else 0))
    n = 8
    p = Problem(n_heads=4, n_kv_heads=2, n_q=n, n_k=n, d=3, k=k, m=m, r=0, causal=causal)
    Q, K = tiny_inputs(rng, p, quantised)
    led = oracle.new_ledger(p)
    mask, pairs = oracle.anchor(p, 0, Q, K, led)
    full, full_pairs = oracle.full_route(p, Q, K)
    assert mask.all()
    expect_pairs = 0
    for h in range(p.n_heads):
        g = h // (p.n_heads // p.n_kv_heads)
        for i in range(n):
            row = h * n + i
            ni = i + 1 if causal else n
            expect_pairs += ni
            s = exact_scores(Q[h, i], K[g, :ni])
            ids = list(range(ni))
            R = brute_topset(s, ids, min(k, ni))
            rest = [j for j in ids if j not in R]
            Nn = brute_topset(s, rest, min(m, len(rest))) if m else []
            assert list(led["routes"][row][: len(R)]) == R
            assert (led["routes"][row][len(R):] == -1).all()
            assert list(full[row][: len(R)]) == R
            assert list(led["sent"][row][: len(Nn)]) == Nn
            assert (led["sent"][row][len(Nn): m] == -1).all()
    assert pairs == expect_pairs == full_pairs
    assert (led["build"] == 0).all() and (led["age"] == 0).all()


@pytest.mark.parametrize("causal", [False, True])
def test_anchor_matches_numpy_lexsort(causal):
    rng = np.random.default_rng(7)
    p = Problem(n_heads=3, n_kv_heads=3, n_q=150, n_k=150, d=32, k=20, m=10, r=0, causal=causal)
    Q = rng.standard_normal((3, 150, 32)).astype(np.float32)
    K = rng.standard_normal((3, 150, 32)).astype(np.float32)
    led = oracle.new_ledger(p)
    oracle.anchor(p, 0, Q, K, led)
    for h in range(3):
        S = Q[h].astype(np.float64) @ K[h].astype(np.float64).T
        for i in range(150):
            ni = i + 1 if causal else 150
            s = S[i, :ni]
            order = np.lexsort((np.arange(ni), -s))
            R = np.sort(order[: min(20, ni)])
            N = np.sort(order[min(20, ni): min(30, ni)])
            row = h * 150 + i
            np.testing.assert_array_equal(led["routes"][row][: len(R)], R)
            np.testing.assert_array_equal(led["sent"][row][: len(N)], N)


def test_full_route_scores_and_defining_property():
    rng = np.random.default_rng(11)
    p = Problem(n_heads=2, n_kv_heads=1, n_q=64, n_k=300, d=16, k=12)
    Q = rng.standard_normal((2, 64, 16)).astype(np.float32)
    K = rng.standard_normal((1, 300, 16)).astype(np.float32)
    routes, pairs, scores = oracle.full_route(p, Q, K, with_scores=True)
    assert pairs == 2 * 64 * 300
    for h in range(2):
        S = Q[h].astype(np.float64) @ K[0].astype(np.float64).T
        for i in range(64):
            row = h * 64 + i
            R = routes[row]
            assert np.all(np.diff(R) > 0)
            np.testing.assert_allclose(scores[row], S[i, R], rtol=1e-12, atol=1e-12)
            out = np.setdiff1d(np.arange(300), R)
            assert S[i, R].min() > S[i, out].max()


def test_row_subset_matches_all_rows():
    rng = np.random.default_rng(3)
    p = Problem(n_heads=2, n_kv_heads=2, n_q=40, n_k=40, d=8, k=5, m=3, r=4, causal=True)
    Q = rng.standard_normal((2, 40, 8)).astype(np.float32)
    K = rng.standard_normal((2, 40, 8)).astype(np.float32)
    a = oracle.new_ledger(p)
    oracle.anchor(p, 2, Q, K, a)
    rows = np.array([0, 5, 39, 40, 77])
    b = oracle.new_ledger(p)
    _, pairs = oracle.anchor(p, 2, Q, K, b, rows=rows)
    for key in ("routes", "sent", "build", "age"):
        np.testing.assert_array_equal(a[key][rows], b[key][rows])
    assert pairs == sum(p.n_valid(int(x) % 40) for x in rows)


def test_route_bounds_ranks():
    rng = np.random.default_rng(5)
    p = Problem(n_heads=1, n_kv_heads=1, n_q=10, n_k=50, d=8, k=4, m=3)
    Q = rng.standard_normal((1, 10, 8)).astype(np.float32)
    K = rng.standard_normal((1, 50, 8)).astype(np.float32)
    b = oracle.route_bounds(p, Q, K)
    S = Q[0].astype(np.float64) @ K[0].astype(np.float64).T
    for i in range(10):
        srt = np.sort(S[i])[::-1]
        np.testing.assert_allclose(b[i, :4], [srt[3], srt[4], srt[6], srt[7]], rtol=1e-12)
        assert np.all(b[i, 4:] >= np.abs(b[i, :4]) - 1e-12)


def test_ledger_memory_figure():
    """Sec. 4.4: a 32-bit ledger with n_q = 1024 and c = k+m+r = 64 takes 256 KB."""
    p = Problem(n_heads=1, n_kv_heads=1, n_q=1024, n_k=1024, d=16, k=32, m=16, r=16)
    led = oracle.new_ledger(p)
    assert led["routes"].nbytes + led["sent"].nbytes == 256 * 1024
