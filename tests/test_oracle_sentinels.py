"""Pins of the oracle's random-sentinel sampler: the published splitmix64
outputs, without-replacement validity, uniformity (chi-square) and the miss
probability of Sec. 3.4, Eq. (10)."""
import dataclasses
import math
import os

import numpy as np
import pytest
from scipy import stats

import oracle
from oracle import Problem

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_splitmix64_published_outputs():
    vals = [int(x, 16) for x in open(os.path.join(GOLDEN, "splitmix64_seed0.txt"))
            if x.strip() and not x.startswith("#")]
    golden_inc = 0x9E3779B97F4A7C15
    for n, want in enumerate(vals):
        assert oracle.splitmix64((n * golden_inc) & 0xFFFFFFFFFFFFFFFF) == want


def test_probe_hash_is_chained_output_function():
    f = oracle.splitmix64
    for args in [(0, 0, 0, 0, 0), (12345, 7, 99999, 3, 63), (2**64 - 1, 31, 131071, 31, 64)]:
        s, l, r, sl, t = args
        assert oracle.probe_hash(*args) == f(f(f(f(f(s) ^ l) ^ r) ^ sl) ^ t)


def _draw(p, layer, row, ni, R, N):
    return oracle.random_sentinels(p, layer, row, ni, R, N)


def test_sentinels_valid_and_deterministic():
    p = Problem(1, 1, 1, 100, 4, k=10, m=5, r=8, seed=42)
    R = list(range(0, 20, 2))
    N = [1, 3, 5, 7, 9]
    pool = sorted(set(range(100)) - set(R) - set(N))
    for row in range(200):
        out = _draw(p, 3, row, 100, R, N)
        assert len(set(out.tolist())) == 8
        assert set(out.tolist()) <= set(pool)
        np.testing.assert_array_equal(out, _draw(p, 3, row, 100, R, N))
    a = _draw(p, 3, 0, 100, R, N)
    assert not np.array_equal(a, _draw(dataclasses.replace(p, seed=43), 3, 0, 100, R, N))
    assert not np.array_equal(a, _draw(p, 4, 0, 100, R, N))


def test_small_pool_taken_whole_in_order():
    p = Problem(1, 1, 1, 12, 4, k=6, m=3, r=5, seed=1)
    R = [0, 2, 4, 6, 8, 10]
    N = [1, 3, 5]
    out = _draw(p, 0, 7, 12, R, N)
    np.testing.assert_array_equal(out, [7, 9, 11, -1, -1])
    # causal row with fewer valid chunks than k + m: empty pool
    out = _draw(p, 0, 7, 5, [0, 1, 2, 3, 4], [])
    np.testing.assert_array_equal(out, [-1] * 5)


def test_uniform_over_pool_chi_square():
    """Every pool chunk is drawn with the same probability r/|P|."""
    p = Problem(1, 1, 1, 64, 4, k=8, m=6, r=5, seed=9)
    R = list(range(8))
    N = list(range(8, 14))
    pool = list(range(14, 64))
    counts = np.zeros(64)
    first = np.zeros(64)
    trials = 6000
    for row in range(trials):
        out = _draw(p, 1, row, 64, R, N)
        counts[out] += 1
        first[out[0]] += 1
    assert counts[:14].sum() == 0
    exp = trials * 5 / len(pool)
    chi = stats.chisquare(counts[14:], np.full(len(pool), exp))
    assert chi.pvalue > 1e-4, chi
    chi1 = stats.chisquare(first[14:], np.full(len(pool), trials / len(pool)))
    assert chi1.pvalue > 1e-4, chi1


def _draw_by_definition(p, layer, row, ni, R, N):
    """The sampling rule restated from the hash alone (the probe hash is pinned
    to the published splitmix64 outputs above)."""
    pool = [j for j in range(ni) if j not in set(R) | set(N)]
    if len(pool) <= p.r:
        return pool + [-1] * (p.r - len(pool))
    out = []
    rem = list(pool)
    for s in range(p.r):
        if 2 * len(pool) <= ni:
            y = oracle.probe_hash(p.seed, layer, row, s, 0) % (len(pool) - s)
            x = rem[y]
        else:
            x = None
            for t in range(64):
                cand = oracle.probe_hash(p.seed, layer, row, s, t) % ni
                if cand in rem:
                    x = cand
                    break
            if x is None:
                x = rem[oracle.probe_hash(p.seed, layer, row, s, 64) % len(rem)]
        rem.remove(x)
        out.append(x)
    return out


@pytest.mark.parametrize("ni,nR,nN", [(100, 10, 5), (64, 20, 12), (40, 12, 8), (200, 60, 45), (33, 8, 8)])
def test_draw_matches_definition(ni, nR, nN):
    """Both regimes (rank sampling for pools of at most half the valid chunks,
    rejection otherwise), slot by slot, on many rows."""
    p = Problem(1, 1, 1, ni, 4, k=nR, m=nN, r=9, seed=77)
    rng = np.random.default_rng(ni)
    for row in range(60):
        perm = rng.permutation(ni)
        R, N = sorted(perm[:nR].tolist()), sorted(perm[nR:nR + nN].tolist())
        want = _draw_by_definition(p, 5, row, ni, R, N)
        np.testing.assert_array_equal(_draw(p, 5, row, ni, R, N), want)


def test_rank_regime_uniform():
    """A pool of 10 among 1000 valid chunks is sampled by rank; the draw is
    uniform over the pool and without replacement."""
    p = Problem(1, 1, 1, 1000, 4, k=500, m=490, r=4, seed=5)
    R = list(range(0, 1000, 2))
    N = [j for j in range(1, 1000, 2)][:490]
    pool = sorted(set(range(1000)) - set(R) - set(N))
    assert len(pool) == 10
    counts = np.zeros(1000)
    for row in range(3000):
        out = _draw(p, 0, row, 1000, R, N)
        assert len(set(out.tolist())) == 4 and set(out.tolist()) <= set(pool)
        counts[out] += 1
    chi = stats.chisquare(counts[pool], np.full(10, 3000 * 4 / 10))
    assert chi.pvalue > 1e-4, chi


@pytest.mark.parametrize("N_pool,u,r", [(40, 3, 6), (100, 10, 12), (60, 1, 12)])
def test_miss_probability_eq10(N_pool, u, r):
    """Eq. (10): drawing r of N pool chunks without replacement misses all u
    planted challengers with probability C(N-u, r) / C(N, r) <= (1 - u/N)^r."""
    k, m = 6, 4
    n = k + m + N_pool
    p = Problem(1, 1, 1, n, 4, k=k, m=m, r=r, seed=2024)
    R = list(range(k))
    Nn = list(range(k, k + m))
    challengers = set(range(n - u, n))
    trials = 20000
    miss = 0
    for row in range(trials):
        out = set(_draw(p, 0, row, n, R, Nn).tolist())
        miss += not (out & challengers)
    pm = math.comb(N_pool - u, r) / math.comb(N_pool, r)
    assert pm <= (1 - u / N_pool) ** r + 1e-12
    sd = math.sqrt(pm * (1 - pm) / trials)
    assert abs(miss / trials - pm) < 5 * sd + 1e-9, (miss / trials, pm)
