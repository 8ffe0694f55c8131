"""Pins of the oracle's query-dependent route budgets (Sec. 4.3: the ledger
stores whichever route width the policy requests; Sec. 4.4: ledgers bucketed
by route width): row i routes to its top k_i chunks."""
import dataclasses
import math

import numpy as np
import pytest

import oracle
from oracle import Problem
from paper_2609_07306_amd import synth


def _lexsort_topk(Q, K, p, row, ki):
    """The k_i best valid chunks of a row by (score desc, id asc), from numpy's
    lexsort on binary64 scores."""
    h, i = divmod(row, p.n_q)
    g = h // (p.n_heads // p.n_kv_heads)
    ni = p.n_valid(i)
    s = K[g, :ni].astype(np.float64) @ Q[h, i].astype(np.float64)
    order = np.lexsort((np.arange(ni), -s))
    return sorted(order[:min(ki, ni)].tolist()), sorted(order[min(ki, ni):min(ki, ni) + p.m].tolist())


@pytest.mark.parametrize("causal", [False, True])
def test_per_row_widths_match_lexsort(causal):
    rng = np.random.default_rng(21)
    H, n, d, k, m = 3, 50, 16, 9, 4
    Q = rng.standard_normal((H, n, d)).astype(np.float32)
    K = rng.standard_normal((1, n, d)).astype(np.float32)
    kr = rng.integers(1, k + 1, size=H * n).astype(np.int32)
    p = Problem(H, 1, n, n, d, k, m, 3, causal, k_rows=kr)
    routes, _ = oracle.full_route(p, Q, K)
    led = oracle.new_ledger(p)
    oracle.anchor(p, 0, Q, K, led)
    for row in range(p.rows):
        R, N = _lexsort_topk(Q, K, p, row, kr[row])
        got = [x for x in routes[row] if x >= 0]
        assert got == R and all(x == -1 for x in routes[row][len(got):])
        assert [x for x in led["routes"][row] if x >= 0] == R
        assert [x for x in led["sent"][row, :m] if x >= 0] == N


def test_uniform_widths_equal_the_scalar_width():
    w = synth.preset("tiny", rho=0.3, n_layers=4)
    p = Problem(1, 1, w.n, w.n, w.d, w.k, w.m, w.r)
    pk = dataclasses.replace(p, k_rows=np.full(p.rows, w.k, np.int32))
    L = synth.layers(w)
    a, b = oracle.new_ledger(p), oracle.new_ledger(pk)
    for layer, (Qf, Kf, _, _) in enumerate(L):
        if layer == 0:
            oracle.anchor(p, 0, Qf, Kf, a)
            oracle.anchor(pk, 0, Qf, Kf, b)
        else:
            oa, ob = oracle.relay(p, layer, Qf, Kf, a), oracle.relay(pk, layer, Qf, Kf, b)
            np.testing.assert_array_equal(oa["mask"], ob["mask"])
            assert oa["pairs"] == ob["pairs"]
        for key in a:
            np.testing.assert_array_equal(a[key], b[key])


def test_forced_refresh_with_budgets_is_full_routing():
    """With gamma = +inf every row with a sentinel refreshes to its exact top
    k_i; alpha is the minimum over its k_i routed chunks."""
    w = synth.preset("tiny", rho=0.6, n_layers=3)
    kr = (np.arange(w.rows) % w.k + 1).astype(np.int32)
    p = Problem(1, 1, w.n, w.n, w.d, w.k, w.m, w.r, False, math.inf, k_rows=kr)
    L = synth.layers(w)
    led = oracle.new_ledger(p)
    oracle.anchor(p, 0, L[0][0], L[0][1], led)
    for layer in (1, 2):
        Qf, Kf = L[layer][0], L[layer][1]
        before = led["routes"].copy()
        out = oracle.relay(p, layer, Qf, Kf, led)
        exact, _ = oracle.full_route(p, Qf, Kf)
        np.testing.assert_array_equal(led["routes"], exact)
        assert out["mask"].all()
        # alpha: the smallest current score of the route the layer started from
        for row in (0, 5, w.rows - 1):
            ids = [x for x in before[row] if x >= 0]
            assert len(ids) == kr[row]
            s = Kf[0, ids].astype(np.float64) @ Qf[0, row].astype(np.float64)
            assert out["alpha"][row] == pytest.approx(s.min(), rel=1e-12, abs=1e-15)


def test_route_bounds_follow_the_row_width():
    rng = np.random.default_rng(4)
    n, d, k = 40, 8, 6
    Q = rng.standard_normal((1, n, d)).astype(np.float32)
    K = rng.standard_normal((1, n, d)).astype(np.float32)
    kr = np.full(n, 2, np.int32)
    p = Problem(1, 1, n, n, d, k, 3, 0, k_rows=kr)
    b = oracle.route_bounds(p, Q, K)
    s = np.sort(K[0].astype(np.float64) @ Q[0, 7].astype(np.float64))[::-1]
    assert b[7, 0] == s[1] and b[7, 1] == s[2] and b[7, 2] == s[4] and b[7, 3] == s[5]
