"""Pins of the oracle's sentinel and trigger variants (Sec. 3.1 item 3;
Sec. 3.2 Eq. (8) with gamma_i; Sec. 3.2 Hysteresis): the mandatory sink and
recent sentinels, per-row guard margins and the minimum reuse horizon."""
import dataclasses
import math

import numpy as np
import pytest

import oracle
from oracle import Problem
from paper_2609_07306_amd import synth


def rollout(p, w, layers=None):
    L = synth.layers(w)
    led = oracle.new_ledger(p)
    outs = []
    for layer, (Qf, Kf, _, _) in enumerate(L[: layers or len(L)]):
        if layer == 0:
            oracle.anchor(p, 0, Qf, Kf, led)
            outs.append(None)
        else:
            outs.append(oracle.relay(p, layer, Qf, Kf, led))
    return led, outs, L


@pytest.mark.parametrize("causal", [False, True])
def test_mandatory_sentinel_sets(causal):
    """After an anchor every row's mandatory slots hold, ascending and -1
    padded, exactly the valid sink chunks j < n_sink and recent chunks (the
    n_recent valid chunks up to the row's position) that are not already in
    R or N; random sentinels avoid them."""
    w = synth.preset("tiny", causal=causal, n=64, k=5, m=3, r=4, n_layers=1)
    p = Problem(1, 1, 64, 64, w.d, 5, 3, 4, causal, 0.0, 0, n_sink=2, n_recent=3)
    led, _, _ = rollout(p, w)
    for row in range(p.rows):
        i = row % p.n_q
        ni = p.n_valid(i)
        R = set(x for x in led["routes"][row] if x >= 0)
        N = set(x for x in led["sent"][row, :3] if x >= 0)
        rand = [x for x in led["sent"][row, 3:7] if x >= 0]
        mand = led["sent"][row, 7:]
        pos = min(i, ni - 1)
        want = sorted(({j for j in range(min(2, ni))} | {j for j in range(max(0, pos - 2), pos + 1)}) - R - N)
        got = [x for x in mand if x >= 0]
        assert got == want, (row, got, want)
        assert all(x == -1 for x in mand[len(got):])
        assert not (set(rand) & (R | N | set(got)))
        assert len(rand) == min(4, ni - len(R) - len(N) - len(got))


def _planted(n_sink, n_recent, chunk):
    """One row whose best chunk at layer 1 is `chunk`, a chunk with a low score
    at layer 0; no random sentinels, so only a mandatory sentinel can see it."""
    rng = np.random.default_rng(3)
    n, d = 32, 16
    q = rng.standard_normal(d).astype(np.float32)
    K0 = rng.standard_normal((n, d)).astype(np.float32)
    K0[chunk] = -2.0 * q  # far below the cut at layer 0
    K1 = K0.copy()
    K1[chunk] = 3.0 * q   # the best chunk at layer 1
    Q = np.tile(q, (1, n, 1)).astype(np.float32)
    p = Problem(1, 1, n, n, d, 4, 2, 0, False, 0.0, 0, n_sink=n_sink, n_recent=n_recent)
    led = oracle.new_ledger(p)
    oracle.anchor(p, 0, Q, K0[None], led)
    row = n - 1
    # not routed, not a near-miss; only a mandatory slot may hold it
    assert chunk not in led["routes"][row] and chunk not in led["sent"][row, : p.m + p.r]
    assert (chunk in led["sent"][row, p.m + p.r:]) == (n_sink + n_recent > 0)
    out = oracle.relay(p, 1, Q, K1[None], led)
    exact, _ = oracle.full_route(p, Q, K1[None])
    return out["mask"][row], chunk in led["routes"][row], oracle.recall(led["routes"][row:], exact[row:])


def test_sink_sentinel_catches_a_challenger():
    """A chunk that overtakes the route is invisible without a sentinel on it
    (the route is kept, recall drops); as a mandatory sink sentinel it
    triggers the refresh that brings it into the route."""
    mask0, in0, rec0 = _planted(0, 0, 0)
    assert mask0 == 0 and not in0 and rec0 < 1.0
    mask1, in1, rec1 = _planted(1, 0, 0)
    assert mask1 == 1 and in1 and rec1 == 1.0


def test_recent_sentinel_catches_a_challenger():
    """The same with the row's most recent chunk (its own position)."""
    mask0, in0, _ = _planted(0, 0, 31)
    assert mask0 == 0 and not in0
    mask1, in1, rec1 = _planted(0, 1, 31)
    assert mask1 == 1 and in1 and rec1 == 1.0


@pytest.mark.parametrize("causal", [False, True])
def test_per_row_gamma(causal):
    """gamma_i = +inf refreshes exactly the rows with a sentinel, -inf none,
    row by row; equal margins reproduce the scalar gamma."""
    w = synth.preset("tiny", causal=causal, rho=0.3, n_layers=3)
    base = Problem(1, 1, w.n, w.n, w.d, w.k, w.m, w.r, causal, 0.05, 0)
    sel = (np.arange(base.rows) % 3) == 0
    g = np.where(sel, math.inf, -math.inf)
    p = dataclasses.replace(base, gamma_rows=g)
    led, outs, _ = rollout(p, w)
    ref, routs, _ = rollout(base, w)
    assert outs[1] is not None
    # a row with no sentinel (causal rows with n_i <= k) is never refreshed
    has_sent = np.array([p.n_valid(i % p.n_q) > p.k for i in range(p.rows)])
    for layer in (1, 2):
        np.testing.assert_array_equal(outs[layer]["mask"].astype(bool), sel & has_sent)
    same = dataclasses.replace(base, gamma_rows=np.full(base.rows, 0.05))
    led2, outs2, _ = rollout(same, w)
    for key in ("routes", "sent", "build", "age"):
        np.testing.assert_array_equal(led2[key], ref[key])
    for a, b in zip(outs2[1:], routs[1:]):
        np.testing.assert_array_equal(a["mask"], b["mask"])


def test_minimum_reuse_horizon():
    """With a horizon of h layers a row (re)built at layer b keeps its route
    at b+1 .. b+h whatever its scores; h = 0 is the plain trigger."""
    w = synth.preset("tiny", rho=0.6, n_layers=6)
    base = Problem(1, 1, w.n, w.n, w.d, w.k, w.m, w.r, False, 0.0, 0)
    h1 = dataclasses.replace(base, min_reuse=1)
    h2 = dataclasses.replace(base, min_reuse=2)
    for p, h in ((h1, 1), (h2, 2)):
        L = synth.layers(w)
        led = oracle.new_ledger(p)
        oracle.anchor(p, 0, L[0][0], L[0][1], led)
        for layer in range(1, 6):
            before = led["build"].copy()
            out = oracle.relay(p, layer, L[layer][0], L[layer][1], led)
            young = layer - before <= h
            assert not out["mask"][young].any()
            assert (led["build"][young] == before[young]).all()
            if layer > h:
                assert out["mask"].any()  # high drift: old rows do refresh
    led0, outs0, _ = rollout(base, w)
    led00, outs00, _ = rollout(dataclasses.replace(base, min_reuse=0), w)
    for key in ("routes", "sent", "build", "age"):
        np.testing.assert_array_equal(led0[key], led00[key])
