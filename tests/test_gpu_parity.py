"""GPU parity of the HIP path with the oracle, through the C ABI.

Routes, near-miss and random sentinels, masks, ages and score-pair counts are
compared bit-exactly on every row whose outcome does not hinge on a near-tie
(see parity_util); scores within 1e-5 (binary32 inputs) or 2e-3 (bf16 inputs)
of the oracle relative to sum_t |q_t k_t|.
"""
import math
import sys
import zlib

import numpy as np
import pytest
import torch

import oracle
from paper_2609_07306_amd import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    torch.cuda.set_device(0)
    yield


def rrmod():
    from paper_2609_07306_amd import routerelay
    return routerelay


def note(msg):
    print(msg, flush=True)
    sys.stdout.flush()


# ------------------------------------------------------------ full routing

FULL_CASES = [
    # name, H, Hkv, n_q, n_k, d, dtype, k, causal
    ("tiny_f32", 1, 1, 128, 128, 64, "f32", 8, False),
    ("ragged_f32", 3, 1, 100, 77, 32, "f32", 5, False),
    ("ragged_causal", 2, 2, 70, 70, 64, "f32", 9, True),
    ("drift_f32", 2, 2, 256, 256, 128, "f32", 16, False),
    ("bf16_d128", 4, 2, 160, 300, 128, "bf16", 32, False),
    ("bf16_causal_gqa", 4, 1, 200, 200, 128, "bf16", 32, True),
    ("bf16_d256", 2, 2, 64, 96, 256, "bf16", 12, False),
    ("bf16_d32_k_eq_nk", 1, 1, 40, 20, 32, "bf16", 20, False),
    ("wide_k", 2, 2, 64, 512, 128, "bf16", 100, False),
    # rows just past a tile boundary of a causal head: one half of the key
    # range holds nearly every valid chunk, so its sub-list overflows
    ("causal_overflow_k48", 8, 2, 256, 256, 128, "bf16", 48, True),
]


def _inputs(rng, H, Hkv, n_q, n_k, d, dtype):
    Q = (rng.standard_normal((H, n_q, d)) / np.sqrt(d)).astype(np.float32)
    K = (rng.standard_normal((Hkv, n_k, d)) / np.sqrt(d)).astype(np.float32)
    if dtype == "bf16":
        Qd, Kd = synth.bf16_round(Q), synth.bf16_round(K)
        return synth.bf16_widen(Qd), synth.bf16_widen(Kd), Qd, Kd
    return Q, K, Q, K


@pytest.mark.parametrize("case", FULL_CASES, ids=[c[0] for c in FULL_CASES])
def test_full_route_parity(case):
    from parity_util import dev, route_ties, TOL
    rr = rrmod()
    name, H, Hkv, n_q, n_k, d, dtype, k, causal = case
    note(f"full route parity: {case}")
    rng = np.random.default_rng(zlib.crc32(name.encode()))
    Qf, Kf, Qd, Kd = _inputs(rng, H, Hkv, n_q, n_k, d, dtype)
    cfg = rr.Config(H, Hkv, n_q, n_k, d, k, 0, 0, dtype, causal)
    p = oracle.Problem(H, Hkv, n_q, n_k, d, k, 0, 0, causal)
    routes = torch.full((cfg.rows, k), -7, dtype=torch.int32, device="cuda")
    scores = torch.zeros((cfg.rows, k), dtype=torch.float32, device="cuda")
    pairs = torch.zeros(1, dtype=torch.int64, device="cuda")
    rr.full_route(cfg, dev(Qd, dtype), dev(Kd, dtype), routes, scores, pairs)
    torch.cuda.synchronize()
    exact, opairs, osc = oracle.full_route(p, Qf, Kf, with_scores=True)
    t1, _ = route_ties(p, Qf, Kf)
    got = routes.cpu().numpy()
    assert int(pairs.item()) == opairs
    assert t1.mean() < 0.05
    bad = np.flatnonzero((got != exact).any(1) & ~t1)
    assert len(bad) == 0, f"rows {bad[:8]}: {got[bad[:2]]} vs {exact[bad[:2]]}"
    # scores of agreeing rows, relative to sum_t |q_t k_t|
    sc = scores.cpu().numpy()
    ok = ~t1
    valid = exact >= 0
    for row in np.flatnonzero(ok)[:400]:
        h, i = divmod(row, n_q)
        g = h // (H // Hkv)
        ids = exact[row][valid[row]]
        absd = np.abs(Qf[h, i].astype(np.float64)[None, :] * Kf[g, ids].astype(np.float64)).sum(1)
        assert np.all(np.abs(sc[row][valid[row]] - osc[row][valid[row]]) <= TOL[dtype] * absd)
        assert np.all(np.isneginf(sc[row][~valid[row]]))


def test_full_route_exact_ties_integer_data():
    """Small-integer inputs make every score exact in binary32, so the GPU and
    the oracle see identical scores with massive exact ties: every row must
    match, exercising the lower-id tie-break and the overflow repair."""
    from parity_util import dev
    rr = rrmod()
    rng = np.random.default_rng(5)
    for dtype in ("f32", "bf16"):
        for causal in (False, True):
            H, n, d, k = 2, 300, 32, 24
            Q = rng.integers(-2, 3, size=(H, n, d)).astype(np.float32)
            K = rng.integers(-1, 2, size=(H, n, d)).astype(np.float32)
            note(f"integer ties: {dtype} causal={causal}")
            Qd = synth.bf16_round(Q) if dtype == "bf16" else Q
            Kd = synth.bf16_round(K) if dtype == "bf16" else K
            cfg = rr.Config(H, H, n, n, d, k, 0, 0, dtype, causal)
            routes = torch.empty((cfg.rows, k), dtype=torch.int32, device="cuda")
            rr.full_route(cfg, dev(Qd, dtype), dev(Kd, dtype), routes)
            torch.cuda.synchronize()
            exact, _ = oracle.full_route(oracle.Problem(H, H, n, n, d, k, causal=causal), Q, K)
            np.testing.assert_array_equal(routes.cpu().numpy(), exact)


def test_all_zero_scores_pick_lowest_ids():
    from parity_util import dev
    rr = rrmod()
    H, n, d, k, m, r = 1, 200, 64, 10, 5, 5
    Q = np.zeros((H, n, d), np.float32)
    K = np.random.default_rng(1).standard_normal((H, n, d)).astype(np.float32)
    cfg = rr.Config(H, H, n, n, d, k, m, r, "f32", False)
    L = rr.Ledger(cfg)
    L.anchor(0, dev(Q, "f32"), dev(K, "f32"))
    from parity_util import ledger_np
    got = ledger_np(L)
    ref = oracle.new_ledger(oracle.Problem(H, H, n, n, d, k, m, r))
    oracle.anchor(oracle.Problem(H, H, n, n, d, k, m, r), 0, Q, K, ref)
    assert (got["routes"] == np.arange(k)).all()
    for key in ("routes", "sent", "build", "age"):
        np.testing.assert_array_equal(got[key], ref[key])
    L.close()


@pytest.mark.parametrize("T_class", ["narrow", "wide"])
@pytest.mark.parametrize("causal", [False, True])
def test_ledger_exact_ties_integer_data(T_class, causal):
    """Anchor, then a relay, on small-integer inputs: every score is exact in
    binary32 on both sides, so the whole ledger (routes, near-miss and random
    sentinels, ages), the mask and alpha / beta must match the oracle on every
    row.  Massive exact ties make the collection sub-lists overflow, which
    drives the bisection repair and its (score, id) tie cut."""
    from parity_util import dev, ledger_np
    rr = rrmod()
    rng = np.random.default_rng(11 if causal else 12)
    H, n, d = 2, 300, 32
    k, m, r = (24, 12, 8) if T_class == "narrow" else (60, 30, 20)
    note(f"integer-tie ledger: {T_class} causal={causal}")
    p = oracle.Problem(H, H, n, n, d, k, m, r, causal, seed=7)
    cfg = rr.Config(H, H, n, n, d, k, m, r, "f32", causal, seed=7)
    L = rr.Ledger(cfg)
    ref = oracle.new_ledger(p)
    for layer in range(3):
        Q = rng.integers(-2, 3, size=(H, n, d)).astype(np.float32)
        K = rng.integers(-1, 2, size=(H, n, d)).astype(np.float32)
        if layer == 0:
            L.anchor(layer, dev(Q, "f32"), dev(K, "f32"))
            oracle.anchor(p, layer, Q, K, ref)
        else:
            mask = torch.empty(cfg.rows, dtype=torch.uint8, device="cuda")
            L.relay(layer, dev(Q, "f32"), dev(K, "f32"), mask=mask)
            out = oracle.relay(p, layer, Q, K, ref)
            np.testing.assert_array_equal(mask.cpu().numpy(), out["mask"])
            alpha, beta, _ = L.relay_stats()
            np.testing.assert_array_equal(alpha.cpu().numpy(), out["alpha"].astype(np.float32))
            np.testing.assert_array_equal(beta.cpu().numpy(), out["beta"].astype(np.float32))
        got = ledger_np(L)
        for key in ("routes", "sent", "build", "age"):
            np.testing.assert_array_equal(got[key], ref[key], err_msg=f"layer {layer} {key}")
    L.close()


@pytest.mark.parametrize("n,k,m,r,causal", [(600, 10, 5, 5, False), (600, 40, 60, 16, True),
                                            (1000, 32, 16, 16, True)])
def test_all_zero_scores_overflow(n, k, m, r, causal):
    """All scores zero: every chunk reaches every threshold, both sub-lists
    overflow, and the result is the lowest ids (R = 0..k-1, N = k..k+m-1)."""
    from parity_util import dev, ledger_np
    rr = rrmod()
    H, d = 2, 64
    note(f"all-zero overflow: n={n} k={k} m={m} r={r} causal={causal}")
    Q = np.zeros((H, n, d), np.float32)
    K = np.random.default_rng(3).standard_normal((H, n, d)).astype(np.float32)
    p = oracle.Problem(H, H, n, n, d, k, m, r, causal)
    cfg = rr.Config(H, H, n, n, d, k, m, r, "f32", causal)
    L = rr.Ledger(cfg)
    L.anchor(0, dev(Q, "f32"), dev(K, "f32"))
    got = ledger_np(L)
    ref = oracle.new_ledger(p)
    oracle.anchor(p, 0, Q, K, ref)
    for key in ("routes", "sent", "build", "age"):
        np.testing.assert_array_equal(got[key], ref[key], err_msg=key)
    L.close()


# ------------------------------------------------------- rollout parity

ROLLOUTS = [
    ("tiny", {}),
    ("tiny", {"causal": True, "n_layers": 6, "anchor_every": 4}),
    ("drift", {"rho": 0.1}),
    ("drift", {"rho": 0.3}),
    ("drift", {"rho": 0.6}),
    ("scale", {"n_heads": 4, "n_kv_heads": 4, "n": 256, "n_layers": 10}),
    ("gqa", {"n_heads": 8, "n_kv_heads": 2, "n": 256, "n_layers": 10}),
    ("longctx", {"n_heads": 2, "n_kv_heads": 2, "n": 512, "n_layers": 10}),
    ("tiny", {"n": 100, "d": 32, "k": 5, "m": 3, "r": 2, "n_heads": 4, "n_kv_heads": 2, "n_layers": 5}),
    ("tiny", {"n": 100, "d": 32, "k": 5, "m": 3, "r": 2, "n_heads": 4, "n_kv_heads": 2, "n_layers": 5,
              "causal": True, "dtype": "bf16"}),
    ("tiny", {"m": 0, "r": 6, "n_layers": 4}),
    ("tiny", {"m": 6, "r": 0, "n_layers": 4}),
    # enough 128-row tiles (one per compute unit) for the dense MFMA rescoring,
    # for each input type and d (d = 256 bf16 takes the single-buffered sweep)
    ("scale", {"n_heads": 256, "n_kv_heads": 256, "n": 128, "n_layers": 6}),
    ("gqa", {"n_heads": 256, "n_kv_heads": 64, "n": 128, "n_layers": 6}),
    ("drift", {"n_heads": 256, "n_kv_heads": 256, "n": 128, "n_layers": 4, "anchor_every": 2}),
    ("drift", {"n_heads": 256, "n_kv_heads": 128, "n": 160, "d": 32, "n_layers": 4, "anchor_every": 2,
               "causal": True}),
    ("scale", {"n_heads": 256, "n_kv_heads": 256, "n": 128, "d": 64, "n_layers": 4, "anchor_every": 2}),
    ("scale", {"n_heads": 256, "n_kv_heads": 256, "n": 128, "d": 256, "n_layers": 4, "anchor_every": 2}),
    # dense rescoring with no near-miss slots, with no random slots, and with
    # the wide route class (k + m > 64, 64-row route tiles)
    ("scale", {"n_heads": 256, "n_kv_heads": 256, "n": 128, "m": 0, "n_layers": 4, "anchor_every": 2}),
    ("scale", {"n_heads": 256, "n_kv_heads": 256, "n": 128, "r": 0, "n_layers": 4, "anchor_every": 2}),
    ("scale", {"n_heads": 256, "n_kv_heads": 256, "n": 192, "k": 48, "m": 24, "r": 8, "n_layers": 4,
               "anchor_every": 2}),
    # dense rescoring in 64-row tiles (fewer 128-row tiles than compute
    # units), with a ragged last tile in the causal case
    ("scale", {"n_heads": 64, "n_kv_heads": 64, "n": 256, "n_layers": 4, "anchor_every": 2}),
    ("gqa", {"n_heads": 64, "n_kv_heads": 16, "n": 160, "n_layers": 4, "anchor_every": 2}),
    # the fidelity studies' shapes: sentinel ablation with no near-miss
    # slots and with no random slots; 384 query rows against 192 key chunks
    ("ablation", {"m": 0, "r": 12, "rho": 0.05, "n_layers": 8}),
    ("ablation", {"m": 24, "r": 0, "rho": 0.05, "n_layers": 8}),
    ("stride", {"rho": 0.2, "n_layers": 8}),
]


@pytest.mark.parametrize("name,kw", ROLLOUTS, ids=[f"{n}-{i}" for i, (n, _) in enumerate(ROLLOUTS)])
def test_rollout_parity(name, kw):
    from parity_util import rollout_compare
    w = synth.preset(name, **kw)
    note(f"rollout parity: {name} {kw}")
    st = rollout_compare(w)
    note(f"  {st}")
    assert st["compared"] >= 0.8 * st["rows"]


# the same schedules with each relay schedule forced: the split one
# (rescoring kernel, then the reroute of the flagged rows compacted per head)
# and the one pass
FORCED_PATH_ROLLOUTS = [ROLLOUTS[i] for i in (0, 1, 3, 6, 7, 9, 10, 11, 12, 13, 15, 17, 18, 20, 21, 22)]


@pytest.mark.parametrize("relay", ["split", "one_pass"])
@pytest.mark.parametrize("name,kw", FORCED_PATH_ROLLOUTS,
                         ids=[f"{n}-{i}" for i, (n, _) in enumerate(FORCED_PATH_ROLLOUTS)])
def test_rollout_parity_forced_relay_path(name, kw, relay):
    from parity_util import rollout_compare
    w = synth.preset(name, **kw)
    note(f"rollout parity ({relay} relay): {name} {kw}")
    st = rollout_compare(w, relay=relay)
    note(f"  {st}")
    assert st["compared"] >= 0.8 * st["rows"]


# Sentinel and trigger variants (Sec. 3.1 item 3; Sec. 3.2 Eq. (8) with
# per-row margins and the hysteresis horizon): mandatory sink and recent
# sentinels on both relay schedules, non-causal and causal, dense and gather
# rescoring, the wide route class, key ranges past the exact draw bitmap
# (n_k > 4096), and the minimum reuse horizon.
VARIANT_ROLLOUTS = [
    ("tiny", {"n_sink": 2, "n_recent": 3, "n_layers": 5}),
    ("tiny", {"n_sink": 1, "n_recent": 2, "causal": True, "n_layers": 5}),
    ("drift", {"n_sink": 4, "n_recent": 4, "n_heads": 4, "n_kv_heads": 4, "n_layers": 6}),
    ("scale", {"n_heads": 256, "n_kv_heads": 256, "n": 128, "n_sink": 2, "n_recent": 2, "n_layers": 4,
               "anchor_every": 2}),
    ("gqa", {"n_heads": 8, "n_kv_heads": 2, "n": 256, "n_sink": 1, "n_recent": 4, "min_reuse": 1,
             "n_layers": 8}),
    ("longctx", {"n_heads": 2, "n_kv_heads": 2, "n": 512, "n_sink": 2, "n_recent": 2, "n_layers": 6}),
    ("scale", {"n": 4608, "n_heads": 1, "n_kv_heads": 1, "d": 32, "n_sink": 2, "n_recent": 3, "n_layers": 3,
               "anchor_every": 2}),
    ("drift", {"n_heads": 4, "n_kv_heads": 4, "n_layers": 6, "rho": 0.6, "min_reuse": 2}),
]


@pytest.mark.parametrize("relay", ["split", "one_pass"])
@pytest.mark.parametrize("name,kw", VARIANT_ROLLOUTS, ids=[f"{n}-{i}" for i, (n, _) in enumerate(VARIANT_ROLLOUTS)])
def test_rollout_parity_sentinel_variants(name, kw, relay):
    from parity_util import rollout_compare
    w = synth.preset(name, **kw)
    if relay == "one_pass" and w.nk > 2048:
        pytest.skip("the one-pass relay holds its tile's ledger bitmaps up to about 2048 key chunks")
    note(f"variant rollout parity ({relay} relay): {name} {kw}")
    st = rollout_compare(w, relay=relay)
    note(f"  {st}")
    assert st["compared"] >= 0.8 * st["rows"]


@pytest.mark.parametrize("relay", ["split", "one_pass"])
def test_rollout_parity_per_row_gamma(relay):
    """Per-row guard margins gamma_i: a mix of 0, small positive, +inf and
    -inf margins, with the reuse horizon on."""
    from parity_util import rollout_compare
    w = synth.preset("drift", n_heads=4, n_kv_heads=4, n_layers=6, rho=0.3, min_reuse=1, n_sink=1, n_recent=1)
    g = np.random.default_rng(9).choice(np.array([0.0, 0.01, 0.05, math.inf, -math.inf], np.float32), size=w.rows)
    note(f"per-row gamma rollout ({relay})")
    st = rollout_compare(w, relay=relay, gamma_rows=g)
    note(f"  {st}")
    assert st["compared"] >= 0.8 * st["rows"] and st["rerouted"] > 0


@pytest.mark.parametrize("gamma", [math.inf, -math.inf, 0.05])
def test_forced_paths(gamma):
    """gamma = +inf refreshes every row (the relay equals full routing);
    gamma = -inf refreshes none (the reroute kernel finds no tiles)."""
    from parity_util import rollout_compare, dev, ledger_np
    rr = rrmod()
    w = synth.preset("drift", n_heads=2, n_kv_heads=2, n_layers=4, rho=0.6)
    note(f"forced path gamma={gamma}")
    rollout_compare(w, gamma=gamma)
    if math.isinf(gamma):
        w2 = w.with_(gamma=gamma)
        cfg = rr.Config.of(w2)
        L = rr.Ledger(cfg)
        lay = synth.layers(w2)
        L.anchor(0, dev(lay[0][2], w.dtype), dev(lay[0][3], w.dtype))
        before = ledger_np(L)
        mask = torch.empty(cfg.rows, dtype=torch.uint8, device="cuda")
        nrr = torch.zeros(1, dtype=torch.int32, device="cuda")
        Q1, K1 = dev(lay[1][2], w.dtype), dev(lay[1][3], w.dtype)
        L.relay(1, Q1, K1, mask=mask, n_rerouted=nrr)
        after = ledger_np(L)
        if gamma < 0:
            assert int(nrr.item()) == 0 and int(mask.sum().item()) == 0
            for key in ("routes", "sent", "build"):
                np.testing.assert_array_equal(after[key], before[key])
        else:
            assert int(nrr.item()) == cfg.rows
            full = torch.empty((cfg.rows, cfg.k), dtype=torch.int32, device="cuda")
            rr.full_route(cfg, Q1, K1, full)
            torch.cuda.synchronize()
            np.testing.assert_array_equal(after["routes"], full.cpu().numpy())
        L.close()


# ------------------------------------------- full-size sampled parity

FULL_SIZE = [
    ("scale", {}),
    ("scale", {"n": 128}),
    ("gqa", {}),
    ("drift", {"rho": 0.3}),
    ("longctx", {}),
    ("scale", {"n": 8192, "n_heads": 2, "n_kv_heads": 2}),
    ("longctx", {"n": 8192, "n_heads": 2, "n_kv_heads": 2}),
]


@pytest.mark.parametrize("name,kw", FULL_SIZE, ids=[f"{n}-{kw.get('n', '')}" for n, kw in FULL_SIZE])
def test_full_size_sampled(name, kw):
    """At the workload's real size, in the launch configuration the benchmark
    uses: an anchor, then a relay in step mode, checked on sampled rows."""
    from parity_util import dev, ledger_np, problem_of, route_ties, trigger_ties, TOL
    rr = rrmod()
    w = synth.preset(name, n_layers=2, **kw)
    note(f"full-size sampled: {w.name} n={w.n} heads={w.n_heads}")
    p = problem_of(w)
    cfg = rr.Config.of(w)
    gen = list(synth.Generator(w))
    rng = np.random.default_rng(0)
    rows = np.unique(np.concatenate([rng.choice(p.rows, 192, replace=False),
                                     [0, p.rows - 1, p.n_q - 1, p.n_q]]))
    L = rr.Ledger(cfg)
    _, Q0f, K0f, Q0d, K0d = gen[0]
    L.anchor(0, dev(Q0d, w.dtype), dev(K0d, w.dtype))
    got0 = ledger_np(L)
    ref = oracle.new_ledger(p)
    oracle.anchor(p, 0, Q0f, K0f, ref, rows=rows)
    t1, t2 = route_ties(p, Q0f, K0f, rows=rows)
    ok = rows[~(t1 | t2)]
    for key in ("routes", "sent", "build", "age"):
        np.testing.assert_array_equal(got0[key][ok], ref[key][ok])
    # step mode: the oracle relays the sampled rows from the GPU's ledger
    _, Q1f, K1f, Q1d, K1d = gen[1]
    mask = torch.empty(cfg.rows, dtype=torch.uint8, device="cuda")
    pairs = torch.zeros(1, dtype=torch.int64, device="cuda")
    L.relay(1, dev(Q1d, w.dtype), dev(K1d, w.dtype), mask=mask, pairs=pairs)
    got1 = ledger_np(L)
    led = {k: v.copy() for k, v in got0.items()}
    out = oracle.relay(p, 1, Q1f, K1f, led, rows=rows)
    gm = mask.cpu().numpy()
    t3 = trigger_ties(p, out)[rows]
    t1b, t2b = route_ties(p, Q1f, K1f, rows=rows)
    om = out["mask"][rows]
    dec = ~t3
    assert np.array_equal(gm[rows][dec], om[dec])
    same = dec & ~(om.astype(bool) & (t1b | t2b))
    for key in ("routes", "sent", "build", "age"):
        np.testing.assert_array_equal(got1[key][rows[same]], led[key][rows[same]])
    # alpha and beta of the sampled rows against the oracle's binary64 scores
    alpha, beta, _ = L.relay_stats()
    torch.cuda.synchronize()
    alpha, beta = alpha.cpu().numpy()[rows], beta.cpu().numpy()[rows]
    tol = TOL[w.dtype]
    oa, ob = out["alpha"][rows], out["beta"][rows]
    fa, fb = np.isfinite(oa), np.isfinite(ob)
    assert np.all(np.abs(alpha[fa] - oa[fa]) <= tol * out["alpha_abs"][rows][fa] + 1e-30)
    assert np.all(np.abs(beta[fb] - ob[fb]) <= tol * out["beta_abs"][rows][fb] + 1e-30)
    assert np.array_equal(np.isposinf(alpha), np.isposinf(oa)) and np.array_equal(np.isneginf(beta), np.isneginf(ob))
    cand = (got0["routes"] >= 0).sum(1) + (got0["sent"] >= 0).sum(1)
    ni = np.minimum(np.arange(p.rows) % p.n_q + 1, p.n_k) if p.causal else np.full(p.rows, p.n_k)
    assert int(pairs.item()) == int(cand.sum() + ni[gm.astype(bool)].sum())
    note(f"  sampled {len(rows)} rows, rerouted fraction {gm.mean():.3f}")
    L.close()


# Full-size rollouts on a head subset: the GPU runs every head of the
# workload (the benchmark's launch configuration), the oracle the rows of a
# few heads, over all 32 layers in segments of one anchor plus seven relays
# (the anchor at the start of each segment rebuilds every ledger entry, so
# segments are independent).
# The long-context workload crowds its top-k boundaries on purpose (a quarter
# of the keys are near-duplicates), so rows whose outcome hinges on a near tie
# accumulate until the next anchor: about a third of the rows are set aside
# by the eighth layer of a segment, hence its lower floor of compared rows.
SUBSET_ROLLOUTS = [
    ("scale", {}, (0, 31), range(0, 32), 0.8),
    ("longctx", {}, (0, 17), range(0, 8), 0.6),
    ("longctx", {}, (0, 17), range(8, 16), 0.6),
    ("longctx", {}, (0, 17), range(16, 24), 0.6),
    ("longctx", {}, (0, 17), range(24, 32), 0.6),
]


@pytest.mark.parametrize("name,kw,heads,layers,floor", SUBSET_ROLLOUTS,
                         ids=[f"{n}-layers{l.start}-{l.stop - 1}" for n, _, _, l, _ in SUBSET_ROLLOUTS])
def test_full_size_head_subset_rollout(name, kw, heads, layers, floor):
    from parity_util import rollout_subset
    w = synth.preset(name, **kw)
    note(f"full-size head-subset rollout: {w.name} n={w.n} heads {heads} of {w.n_heads}, layers {layers.start}..{layers.stop - 1}")
    st = rollout_subset(w, heads, layers, note=note)
    note(f"  {st}")
    assert st["compared"] >= floor * st["rows"]


def test_state_errors():
    from parity_util import dev
    rr = rrmod()
    cfg = rr.Config(1, 1, 64, 64, 64, 4, 2, 2)
    Q = dev(np.zeros((1, 64, 64), np.float32), "f32")
    L = rr.Ledger(cfg)
    with pytest.raises(rr.RRError) as e:
        L.relay(0, Q, Q)
    assert e.value.status == rr.RR_ERR_STATE
    L.anchor(3, Q, Q)
    with pytest.raises(rr.RRError) as e:
        L.relay(2, Q, Q)
    assert e.value.status == rr.RR_ERR_STATE
    L.relay(3, Q, Q)
    L.close()


def test_sweep_cap_counts_unconverged_rows():
    """The collection loop's sweep cap lies above what the bisections need:
    with the default cap no row is counted.  With the cap lowered to one sweep
    (a test hook), rows with all-zero queries -- every chunk ties at score 0,
    so the first collection overflows and needs repair sweeps -- are left
    unsettled: rr_unconverged_rows counts them, and their ledger entries hold
    valid ids only (empty R and N, sentinels from the valid chunks), while
    the other rows settle in one sweep and stay exact."""
    from parity_util import dev, ledger_np
    rr = rrmod()
    rng = np.random.default_rng(5)
    H, n, d, k, m, r = 2, 600, 64, 10, 5, 5
    Q = (rng.standard_normal((H, n, d)) / 8).astype(np.float32)
    Q[:, ::3] = 0.0
    K = (rng.standard_normal((H, n, d)) / 8).astype(np.float32)
    cfg = rr.Config(H, H, n, n, d, k, m, r, "f32", False)
    note("sweep cap: default, then one sweep")
    before = rr.unconverged_rows()
    L = rr.Ledger(cfg)
    L.anchor(0, dev(Q, "f32"), dev(K, "f32"))
    ref = oracle.new_ledger(oracle.Problem(H, H, n, n, d, k, m, r))
    oracle.anchor(oracle.Problem(H, H, n, n, d, k, m, r), 0, Q, K, ref)
    got = ledger_np(L)
    np.testing.assert_array_equal(got["routes"], ref["routes"])
    assert rr.unconverged_rows() == before
    try:
        rr.set_sweep_cap(1)
        L.anchor(1, dev(Q, "f32"), dev(K, "f32"))
        torch.cuda.synchronize()
    finally:
        rr.set_sweep_cap(0)
    counted = rr.unconverged_rows() - before
    got = ledger_np(L)
    empty = (got["routes"] == -1).all(1)
    note(f"  unconverged rows at one sweep: {counted}")
    assert counted > 0 and counted == int(empty.sum())
    assert empty.reshape(H, n)[:, ::3].all()
    assert ((got["sent"] >= -1) & (got["sent"] < n)).all()
    # rows that settled in one sweep are exact
    np.testing.assert_array_equal(got["routes"][~empty], ref["routes"][~empty])
    L.close()
