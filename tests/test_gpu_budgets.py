"""GPU parity of query-dependent route budgets (Sec. 4.3 and 4.4): per-row
route widths k_i in one launch, through the C ABI, against the oracle.

Row i's first k_i route slots hold its k_i best chunks (the rest -1) and its
near-miss sentinels are the m chunks ranked after them; alpha is the minimum
over the k_i routed chunks.  The tie protocol is the one of the other parity
tests, with the boundary ranks taken at k_i and k_i + m."""
import dataclasses
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


def _widths(rng, rows, k):
    """Per-row widths with the extremes 1 and k always present."""
    kr = rng.integers(1, k + 1, size=rows).astype(np.int32)
    kr[0], kr[-1] = 1, k
    return kr


def _kdev(kr):
    return torch.from_numpy(np.ascontiguousarray(kr, dtype=np.int32)).to("cuda")


FULL_CASES = [
    # name, H, Hkv, n_q, n_k, d, dtype, k, causal
    ("ragged_f32", 3, 1, 100, 77, 32, "f32", 5, False),
    ("ragged_causal", 2, 2, 70, 70, 64, "f32", 9, True),
    ("bf16_causal_gqa", 4, 1, 200, 200, 128, "bf16", 32, True),
    ("bf16_d256", 2, 2, 64, 96, 256, "bf16", 12, False),
    ("wide_k", 2, 2, 64, 512, 128, "bf16", 100, False),
]


@pytest.mark.parametrize("case", FULL_CASES, ids=[c[0] for c in FULL_CASES])
def test_full_route_budgets(case):
    from parity_util import dev, route_ties, TOL
    rr = rrmod()
    name, H, Hkv, n_q, n_k, d, dtype, k, causal = case
    note(f"full route with budgets: {case}")
    rng = np.random.default_rng(zlib.crc32(name.encode()) ^ 0x5A)
    Q = (rng.standard_normal((H, n_q, d)) / np.sqrt(d)).astype(np.float32)
    K = (rng.standard_normal((Hkv, n_k, d)) / np.sqrt(d)).astype(np.float32)
    if dtype == "bf16":
        Qd, Kd = synth.bf16_round(Q), synth.bf16_round(K)
        Qf, Kf = synth.bf16_widen(Qd), synth.bf16_widen(Kd)
    else:
        Qd, Kd, Qf, Kf = Q, K, Q, K
    kr = _widths(rng, H * n_q, k)
    cfg = rr.Config(H, Hkv, n_q, n_k, d, k, 0, 0, dtype, causal, k_rows=_kdev(kr))
    p = oracle.Problem(H, Hkv, n_q, n_k, d, k, 0, 0, causal, k_rows=kr)
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
    # every row holds min(k_i, n_i) ids, then -1
    ni = np.minimum(np.arange(cfg.rows) % n_q + 1, n_k) if causal else np.full(cfg.rows, n_k)
    assert np.array_equal((got >= 0).sum(1), np.minimum(kr, ni))
    sc = scores.cpu().numpy()
    valid = exact >= 0
    for row in np.flatnonzero(~t1)[:400]:
        h, i = divmod(row, n_q)
        g = h // (H // Hkv)
        ids = exact[row][valid[row]]
        absd = np.abs(Qf[h, i].astype(np.float64)[None, :] * Kf[g, ids].astype(np.float64)).sum(1)
        assert np.all(np.abs(sc[row][valid[row]] - osc[row][valid[row]]) <= TOL[dtype] * absd)
        assert np.all(np.isneginf(sc[row][~valid[row]]))


@pytest.mark.parametrize("T_class", ["narrow", "wide"])
@pytest.mark.parametrize("causal", [False, True])
def test_budget_ledger_exact_ties_integer_data(T_class, causal):
    """Small-integer inputs (every score exact on both sides, massive exact
    ties): full routing, the anchor ledger and two relay layers with per-row
    widths must match the oracle on every row, including alpha and beta."""
    from parity_util import dev, ledger_np
    rr = rrmod()
    rng = np.random.default_rng(31 if causal else 32)
    H, n, d = 2, 300, 32
    k, m, r = (24, 12, 8) if T_class == "narrow" else (60, 30, 20)
    kr = _widths(rng, H * n, k)
    note(f"integer-tie ledger with budgets: {T_class} causal={causal}")
    p = oracle.Problem(H, H, n, n, d, k, m, r, causal, seed=9, k_rows=kr)
    cfg = rr.Config(H, H, n, n, d, k, m, r, "f32", causal, seed=9, k_rows=_kdev(kr))
    L = rr.Ledger(cfg)
    ref = oracle.new_ledger(p)
    for layer in range(3):
        Q = rng.integers(-2, 3, size=(H, n, d)).astype(np.float32)
        K = rng.integers(-1, 2, size=(H, n, d)).astype(np.float32)
        if layer == 0:
            full = torch.empty((cfg.rows, k), dtype=torch.int32, device="cuda")
            rr.full_route(cfg, dev(Q, "f32"), dev(K, "f32"), full)
            L.anchor(layer, dev(Q, "f32"), dev(K, "f32"))
            oracle.anchor(p, layer, Q, K, ref)
            exact, _ = oracle.full_route(p, Q, K)
            np.testing.assert_array_equal(full.cpu().numpy(), exact)
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


def _run(cfg, lay, n_layers, dtype):
    from parity_util import dev, ledger_np
    rr = rrmod()
    L = rr.Ledger(cfg)
    states = []
    for layer in range(n_layers):
        Q, K = dev(lay[layer][2], dtype), dev(lay[layer][3], dtype)
        mask = torch.zeros(cfg.rows, dtype=torch.uint8, device="cuda")
        if layer == 0:
            L.anchor(0, Q, K)
        else:
            L.relay(layer, Q, K, mask=mask)
        st = ledger_np(L)
        st["mask"] = mask.cpu().numpy()
        states.append(st)
    L.close()
    return states


@pytest.mark.parametrize("relay", ["split", "one_pass"])
def test_uniform_and_clamped_widths(relay):
    """Every k_i = k reproduces the scalar width bit for bit; widths outside
    [1, k] act as the nearest bound."""
    rr = rrmod()
    w = synth.preset("drift", n_heads=4, n_kv_heads=4, n_layers=4, rho=0.3)
    lay = synth.layers(w)
    base = dataclasses.replace(rr.Config.of(w), relay=relay)
    note(f"uniform / clamped widths ({relay})")
    scalar = _run(base, lay, 4, w.dtype)
    uniform = _run(dataclasses.replace(base, k_rows=_kdev(np.full(w.rows, w.k))), lay, 4, w.dtype)
    rng = np.random.default_rng(2)
    kr = rng.integers(1, w.k + 1, size=w.rows).astype(np.int32)
    wild = kr.copy()
    wild[kr == 1] = rng.choice(np.array([0, -5, -(2 ** 31)], np.int32), size=int((kr == 1).sum()))
    wild[kr == w.k] = rng.choice(np.array([w.k + 1, 1000, 2 ** 31 - 1], np.int32), size=int((kr == w.k).sum()))
    assert (kr == 1).any() and (kr == w.k).any()
    inside = _run(dataclasses.replace(base, k_rows=_kdev(kr)), lay, 4, w.dtype)
    outside = _run(dataclasses.replace(base, k_rows=_kdev(wild)), lay, 4, w.dtype)
    for a, b, c, d in zip(scalar, uniform, inside, outside):
        for key in a:
            np.testing.assert_array_equal(a[key], b[key], err_msg=key)
            np.testing.assert_array_equal(c[key], d[key], err_msg=key)


BUDGET_ROLLOUTS = [
    ("drift", {"n_heads": 4, "n_kv_heads": 4, "n_layers": 8, "rho": 0.3}),
    ("tiny", {"n": 100, "d": 32, "k": 5, "m": 3, "r": 2, "n_heads": 4, "n_kv_heads": 2, "n_layers": 5,
              "causal": True, "dtype": "bf16"}),
    ("gqa", {"n_heads": 8, "n_kv_heads": 2, "n": 256, "n_layers": 6, "n_sink": 2, "n_recent": 2}),
    # dense rescoring tiles (enough 128-row tiles) whose threshold seeds are
    # taken at the widest T = k + m
    ("scale", {"n_heads": 256, "n_kv_heads": 256, "n": 128, "n_layers": 4, "anchor_every": 2}),
    # the wide route class (k + m > 64)
    ("scale", {"n_heads": 8, "n_kv_heads": 8, "n": 192, "k": 48, "m": 24, "r": 8, "n_layers": 5}),
    ("longctx", {"n_heads": 2, "n_kv_heads": 2, "n": 512, "n_layers": 6, "min_reuse": 1}),
]


@pytest.mark.parametrize("relay", ["split", "one_pass"])
@pytest.mark.parametrize("name,kw", BUDGET_ROLLOUTS, ids=[f"{n}-{i}" for i, (n, _) in enumerate(BUDGET_ROLLOUTS)])
def test_rollout_parity_budgets(name, kw, relay):
    from parity_util import rollout_compare
    w = synth.preset(name, **kw)
    kr = synth.route_budgets(w)
    note(f"budget rollout {name} {kw} ({relay}); widths {sorted(set(kr.tolist()))}")
    st = rollout_compare(w, relay=relay, k_rows=kr)
    note(f"  {st}")
    floor = 0.6 if w.near_ties else 0.8
    assert st["compared"] >= floor * st["rows"] and st["rerouted"] > 0


@pytest.mark.parametrize("relay", ["split", "one_pass"])
def test_static_relay_with_budgets(relay):
    """The allocation-free relay honours the per-row widths like the ledger
    relay."""
    rr = rrmod()
    dev = torch.device("cuda", 0)
    w = synth.preset("gqa", n_heads=8, n_kv_heads=2, n=160, rho=0.1)
    kr = synth.route_budgets(w)
    cfg = dataclasses.replace(rr.Config.of(w), relay=relay, k_rows=_kdev(kr))
    note(f"static relay with budgets ({relay})")
    led = rr.Ledger(cfg)
    lay = synth.layers(w.with_(n_layers=4))
    led.anchor(0, rr.to_device(lay[0][2], w.dtype, dev), rr.to_device(lay[0][3], w.dtype, dev))
    own = led.export()
    outs = [dict(routes=torch.full((cfg.rows, cfg.k), -7, dtype=torch.int32, device=dev),
                 mask=torch.full((cfg.rows,), 7, dtype=torch.uint8, device=dev),
                 pairs=torch.zeros(1, dtype=torch.int64, device=dev),
                 n_rerouted=torch.zeros(1, dtype=torch.int32, device=dev)) for _ in range(2)]
    for layer in range(1, 4):
        Q, K = rr.to_device(lay[layer][2], w.dtype, dev), rr.to_device(lay[layer][3], w.dtype, dev)
        led.relay(layer, Q, K, **outs[0])
        rr.relay_static(cfg, layer, Q, K, own, **outs[1])
        torch.cuda.synchronize()
        for key in outs[0]:
            assert torch.equal(outs[0][key], outs[1][key]), f"layer {layer}: {key}"
        ref = led.export()
        torch.cuda.synchronize()
        for key in ("routes", "sent", "build", "age"):
            assert torch.equal(ref[key], own[key]), f"layer {layer}: ledger {key}"
        routes = outs[0]["routes"].cpu().numpy()
        ni = np.minimum(np.arange(cfg.rows) % w.n + 1, w.n) if w.causal else np.full(cfg.rows, w.n)
        assert np.array_equal((routes >= 0).sum(1), np.minimum(kr, ni))
    led.close()
