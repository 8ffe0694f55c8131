"""Tie-aware comparison of the GPU path with the oracle.

A row is compared bit-exactly unless its outcome hinges on a near-tie that
binary32 accumulation may legitimately order differently from the oracle's
binary64 scores:
  T1  top-k boundary:      s_(k) - s_(k+1)   < tau
  T2  near-miss boundary:  s_(k+m) - s_(k+m+1) < tau
  T3  trigger:             |alpha - (beta + gamma)| < tau
with tau = max(1e-4 * max|s|, 2 d 2^-24 * max sum_t |q_t k_t|): the relative
band of the accepted tie rule, never narrower than the binary32 dot-product
error bound.  A row whose outcome was excluded stays excluded (tainted) until
the next anchor rebuilds it without a tie.

Scores (alpha, beta) are checked two ways: within TOL of sum_t |q_t k_t|
(the dot product's condition scale) on every trusted row, and within TOL of
|s| itself -- the literal relative error -- wherever the binary32
accumulation bound 2 d 2^-24 sum_t |q_t k_t| lies below TOL |s| (elsewhere a
binary32 dot product cannot promise that relative error).  The largest
literal |delta| / |s| over all trusted rows is reported.
"""
from __future__ import annotations

import dataclasses

import numpy as np
import torch

import oracle
from paper_2609_07306_amd import routerelay as rr
from paper_2609_07306_amd import synth

TOL = {"f32": 1e-5, "bf16": 2e-3}


def problem_of(w, **kw) -> oracle.Problem:
    p = oracle.Problem(w.n_heads, w.n_kv_heads, w.n, w.nk, w.d, w.k, w.m, w.r, w.causal, w.gamma, w.seed,
                       n_sink=w.n_sink, n_recent=w.n_recent, min_reuse=w.min_reuse)
    return dataclasses.replace(p, **kw) if kw else p


def tau(sa, sb, aa, ab, d):
    with np.errstate(invalid="ignore"):
        t = np.maximum(1e-4 * np.maximum(np.abs(sa), np.abs(sb)), 2 * d * 2.0 ** -24 * np.maximum(aa, ab))
    return np.nan_to_num(t, nan=0.0)


def gap_tie(sa, sb, aa, ab, d):
    """True where both ranks exist and their gap is inside the band."""
    with np.errstate(invalid="ignore"):
        g = sa - sb
        return np.nan_to_num(g, nan=np.inf) < tau(sa, sb, aa, ab, d)


def route_ties(p, Qf, Kf, rows=None):
    b = oracle.route_bounds(p, Qf, Kf, rows)
    t1 = gap_tie(b[:, 0], b[:, 1], b[:, 4], b[:, 5], p.d)
    t2 = gap_tie(b[:, 2], b[:, 3], b[:, 6], b[:, 7], p.d)
    return t1, t2


def trigger_ties(p, out):
    g = p.gamma_rows if p.gamma_rows is not None else np.full(len(out["alpha"]), p.gamma)
    with np.errstate(invalid="ignore"):
        diff = np.where(np.isfinite(g), np.abs(out["alpha"] - (out["beta"] + g)), np.inf)
        t = tau(out["alpha"], out["beta"], out["alpha_abs"], out["beta_abs"], p.d)
        tie = np.nan_to_num(diff, nan=np.inf) < t
    return tie


def dev(x, dtype):
    return rr.to_device(x, dtype, torch.device("cuda", torch.cuda.current_device()))


def ledger_np(L: rr.Ledger):
    e = L.export()
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in e.items()}


def score_check(got, ref, ref_abs, d, dtype, stats=None):
    """Checks binary32 scores against the oracle's binary64 ones (finite
    entries): within TOL * sum|qk| everywhere, within TOL * |s| where the
    accumulation bound allows; accumulates the literal relative error."""
    tol = TOL[dtype]
    fin = np.isfinite(ref)
    got, ref, ref_abs = got[fin], ref[fin], ref_abs[fin]
    delta = np.abs(got.astype(np.float64) - ref)
    assert np.all(delta <= tol * ref_abs + 1e-30), f"score error {delta.max()} beyond {tol} * sum|qk|"
    lit = 2 * d * 2.0 ** -24 * ref_abs <= tol * np.abs(ref)
    assert np.all(delta[lit] <= tol * np.abs(ref[lit])), "literal relative score error beyond tolerance"
    if stats is not None:
        with np.errstate(divide="ignore", invalid="ignore"):
            rel = np.where(ref != 0, delta / np.abs(ref), 0.0)
        if len(rel):
            stats["rel_err_max"] = max(stats.get("rel_err_max", 0.0), float(rel.max()))
        stats["rel_checked"] = stats.get("rel_checked", 0) + int(lit.sum())
        stats["scores_checked"] = stats.get("scores_checked", 0) + int(fin.sum())


def n_valid_rows(p):
    i = np.arange(p.rows) % p.n_q
    return np.minimum(i + 1, p.n_k) if p.causal else np.full(p.rows, p.n_k)


def rollout_compare(w, gamma=None, check_scores=True, relay="auto", gamma_rows=None, k_rows=None):
    """Runs the workload's anchor/relay schedule on the GPU and on the oracle
    (relay: the relay schedule, "auto", "one_pass" or "split"; gamma_rows:
    per-row guard margins, binary32 values, or None; k_rows: per-row route
    widths in [1, k], or None).

    Returns a dict of statistics; raises AssertionError on any mismatch of a
    trusted row."""
    if gamma is not None:
        w = w.with_(gamma=gamma)
    p = problem_of(w)
    cfg = dataclasses.replace(rr.Config.of(w), relay=relay)
    if gamma_rows is not None:
        g32 = np.ascontiguousarray(gamma_rows, dtype=np.float32)
        p = dataclasses.replace(p, gamma_rows=g32.astype(np.float64))
        cfg = dataclasses.replace(cfg, gamma_rows=torch.from_numpy(g32).to(torch.device("cuda", torch.cuda.current_device())))
    if k_rows is not None:
        k32 = np.ascontiguousarray(k_rows, dtype=np.int32)
        p = dataclasses.replace(p, k_rows=k32)
        cfg = dataclasses.replace(cfg, k_rows=torch.from_numpy(k32).to(torch.device("cuda", torch.cuda.current_device())))
    L = rr.Ledger(cfg)
    ref = oracle.new_ledger(p)
    trusted = np.zeros(p.rows, dtype=bool)
    ni = n_valid_rows(p)
    device = torch.device("cuda", torch.cuda.current_device())
    mask_t = torch.empty(p.rows, dtype=torch.uint8, device=device)
    pairs_t = torch.zeros(1, dtype=torch.int64, device=device)
    nrr_t = torch.zeros(1, dtype=torch.int32, device=device)
    stats = {"rows": 0, "compared": 0, "ties": 0, "rerouted": 0, "relay_rows": 0, "pair_rows_compared": 0}
    for layer, Qf, Kf, Qd, Kd in synth.Generator(w):
        Q, K = dev(Qd, w.dtype), dev(Kd, w.dtype)
        t1, t2 = route_ties(p, Qf, Kf)
        if w.is_anchor(layer):
            L.anchor(layer, Q, K, pairs=pairs_t)
            _, opairs = oracle.anchor(p, layer, Qf, Kf, ref)
            got = ledger_np(L)
            assert int(pairs_t.item()) == opairs
            trusted = ~(t1 | t2)
            for key in ("routes", "sent", "build", "age"):
                a, b = got[key][trusted], ref[key][trusted]
                assert np.array_equal(a, b), f"anchor layer {layer}: {key} differs on {np.flatnonzero((a != b).reshape(len(a), -1).any(1))[:8]}"
        else:
            before = ledger_np(L)
            L.relay(layer, Q, K, mask=mask_t, pairs=pairs_t, n_rerouted=nrr_t)
            out = oracle.relay(p, layer, Qf, Kf, ref)
            got = ledger_np(L)
            gmask = mask_t.cpu().numpy().astype(bool)
            omask = out["mask"].astype(bool)
            t3 = trigger_ties(p, out)
            decided = trusted & ~t3
            bad = np.flatnonzero(decided & (gmask != omask))
            assert len(bad) == 0, f"relay layer {layer}: mask differs on rows {bad[:8]}"
            new_trusted = decided & ~(omask & (t1 | t2))
            for key in ("routes", "sent", "build", "age"):
                a, b = got[key][new_trusted], ref[key][new_trusted]
                assert np.array_equal(a, b), f"relay layer {layer}: {key} differs"
            # score pairs: the kernel's total is the sum of its rows'
            # contributions (|A_i| of the ledger it started from, plus n_i when
            # rerouted); on every decided row that contribution equals the
            # oracle's, and the totals agree once the other rows are set aside
            cand = (before["routes"] >= 0).sum(1) + (before["sent"] >= 0).sum(1)
            gpu_row_pairs = cand + gmask.astype(np.int64) * ni
            assert int(pairs_t.item()) == int(gpu_row_pairs.sum())
            assert int(nrr_t.item()) == int(gmask.sum())
            bad = np.flatnonzero(decided & (gpu_row_pairs != out["row_pairs"]))
            assert len(bad) == 0, f"relay layer {layer}: score pairs differ on rows {bad[:8]}"
            assert int(pairs_t.item()) - int(gpu_row_pairs[~decided].sum()) == \
                out["pairs"] - int(out["row_pairs"][~decided].sum())
            stats["pair_rows_compared"] += int(decided.sum())
            if np.array_equal(gmask, omask) and trusted.all():
                assert int(pairs_t.item()) == out["pairs"]
            if check_scores:
                alpha, beta, ids = L.relay_stats()
                torch.cuda.synchronize()
                alpha, beta = alpha.cpu().numpy(), beta.cpu().numpy()
                # the rerouted rows of each head, ascending, then -1
                ids = ids.cpu().numpy().reshape(p.n_heads, p.n_q)
                for h in range(p.n_heads):
                    fl = np.flatnonzero(gmask.reshape(p.n_heads, p.n_q)[h])
                    np.testing.assert_array_equal(ids[h, :len(fl)], fl)
                    assert np.all(ids[h, len(fl):] == -1)
                ok = trusted
                score_check(alpha[ok], out["alpha"][ok], out["alpha_abs"][ok], p.d, w.dtype, stats)
                score_check(beta[ok], out["beta"][ok], out["beta_abs"][ok], p.d, w.dtype, stats)
                assert np.all(np.isneginf(beta[ok & ~np.isfinite(out["beta"])]))
                assert np.all(np.isposinf(alpha[ok & np.isposinf(out["alpha"])]))
            stats["rerouted"] += int(gmask.sum())
            stats["relay_rows"] += p.rows
            trusted = new_trusted
        stats["rows"] += p.rows
        stats["compared"] += int(trusted.sum())
        stats["ties"] += int((~trusted).sum())
    L.close()
    return stats


def _oracle_threads(fn, p, head_rows):
    """Runs fn(rows) for each head's row block in its own thread (the C
    oracle holds no global state and ctypes releases the GIL; the heads'
    rows are disjoint, so the ledger arrays are written without overlap)."""
    from concurrent.futures import ThreadPoolExecutor
    with ThreadPoolExecutor(max_workers=len(head_rows)) as ex:
        return list(ex.map(fn, head_rows))


def rollout_subset(w, heads, layers, relay="auto", note=print):
    """The workload at its full size on the GPU (every head, the launch
    configuration the benchmark times) against the oracle on the rows of the
    listed query heads only, over ``layers`` (a range that starts at an
    anchor layer).  Every anchor and relay layer is compared tie-aware on
    those rows: ledger rows, mask, alpha / beta, per-row score pairs.
    Returns the statistics dict of rollout_compare."""
    p = problem_of(w)
    assert w.is_anchor(layers.start), "a subset rollout starts at an anchor"
    cfg = dataclasses.replace(rr.Config.of(w), relay=relay)
    L = rr.Ledger(cfg)
    ref = oracle.new_ledger(p)
    head_rows = [np.arange(h * p.n_q, (h + 1) * p.n_q, dtype=np.int64) for h in heads]
    rows = np.concatenate(head_rows)
    ni = n_valid_rows(p)[rows]
    trusted = np.zeros(len(rows), dtype=bool)
    device = torch.device("cuda", torch.cuda.current_device())
    mask_t = torch.empty(p.rows, dtype=torch.uint8, device=device)
    pairs_t = torch.zeros(1, dtype=torch.int64, device=device)
    stats = {"rows": 0, "compared": 0, "ties": 0, "rerouted": 0, "relay_rows": 0, "pair_rows_compared": 0,
             "tie_rows_per_layer": []}

    def sub(led):
        return {k: v[rows] for k, v in led.items()}

    for layer, Qf, Kf, Qd, Kd in synth.Generator(w):
        if layer < layers.start:
            continue
        if layer >= layers.stop:
            break
        Q, K = dev(Qd, w.dtype), dev(Kd, w.dtype)
        bounds = np.concatenate(_oracle_threads(lambda r: oracle.route_bounds(p, Qf, Kf, r), p, head_rows))
        t1 = gap_tie(bounds[:, 0], bounds[:, 1], bounds[:, 4], bounds[:, 5], p.d)
        t2 = gap_tie(bounds[:, 2], bounds[:, 3], bounds[:, 6], bounds[:, 7], p.d)
        if w.is_anchor(layer):
            L.anchor(layer, Q, K)
            _oracle_threads(lambda r: oracle.anchor(p, layer, Qf, Kf, ref, rows=r), p, head_rows)
            got = sub(ledger_np(L))
            trusted = ~(t1 | t2)
            for key in ("routes", "sent", "build", "age"):
                a, b = got[key][trusted], ref[key][rows][trusted]
                assert np.array_equal(a, b), f"anchor layer {layer}: {key} differs"
            stats["tie_rows_per_layer"].append(int((t1 | t2).sum()))
        else:
            before = sub(ledger_np(L))
            L.relay(layer, Q, K, mask=mask_t, pairs=pairs_t)
            outs = _oracle_threads(lambda r: oracle.relay(p, layer, Qf, Kf, ref, rows=r), p, head_rows)
            out = {k: np.concatenate([o[k][r] for o, r in zip(outs, head_rows)])
                   for k in ("mask", "row_pairs", "alpha", "beta", "alpha_abs", "beta_abs")}
            got = sub(ledger_np(L))
            gmask = mask_t.cpu().numpy().astype(bool)[rows]
            omask = out["mask"].astype(bool)
            with np.errstate(invalid="ignore"):
                t3 = (np.abs(out["alpha"] - (out["beta"] + p.gamma)) <
                      tau(out["alpha"], out["beta"], out["alpha_abs"], out["beta_abs"], p.d))
            decided = trusted & ~t3
            bad = np.flatnonzero(decided & (gmask != omask))
            assert len(bad) == 0, f"relay layer {layer}: mask differs on rows {rows[bad[:8]]}"
            new_trusted = decided & ~(omask & (t1 | t2))
            for key in ("routes", "sent", "build", "age"):
                a, b = got[key][new_trusted], ref[key][rows][new_trusted]
                assert np.array_equal(a, b), f"relay layer {layer}: {key} differs"
            cand = (before["routes"] >= 0).sum(1) + (before["sent"] >= 0).sum(1)
            gpu_row_pairs = cand + gmask.astype(np.int64) * ni
            bad = np.flatnonzero(decided & (gpu_row_pairs != out["row_pairs"]))
            assert len(bad) == 0, f"relay layer {layer}: score pairs differ on rows {rows[bad[:8]]}"
            stats["pair_rows_compared"] += int(decided.sum())
            alpha, beta, _ = L.relay_stats()
            torch.cuda.synchronize()
            alpha, beta = alpha.cpu().numpy()[rows], beta.cpu().numpy()[rows]
            score_check(alpha[trusted], out["alpha"][trusted], out["alpha_abs"][trusted], p.d, w.dtype, stats)
            score_check(beta[trusted], out["beta"][trusted], out["beta_abs"][trusted], p.d, w.dtype, stats)
            stats["rerouted"] += int(gmask.sum())
            stats["relay_rows"] += len(rows)
            stats["tie_rows_per_layer"].append(int((~new_trusted).sum()))
            trusted = new_trusted
        stats["rows"] += len(rows)
        stats["compared"] += int(trusted.sum())
        stats["ties"] += int((~trusted).sum())
        note(f"  layer {layer}: compared {int(trusted.sum())} of {len(rows)} rows")
    L.close()
    return stats


def step_compare(w, heads=None, relay="auto", k_rows=None, gamma_rows=None, note=print):
    """Step mode: before each relay layer the oracle's ledger is imported into
    the GPU ledger (on the rows compared; the GPU keeps its own state on the
    others), so both sides start every layer from the same state and each
    layer is compared on its own near-ties only (T1 / T2 of that layer, T3 of
    that relay), with no taint carried between layers.  heads: the query
    heads whose rows the oracle computes (None: all).  Anchors are compared
    the same way.  Returns per-layer statistics."""
    p = problem_of(w)
    cfg = dataclasses.replace(rr.Config.of(w), relay=relay)
    device = torch.device("cuda", torch.cuda.current_device())
    if k_rows is not None:
        k32 = np.ascontiguousarray(k_rows, dtype=np.int32)
        p = dataclasses.replace(p, k_rows=k32)
        cfg = dataclasses.replace(cfg, k_rows=torch.from_numpy(k32).to(device))
    if gamma_rows is not None:
        g32 = np.ascontiguousarray(gamma_rows, dtype=np.float32)
        p = dataclasses.replace(p, gamma_rows=g32.astype(np.float64))
        cfg = dataclasses.replace(cfg, gamma_rows=torch.from_numpy(g32).to(device))
    heads = list(range(p.n_heads)) if heads is None else list(heads)
    head_rows = [np.arange(h * p.n_q, (h + 1) * p.n_q, dtype=np.int64) for h in heads]
    rows = np.concatenate(head_rows)
    ni = n_valid_rows(p)[rows]
    gam = (p.gamma_rows[rows] if p.gamma_rows is not None else np.full(len(rows), p.gamma))
    L = rr.Ledger(cfg)
    ref = oracle.new_ledger(p)
    mask_t = torch.empty(p.rows, dtype=torch.uint8, device=device)
    pairs_t = torch.zeros(1, dtype=torch.int64, device=device)
    stats = {"layers": 0, "rows": 0, "compared": 0, "mask_compared": 0, "rerouted": 0}
    for layer, Qf, Kf, Qd, Kd in synth.Generator(w):
        Q, K = dev(Qd, w.dtype), dev(Kd, w.dtype)
        bounds = np.concatenate(_oracle_threads(lambda r: oracle.route_bounds(p, Qf, Kf, r), p, head_rows))
        t1 = gap_tie(bounds[:, 0], bounds[:, 1], bounds[:, 4], bounds[:, 5], p.d)
        t2 = gap_tie(bounds[:, 2], bounds[:, 3], bounds[:, 6], bounds[:, 7], p.d)
        if w.is_anchor(layer):
            L.anchor(layer, Q, K)
            _oracle_threads(lambda r: oracle.anchor(p, layer, Qf, Kf, ref, rows=r), p, head_rows)
            trusted = ~(t1 | t2)
            omask = np.ones(len(rows), dtype=bool)
        else:
            # both sides start the layer from the oracle's state
            cur = ledger_np(L)
            for key in ("routes", "sent", "build", "age"):
                cur[key][rows] = ref[key][rows]
            imp = {k: torch.from_numpy(np.ascontiguousarray(v)).to(device) for k, v in cur.items()}
            L.import_(layer - 1, imp["routes"], imp["sent"] if p.sent_width else None, imp["build"], imp["age"])
            L.relay(layer, Q, K, mask=mask_t, pairs=pairs_t)
            outs = _oracle_threads(lambda r: oracle.relay(p, layer, Qf, Kf, ref, rows=r), p, head_rows)
            out = {k: np.concatenate([o[k][r] for o, r in zip(outs, head_rows)])
                   for k in ("mask", "row_pairs", "alpha", "beta", "alpha_abs", "beta_abs")}
            gmask = mask_t.cpu().numpy().astype(bool)[rows]
            omask = out["mask"].astype(bool)
            with np.errstate(invalid="ignore"):
                diff = np.where(np.isfinite(gam), np.abs(out["alpha"] - (out["beta"] + gam)), np.inf)
                t3 = np.nan_to_num(diff, nan=np.inf) < tau(out["alpha"], out["beta"], out["alpha_abs"],
                                                          out["beta_abs"], p.d)
            decided = ~t3
            bad = np.flatnonzero(decided & (gmask != omask))
            assert len(bad) == 0, f"step layer {layer}: mask differs on rows {rows[bad[:8]]}"
            sent_rows = cur["sent"][rows] if p.sent_width else np.zeros((len(rows), 0), np.int32)
            cand = (cur["routes"][rows] >= 0).sum(1) + (sent_rows >= 0).sum(1)
            gpu_row_pairs = cand + gmask.astype(np.int64) * ni
            bad = np.flatnonzero(decided & (gpu_row_pairs != out["row_pairs"]))
            assert len(bad) == 0, f"step layer {layer}: score pairs differ on rows {rows[bad[:8]]}"
            trusted = decided & ~(omask & (t1 | t2))
            alpha, beta, _ = L.relay_stats()
            torch.cuda.synchronize()
            alpha, beta = alpha.cpu().numpy()[rows], beta.cpu().numpy()[rows]
            score_check(alpha, out["alpha"], out["alpha_abs"], p.d, w.dtype, stats)
            score_check(beta, out["beta"], out["beta_abs"], p.d, w.dtype, stats)
            stats["mask_compared"] += int(decided.sum())
            stats["rerouted"] += int(gmask.sum())
        got = ledger_np(L)
        for key in ("routes", "sent", "build", "age"):
            a, b = got[key][rows][trusted], ref[key][rows][trusted]
            assert np.array_equal(a, b), f"step layer {layer}: {key} differs on rows " \
                f"{rows[np.flatnonzero((a != b).reshape(len(a), -1).any(1))[:8]]}"
        stats["layers"] += 1
        stats["rows"] += len(rows)
        stats["compared"] += int(trusted.sum())
        note(f"  step layer {layer}: compared {int(trusted.sum())} of {len(rows)} rows")
    L.close()
    return stats
