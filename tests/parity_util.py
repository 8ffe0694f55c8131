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
    p = oracle.Problem(w.n_heads, w.n_kv_heads, w.n, w.n, w.d, w.k, w.m, w.r, w.causal, w.gamma, w.seed)
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
    if not np.isfinite(p.gamma):
        return np.zeros(len(out["alpha"]), dtype=bool)
    with np.errstate(invalid="ignore"):
        diff = np.abs(out["alpha"] - (out["beta"] + p.gamma))
        t = tau(out["alpha"], out["beta"], out["alpha_abs"], out["beta_abs"], p.d)
        tie = np.nan_to_num(diff, nan=np.inf) < t
    return tie


def dev(x, dtype):
    return rr.to_device(x, dtype, torch.device("cuda", torch.cuda.current_device()))


def ledger_np(L: rr.Ledger):
    e = L.export()
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in e.items()}


def n_valid_rows(p):
    i = np.arange(p.rows) % p.n_q
    return np.minimum(i + 1, p.n_k) if p.causal else np.full(p.rows, p.n_k)


def rollout_compare(w, gamma=None, check_scores=True, relay="auto"):
    """Runs the workload's anchor/relay schedule on the GPU and on the oracle
    (relay: the relay schedule, "auto", "one_pass" or "split").

    Returns a dict of statistics; raises AssertionError on any mismatch of a
    trusted row."""
    if gamma is not None:
        w = w.with_(gamma=gamma)
    p = problem_of(w)
    cfg = dataclasses.replace(rr.Config.of(w), relay=relay)
    L = rr.Ledger(cfg)
    ref = oracle.new_ledger(p)
    trusted = np.zeros(p.rows, dtype=bool)
    ni = n_valid_rows(p)
    device = torch.device("cuda", torch.cuda.current_device())
    mask_t = torch.empty(p.rows, dtype=torch.uint8, device=device)
    pairs_t = torch.zeros(1, dtype=torch.int64, device=device)
    nrr_t = torch.zeros(1, dtype=torch.int32, device=device)
    stats = {"rows": 0, "compared": 0, "ties": 0, "rerouted": 0, "relay_rows": 0}
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
            # score pairs: the GPU's own accounting, and equality with the oracle
            cand = (before["routes"] >= 0).sum(1) + (before["sent"] >= 0).sum(1)
            assert int(pairs_t.item()) == int(cand.sum() + ni[gmask].sum())
            assert int(nrr_t.item()) == int(gmask.sum())
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
                tol = TOL[w.dtype]
                ok = trusted
                assert np.all(np.abs(alpha[ok] - out["alpha"][ok]) <= tol * out["alpha_abs"][ok] + 1e-30)
                fin = ok & np.isfinite(out["beta"])
                assert np.all(np.abs(beta[fin] - out["beta"][fin]) <= tol * out["beta_abs"][fin] + 1e-30)
                assert np.all(np.isneginf(beta[ok & ~np.isfinite(out["beta"])]))
            stats["rerouted"] += int(gmask.sum())
            stats["relay_rows"] += p.rows
            trusted = new_trusted
        stats["rows"] += p.rows
        stats["compared"] += int(trusted.sum())
        stats["ties"] += int((~trusted).sum())
    L.close()
    return stats
