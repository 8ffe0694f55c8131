#!/usr/bin/env python3
"""Benchmark of the RouteRelay route-maintenance path on one MI355X.

Workload (default): the routing-scale configuration at n_k = 1024 -- 32 query
heads x 1024 query chunks, 1024 key chunks, d = 128, bf16 inputs with binary32
accumulation, k = 32, m = 16, r = 16, 32 layers with an anchor every 8 layers,
64-cluster synthetic chunks drifting with rho = 0.3 (paper_2609_07306_amd.synth).

A step is one pass of the whole path over all 32 layers: anchors (GEMM + TopK
+ ledger build) at layers 0, 8, 16, 24 and relay layers (rescoring, trigger,
compaction, row-selective GEMM + TopK, ledger update) elsewhere.  All inputs
are resident in HBM before timing.  The baseline step runs full routing
(the same GEMM + TopK kernel) at every layer.

Output: one JSON line.  ``value`` = routed rows per second per layer of the
RouteRelay schedule (H * n_q * L / step time).  ``roofline`` describes the
kernel with the largest share of the step, timed with HIP events the library
records on its launch stream; ``cpu_baseline`` times the oracle on a head
subset of the same workload on this host.
"""
from __future__ import annotations

import argparse
import dataclasses
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK = {"hbm": 8000.0, "mfma_bf16": 2500.0, "mfma_f32": 157.3}  # GB/s, TFLOP/s

# HBM bytes per launch of the dominant kernel, from byte-counter passes
# (FETCH_SIZE, WRITE_SIZE, calibrated on a copy of known size) recorded in
# this profile; valid only while the kernel's sources hash to the recorded value.
TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "route_rescore_scale_n1024_hbm_bytes.md")
TRAFFIC_SOURCES = ["paper_2609_07306_amd/csrc/rr_route_impl.hpp", "paper_2609_07306_amd/csrc/rr_device.hpp",
                   "paper_2609_07306_amd/csrc/rr_internal.hpp", "paper_2609_07306_amd/csrc/rr_route_bf16_reroute.hip",
                   "paper_2609_07306_amd/build.py"]


def recorded_traffic(kernel: str):
    """Counter-measured HBM bytes per launch of `kernel`, or None if not recorded
    or if the kernel's sources changed since the counters were taken."""
    import hashlib
    import re
    try:
        text = open(TRAFFIC_PROFILE).read()
    except OSError:
        return None
    m = re.search(r"bench-traffic kernel=(\w+) bytes_per_launch=(\d+) sources_sha256=([0-9a-f]+)", text)
    if not m or m.group(1) != kernel:
        return None
    h = hashlib.sha256()
    for f in TRAFFIC_SOURCES:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return int(m.group(2)) if h.hexdigest() == m.group(3) else None


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="scale", help="synth preset (scale, drift, gqa, longctx, tiny)")
    ap.add_argument("--n", type=int, default=None, help="chunk count override (n_q = n_k)")
    ap.add_argument("--rho", type=float, default=None)
    ap.add_argument("--relay", default="auto", choices=("auto", "one_pass", "split"),
                    help="relay schedule (auto: one pass for causal inputs, else rescoring + compacted reroute)")
    ap.add_argument("--cpu-heads", type=int, default=2, help="heads in the oracle's timed sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-full", action="store_true", help="skip the full-routing baseline")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a device-to-device copy of MIB MiB (calibrates the HBM byte counters)")
    return ap.parse_args()


def describe(w) -> str:
    parts = [f"{w.name}: {w.n_heads} query heads / {w.n_kv_heads} key heads x {w.n} chunks",
             f"d={w.d} {w.dtype}", f"k={w.k} m={w.m} r={w.r}",
             f"{w.n_layers} layers, anchor every {w.anchor_every or w.n_layers}",
             f"{w.clusters} clusters, rho={w.rho}"]
    if w.causal:
        parts.append("causal chunk mask")
    if w.near_ties:
        parts.append("25% near-tie duplicate keys")
    return ", ".join(parts)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the path shards by "
              "head with no exchange, so N GPUs would each run this workload's 1/N share.",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2609_07306_amd import routerelay as rr
    from paper_2609_07306_amd import synth

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    torch.cuda.set_device(0)
    dev = torch.device("cuda", 0)
    if args.copy_calibration:
        # one plain copy of a known size: the FETCH_SIZE / WRITE_SIZE counters
        # of this dispatch give the scale factor of the byte counters
        n = args.copy_calibration << 20
        src = torch.ones(n, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": n}))
        return

    kw = {}
    if args.n:
        kw["n"] = args.n
    if args.rho is not None:
        kw["rho"] = args.rho
    w = synth.preset(args.workload, **kw)
    cfg = dataclasses.replace(rr.Config.of(w), relay=args.relay)
    rows, L = cfg.rows, w.n_layers
    e_bytes = 2 if w.dtype == "bf16" else 4
    print(f"[bench] generating {describe(w)}", file=sys.stderr, flush=True)

    # ---- inputs, resident in HBM before any timing
    hs = min(args.cpu_heads, w.n_heads)
    group = w.n_heads // w.n_kv_heads
    hs = max(group, (hs // group) * group)
    Qd, Kd, cpu_sample = [], [], []
    for layer, Qf, Kf, Qx, Kx in synth.Generator(w):
        Qd.append(rr.to_device(Qx, w.dtype, dev))
        Kd.append(rr.to_device(Kx, w.dtype, dev))
        if not args.no_cpu_baseline:
            cpu_sample.append((np.ascontiguousarray(Qf[:hs]), np.ascontiguousarray(Kf[: hs // group])))
    torch.cuda.synchronize()
    print("[bench] inputs resident", file=sys.stderr, flush=True)

    led = rr.Ledger(cfg)
    masks = torch.zeros((L, rows), dtype=torch.uint8, device=dev)
    pairs = torch.zeros((L, 1), dtype=torch.int64, device=dev)
    nrr = torch.zeros((L, 1), dtype=torch.int32, device=dev)
    full_routes = torch.empty((L, rows, w.k), dtype=torch.int32, device=dev)
    relay_routes = torch.empty((L, rows, w.k), dtype=torch.int32, device=dev)

    def relay_step(keep_routes=False, marks=None):
        for l in range(L):
            if marks is not None:
                marks[l].record()
            out = relay_routes[l] if keep_routes else None
            if w.is_anchor(l):
                led.anchor(l, Qd[l], Kd[l], routes=out, pairs=pairs[l])
            else:
                led.relay(l, Qd[l], Kd[l], routes=out, mask=masks[l], pairs=pairs[l], n_rerouted=nrr[l])
        if marks is not None:
            marks[L].record()

    def full_step():
        for l in range(L):
            rr.full_route(cfg, Qd[l], Kd[l], full_routes[l])

    def timed(fn, steps):
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(steps):
            fn()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / steps

    for _ in range(args.warmup):
        relay_step()
        if not args.no_full:
            full_step()
    torch.cuda.synchronize()
    print("[bench] warm", file=sys.stderr, flush=True)

    # ---- timed region: the RouteRelay schedule, then the baseline
    ms_step = timed(relay_step, args.steps)
    ms_full = timed(full_step, args.steps) if not args.no_full else float("nan")
    print(f"[bench] relay step {ms_step:.3f} ms, full step {ms_full:.3f} ms", file=sys.stderr, flush=True)

    # ---- per-layer durations (events between library calls on the stream)
    lay_ms = np.zeros(L)
    for _ in range(args.steps):
        marks = [torch.cuda.Event(enable_timing=True) for _ in range(L + 1)]
        relay_step(marks=marks)
        torch.cuda.synchronize()
        lay_ms += [marks[l].elapsed_time(marks[l + 1]) for l in range(L)]
    lay_ms /= args.steps
    anchor_l = [l for l in range(L) if w.is_anchor(l)]
    relay_l = [l for l in range(L) if not w.is_anchor(l)]

    # ---- per-kernel durations: library-recorded HIP events on the launch stream
    rr.profile_start()
    for _ in range(args.steps):
        relay_step()
        if not args.no_full:
            full_step()
    prof = rr.profile_stop()

    # ---- fidelity of one step (outside timing)
    relay_step(keep_routes=True)
    if args.no_full:
        full_step()
    torch.cuda.synchronize()
    hit = tot = 0
    for l in range(L):
        a, b = relay_routes[l], full_routes[l]
        va = a >= 0
        eq = (a.unsqueeze(2) == b.unsqueeze(1)) & va.unsqueeze(2)
        hit += int(eq.any(1).sum().item())
        tot += int((b >= 0).sum().item())
    recall = hit / tot
    n_i = np.minimum(np.arange(w.n) + 1, w.n) if w.causal else np.full(w.n, w.n)
    full_pairs_layer = int(n_i.sum()) * w.n_heads
    pairs_np = pairs.cpu().numpy().ravel()
    rer = nrr.cpu().numpy().ravel()
    rer_relay = float(sum(rer[l] for l in relay_l)) / (rows * max(1, len(relay_l)))
    rer_all = float(len(anchor_l) * rows + sum(rer[l] for l in relay_l)) / (rows * L)
    pair_frac = float(pairs_np.sum()) / (full_pairs_layer * L)

    # ---- roofline per kernel kind
    c = w.k + w.m + w.r
    kvb = w.n_kv_heads * w.n * w.d * e_bytes
    mean_rerouted = float(sum(rer[l] for l in relay_l)) / max(1, len(relay_l))
    mean_ni = float(n_i.mean())
    mpeak = PEAK["mfma_bf16"] if w.dtype == "bf16" else PEAK["mfma_f32"]
    alg = {
        # per launch: (bound, algorithmic amount, unit, peak)
        "rescore": ("hbm", (rows * (c * 4 + w.d * e_bytes + 18) + kvb) / 1e9, "GB/s", PEAK["hbm"]),
        "anchor": ("mfma", 2.0 * w.d * full_pairs_layer / 1e12, "TFLOP/s", mpeak),
        "reroute": ("mfma", 2.0 * w.d * mean_rerouted * mean_ni / 1e12, "TFLOP/s", mpeak),
        "full": ("mfma", 2.0 * w.d * full_pairs_layer / 1e12, "TFLOP/s", mpeak),
        # one-pass relay: the ledger's candidates rescored, the flagged rows routed
        "relay": ("mfma", 2.0 * w.d * (rows * c + mean_rerouted * mean_ni) / 1e12, "TFLOP/s", mpeak),
    }
    kernels = {}
    for kind, (tms, n) in prof.items():
        if n == 0:
            continue
        us = 1e3 * tms / n
        bound, amount, unit, peak = alg[kind]
        achieved = amount / (us * 1e-6)
        kernels[kind] = {"us_per_launch": round(us, 3), "launches_per_step": n // args.steps,
                         "bound": bound, "achieved": round(achieved, 3), "unit": unit,
                         "peak": peak, "frac": round(achieved / peak, 4),
                         "share_of_step": None}
    path_kinds = ("anchor", "reroute", "rescore", "relay")
    path_ms = sum(prof[k][0] for k in path_kinds) / args.steps
    for kind in path_kinds:
        if kind in kernels:
            kernels[kind]["share_of_step"] = round(prof[kind][0] / args.steps / ms_step, 4)
    dom = max(path_kinds, key=lambda k: prof[k][0])
    dk = kernels[dom]
    # the recorded counters belong to the default workload (routing scale, n = 1024)
    default_workload = args.workload == "scale" and w.n == 1024 and args.rho is None and args.relay == "auto"
    roofline = {"kernel": dom, "bound": dk["bound"], "achieved": dk["achieved"], "peak": dk["peak"],
                "unit": dk["unit"], "frac": dk["frac"],
                "traffic": recorded_traffic(dom) if default_workload else None}

    value = rows * L / (ms_step * 1e-3)
    out = {
        "metric": "route rows/s per layer, RouteRelay anchor+relay schedule (vs GPU full routing)",
        "value": round(value, 1),
        "unit": "rows/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {"workload": describe(w), "rows_per_layer": rows, "layers": L},
        "full_route_rows_per_s": round(rows * L / (ms_full * 1e-3), 1) if not args.no_full else None,
        "full_ms_per_step": round(ms_full, 4) if not args.no_full else None,
        "speedup_vs_full": round(ms_full / ms_step, 3) if not args.no_full else None,
        "relay_layer_rows_per_s": round(rows / (1e-3 * lay_ms[relay_l].mean()), 1) if relay_l else None,
        "anchor_layer_rows_per_s": round(rows / (1e-3 * lay_ms[anchor_l].mean()), 1),
        "relay_layer_us": round(1e3 * float(lay_ms[relay_l].mean()), 2) if relay_l else None,
        "anchor_layer_us": round(1e3 * float(lay_ms[anchor_l].mean()), 2),
        "recall": round(recall, 6),
        "rerouted_frac_relay_layers": round(rer_relay, 4),
        "rerouted_frac_all_layers": round(rer_all, 4),
        "score_pair_frac": round(pair_frac, 4),
        "kernel_ms_per_step": round(path_ms, 4),
        "kernels": kernels,
        "roofline": roofline,
    }

    # ---- CPU baseline: the oracle, single-threaded, on a head subset
    if not args.no_cpu_baseline:
        import oracle
        p = oracle.Problem(hs, hs // group, w.n, w.n, w.d, w.k, w.m, w.r, w.causal, w.gamma, w.seed)
        ref = oracle.new_ledger(p)
        t0 = time.perf_counter()
        for l, (Qs, Ks) in enumerate(cpu_sample):
            if w.is_anchor(l):
                oracle.anchor(p, l, Qs, Ks, ref)
            else:
                oracle.relay(p, l, Qs, Ks, ref)
        dt = time.perf_counter() - t0
        out["cpu_baseline"] = {
            "value": round(p.rows * L / dt, 1), "unit": "rows/s", "cores": 1, "kind": "oracle",
            "sample": f"{hs} of {w.n_heads} query heads ({p.rows} rows) x {L} layers of the same "
                      f"workload, binary64 C oracle, {dt:.1f} s",
        }
    print(json.dumps(out))
    led.close()


if __name__ == "__main__":
    main()
