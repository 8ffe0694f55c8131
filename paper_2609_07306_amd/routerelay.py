"""ctypes binding of librouterelay.so (C ABI in include/routerelay.h).

Argument marshalling only: every step of the path runs in the library's HIP
kernels.  Tensors are torch device tensors that supply ``data_ptr()``; the
stream is torch's current stream unless one is given.  Importing this module
loads the library and raises ImportError if it has not been built.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "librouterelay.so")

RR_OK, RR_ERR_INVALID, RR_ERR_OOM, RR_ERR_HIP, RR_ERR_STATE, RR_ERR_UNSUPPORTED = 0, -1, -2, -3, -4, -5
RR_F32, RR_BF16 = 0, 1
RR_OPT_SPLIT_RELAY, RR_OPT_ONE_PASS_RELAY = 1, 2

EXPORTED = (
    "rr_ledger_create", "rr_ledger_destroy", "rr_anchor_route", "rr_relay_layer", "rr_full_route",
    "rr_ledger_routes", "rr_ledger_export", "rr_ledger_import", "rr_ledger_relay_stats",
    "rr_ledger_index_bytes", "rr_status_string", "rr_last_error", "rr_profile_start",
    "rr_profile_stop", "rr_unconverged_rows", "rr_set_sweep_cap", "rr_relay_layer_static",
    "rr_pool_chunks", "rr_expand_tokens", "rr_sparse_attention",
)
KERNEL_KINDS = ("full", "anchor", "reroute", "rescore", "relay", "pool", "expand", "attention")


class RRError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{msg} (status {status})")
        self.status = status


class _Config(ctypes.Structure):
    _fields_ = [
        ("n_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32), ("n_q", ctypes.c_int32),
        ("n_k", ctypes.c_int32), ("d", ctypes.c_int32), ("k", ctypes.c_int32), ("m", ctypes.c_int32),
        ("r", ctypes.c_int32), ("dtype", ctypes.c_int32), ("causal", ctypes.c_int32),
        ("gamma", ctypes.c_float), ("options", ctypes.c_uint32), ("seed", ctypes.c_uint64),
        ("n_sink", ctypes.c_int32), ("n_recent", ctypes.c_int32), ("min_reuse", ctypes.c_int32),
        ("reserved", ctypes.c_int32), ("gamma_rows", ctypes.c_void_p), ("k_rows", ctypes.c_void_p),
    ]


class _AttnConfig(ctypes.Structure):
    _fields_ = [
        ("n_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32), ("n_tokens", ctypes.c_int32),
        ("d", ctypes.c_int32), ("chunk", ctypes.c_int32), ("k", ctypes.c_int32), ("causal", ctypes.c_int32),
        ("dtype", ctypes.c_int32), ("scale", ctypes.c_float), ("reserved", ctypes.c_int32),
    ]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built: run `python -m paper_2609_07306_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i32, cfgp = ctypes.c_void_p, ctypes.c_int32, ctypes.POINTER(_Config)
    sig = {
        "rr_ledger_create": (ctypes.c_int, [cfgp, ctypes.POINTER(vp)]),
        "rr_ledger_destroy": (ctypes.c_int, [vp]),
        "rr_anchor_route": (ctypes.c_int, [vp, i32, vp, vp, vp, vp, vp]),
        "rr_relay_layer": (ctypes.c_int, [vp, i32, vp, vp, vp, vp, vp, vp, vp]),
        "rr_full_route": (ctypes.c_int, [cfgp, vp, vp, vp, vp, vp, vp]),
        "rr_ledger_routes": (vp, [vp]),
        "rr_ledger_export": (ctypes.c_int, [vp, vp, vp, vp, vp, vp]),
        "rr_ledger_import": (ctypes.c_int, [vp, i32, vp, vp, vp, vp, vp]),
        "rr_ledger_relay_stats": (ctypes.c_int, [vp, vp, vp, vp, vp]),
        "rr_ledger_index_bytes": (ctypes.c_size_t, [cfgp]),
        "rr_status_string": (ctypes.c_char_p, [ctypes.c_int]),
        "rr_last_error": (ctypes.c_char_p, []),
        "rr_profile_start": (ctypes.c_int, []),
        "rr_profile_stop": (ctypes.c_int, [vp, vp, i32]),
        "rr_unconverged_rows": (ctypes.c_int, [ctypes.POINTER(ctypes.c_uint64)]),
        "rr_set_sweep_cap": (ctypes.c_int, [i32]),
        "rr_relay_layer_static": (ctypes.c_int, [cfgp, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]),
        "rr_pool_chunks": (ctypes.c_int, [vp, i32, i32, i32, i32, i32, vp, vp]),
        "rr_expand_tokens": (ctypes.c_int, [vp, ctypes.c_int64, i32, i32, i32, vp, vp]),
        "rr_sparse_attention": (ctypes.c_int, [ctypes.POINTER(_AttnConfig), vp, vp, vp, vp, vp, vp]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    return lib


lib = _load()


def _check(status: int):
    if status != RR_OK:
        raise RRError(status, lib.rr_last_error().decode())


_RELAY_OPTIONS = {"auto": 0, "split": RR_OPT_SPLIT_RELAY, "one_pass": RR_OPT_ONE_PASS_RELAY}


@dataclass(frozen=True)
class Config:
    """Shape and rule parameters (rr_config)."""
    n_heads: int
    n_kv_heads: int
    n_q: int
    n_k: int
    d: int
    k: int
    m: int = 0
    r: int = 0
    dtype: str = "f32"  # "f32" | "bf16"
    causal: bool = False
    gamma: float = 0.0
    seed: int = 0
    relay: str = "auto"  # relay schedule: "auto" | "one_pass" | "split" (rr_option)
    n_sink: int = 0      # mandatory sentinels: sink chunks ...
    n_recent: int = 0    # ... and recent chunks
    min_reuse: int = 0   # minimum reuse horizon (layers)
    gamma_rows: object = None  # per-row guard margins: float32 device tensor [rows], or None
    k_rows: object = None      # per-row route widths in [1, k]: int32 device tensor [rows], or None

    @property
    def rows(self) -> int:
        return self.n_heads * self.n_q

    @property
    def sent_width(self) -> int:
        return self.m + self.r + self.n_sink + self.n_recent

    def c(self) -> _Config:
        g = None
        if self.gamma_rows is not None:
            t = self.gamma_rows
            if t.dtype != torch.float32 or tuple(t.shape) != (self.rows,):
                raise ValueError("gamma_rows must be a float32 tensor with one entry per row")
            g = _ptr(t)
        kr = None
        if self.k_rows is not None:
            t = self.k_rows
            if t.dtype != torch.int32 or tuple(t.shape) != (self.rows,):
                raise ValueError("k_rows must be an int32 tensor with one entry per row")
            kr = _ptr(t)
        return _Config(self.n_heads, self.n_kv_heads, self.n_q, self.n_k, self.d, self.k, self.m,
                       self.r, RR_BF16 if self.dtype == "bf16" else RR_F32, int(self.causal),
                       float(self.gamma), _RELAY_OPTIONS[self.relay],
                       int(self.seed) & 0xFFFFFFFFFFFFFFFF, int(self.n_sink), int(self.n_recent),
                       int(self.min_reuse), 0, g, kr)

    @staticmethod
    def of(w) -> "Config":
        """From a synth.Workload."""
        return Config(w.n_heads, w.n_kv_heads, w.n, w.nk, w.d, w.k, w.m, w.r, w.dtype, w.causal,
                      w.gamma, w.seed, n_sink=w.n_sink, n_recent=w.n_recent, min_reuse=w.min_reuse)


def _ptr(t):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("tensor must be on the GPU")
    if not t.is_contiguous():
        raise ValueError("tensor must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _inputs(cfg: Config, Q, K):
    want = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    if Q.dtype != want or K.dtype != want:
        raise TypeError(f"Qc/Kc must be {want}")
    if tuple(Q.shape) != (cfg.n_heads, cfg.n_q, cfg.d) or tuple(K.shape) != (cfg.n_kv_heads, cfg.n_k, cfg.d):
        raise ValueError(f"shapes {tuple(Q.shape)}, {tuple(K.shape)} do not match the config")
    return _ptr(Q), _ptr(K)


def _out(t, shape, dtype):
    if t is None:
        return None
    if tuple(t.shape) != tuple(shape) or t.dtype != dtype:
        raise ValueError(f"output must be {dtype} of shape {shape}")
    return _ptr(t)


def profile_start():
    """Start bracketing every library kernel launch with HIP events."""
    _check(lib.rr_profile_start())


def profile_stop():
    """Stop profiling; returns {kind: (total_ms, launches)}."""
    ms = (ctypes.c_double * len(KERNEL_KINDS))()
    n = (ctypes.c_int64 * len(KERNEL_KINDS))()
    _check(lib.rr_profile_stop(ms, n, len(KERNEL_KINDS)))
    return {k: (ms[i], n[i]) for i, k in enumerate(KERNEL_KINDS)}


def unconverged_rows() -> int:
    """Rows (on the current device, since load) whose selection stopped at the sweep cap."""
    c = ctypes.c_uint64()
    _check(lib.rr_unconverged_rows(ctypes.byref(c)))
    return int(c.value)


def set_sweep_cap(cap: int):
    """Test hook: collection sweeps allowed per route tile (0: default)."""
    _check(lib.rr_set_sweep_cap(int(cap)))


def index_bytes(cfg: Config) -> int:
    return int(lib.rr_ledger_index_bytes(ctypes.byref(cfg.c())))


def full_route(cfg: Config, Q, K, routes, scores=None, pairs=None, stream=None):
    """rr_full_route: every row's top-k (Eq. (1)-(2)) into ``routes`` [rows, k] int32."""
    q, k = _inputs(cfg, Q, K)
    _check(lib.rr_full_route(ctypes.byref(cfg.c()), q, k, _out(routes, (cfg.rows, cfg.k), torch.int32),
                             _out(scores, (cfg.rows, cfg.k), torch.float32),
                             _out(pairs, (1,), torch.int64), _stream(stream)))


def relay_static(cfg: Config, layer: int, Q, K, ledger, routes=None, mask=None, pairs=None, n_rerouted=None,
                 stream=None):
    """rr_relay_layer_static: a relay layer on a caller-owned ledger (a dict of
    int32 device tensors as Ledger.export returns), updated in place; the
    library allocates nothing."""
    q, k = _inputs(cfg, Q, K)
    c = cfg
    _check(lib.rr_relay_layer_static(
        ctypes.byref(cfg.c()), layer, q, k, _out(ledger["routes"], (c.rows, c.k), torch.int32),
        _out(ledger["sent"], (c.rows, c.sent_width), torch.int32) if c.sent_width else None,
        _out(ledger["build"], (c.rows,), torch.int32), _out(ledger["age"], (c.rows,), torch.int32),
        _out(routes, (c.rows, c.k), torch.int32), _out(mask, (c.rows,), torch.uint8),
        _out(pairs, (1,), torch.int64), _out(n_rerouted, (1,), torch.int32), _stream(stream)))


class Ledger:
    """rr_ledger: the per-row route ledger on the current device."""

    def __init__(self, cfg: Config):
        self.cfg = cfg
        h = ctypes.c_void_p()
        _check(lib.rr_ledger_create(ctypes.byref(cfg.c()), ctypes.byref(h)))
        self._h = h

    def close(self):
        if getattr(self, "_h", None) and self._h.value:
            lib.rr_ledger_destroy(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    @property
    def handle(self):
        return self._h

    def anchor(self, layer: int, Q, K, routes=None, pairs=None, stream=None):
        q, k = _inputs(self.cfg, Q, K)
        c = self.cfg
        _check(lib.rr_anchor_route(self._h, layer, q, k, _out(routes, (c.rows, c.k), torch.int32),
                                   _out(pairs, (1,), torch.int64), _stream(stream)))

    def relay(self, layer: int, Q, K, routes=None, mask=None, pairs=None, n_rerouted=None, stream=None):
        q, k = _inputs(self.cfg, Q, K)
        c = self.cfg
        _check(lib.rr_relay_layer(self._h, layer, q, k, _out(routes, (c.rows, c.k), torch.int32),
                                  _out(mask, (c.rows,), torch.uint8), _out(pairs, (1,), torch.int64),
                                  _out(n_rerouted, (1,), torch.int32), _stream(stream)))

    def routes_ptr(self) -> int:
        return int(lib.rr_ledger_routes(self._h) or 0)

    def export(self, stream=None):
        """Copies of the ledger state: dict of int32 device tensors."""
        c = self.cfg
        dev = torch.device("cuda", torch.cuda.current_device())
        out = {
            "routes": torch.empty((c.rows, c.k), dtype=torch.int32, device=dev),
            "sent": torch.empty((c.rows, c.sent_width), dtype=torch.int32, device=dev),
            "build": torch.empty((c.rows,), dtype=torch.int32, device=dev),
            "age": torch.empty((c.rows,), dtype=torch.int32, device=dev),
        }
        _check(lib.rr_ledger_export(self._h, _ptr(out["routes"]), _ptr(out["sent"]) if c.sent_width else None,
                                    _ptr(out["build"]), _ptr(out["age"]), _stream(stream)))
        return out

    def import_(self, layer: int, routes, sent, build, age, stream=None):
        c = self.cfg
        _check(lib.rr_ledger_import(self._h, layer, _out(routes, (c.rows, c.k), torch.int32),
                                    _out(sent, (c.rows, c.sent_width), torch.int32) if c.sent_width else None,
                                    _out(build, (c.rows,), torch.int32), _out(age, (c.rows,), torch.int32),
                                    _stream(stream)))

    def relay_stats(self, stream=None):
        c = self.cfg
        dev = torch.device("cuda", torch.cuda.current_device())
        alpha = torch.empty(c.rows, dtype=torch.float32, device=dev)
        beta = torch.empty(c.rows, dtype=torch.float32, device=dev)
        ids = torch.empty(c.rows, dtype=torch.int32, device=dev)
        _check(lib.rr_ledger_relay_stats(self._h, _ptr(alpha), _ptr(beta), _ptr(ids), _stream(stream)))
        return alpha, beta, ids


def to_device(x_dev, dtype: str, device="cuda"):
    """numpy array from synth (binary32 values or bf16 bits) -> torch device tensor."""
    import numpy as np
    if dtype == "bf16":
        t = torch.from_numpy(np.ascontiguousarray(x_dev).view(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(x_dev, dtype=np.float32))
    return t.to(device)


# ------------------------------------------------- either side of the path

def n_chunks(n_tokens: int, chunk: int) -> int:
    return -(-n_tokens // chunk)


def pool_chunks(X, chunk: int, out=None, stream=None):
    """rr_pool_chunks: X [H, n_tokens, d] (float32 or bfloat16 device tensor)
    -> [H, n_chunks, d] chunk means of the same dtype."""
    if X.dim() != 3 or X.dtype not in (torch.float32, torch.bfloat16):
        raise TypeError("X must be a [H, n_tokens, d] float32 or bfloat16 tensor")
    H, n, d = X.shape
    shape = (H, n_chunks(n, chunk), d)
    if out is None:
        out = torch.empty(shape, dtype=X.dtype, device=X.device)
    dt = RR_BF16 if X.dtype == torch.bfloat16 else RR_F32
    _check(lib.rr_pool_chunks(_ptr(X), H, n, d, chunk, dt, _out(out, shape, X.dtype), _stream(stream)))
    return out


def expand_tokens(routes, chunk: int, n_tokens: int, out=None, stream=None):
    """rr_expand_tokens: routes [rows, k] int32 -> token ids [rows, k*chunk]."""
    if routes.dim() != 2 or routes.dtype != torch.int32:
        raise TypeError("routes must be a [rows, k] int32 tensor")
    rows, k = routes.shape
    shape = (rows, k * chunk)
    if out is None:
        out = torch.empty(shape, dtype=torch.int32, device=routes.device)
    _check(lib.rr_expand_tokens(_ptr(routes), rows, k, chunk, n_tokens, _out(out, shape, torch.int32),
                                _stream(stream)))
    return out


def sparse_attention(Q, K, V, routes, chunk: int, causal: bool, scale: float = 0.0, out=None, stream=None):
    """rr_sparse_attention: Q [H, n, d], K and V [H_kv, n, d] bfloat16,
    routes [H * n_chunks, k] int32 -> O [H, n, d] bfloat16."""
    for t in (Q, K, V):
        if t.dim() != 3 or t.dtype != torch.bfloat16:
            raise TypeError("Q, K and V must be 3-d bfloat16 tensors")
    H, n, d = Q.shape
    Hkv = K.shape[0]
    if tuple(K.shape) != (Hkv, n, d) or tuple(V.shape) != (Hkv, n, d):
        raise ValueError("K and V must be [H_kv, n_tokens, d]")
    nc = n_chunks(n, chunk)
    if routes.dim() != 2 or routes.dtype != torch.int32 or routes.shape[0] != H * nc:
        raise ValueError("routes must be [H * n_chunks, k] int32")
    if out is None:
        out = torch.empty_like(Q)
    cfg = _AttnConfig(H, Hkv, n, d, chunk, routes.shape[1], int(causal), RR_BF16, float(scale), 0)
    _check(lib.rr_sparse_attention(ctypes.byref(cfg), _ptr(Q), _ptr(K), _ptr(V), _ptr(routes),
                                   _out(out, (H, n, d), torch.bfloat16), _stream(stream)))
    return out

