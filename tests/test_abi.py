"""The C ABI library loads, exports every symbol the header declares, and
rejects invalid arguments before it touches the GPU (these run without one)."""
import ctypes
import math
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "routerelay.h")


def _rr():
    from paper_2609_07306_amd import routerelay
    return routerelay


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(rr_[a-z_]+)\s*\(", src)))


def test_header_declares_the_path():
    names = declared_functions()
    for f in ("rr_ledger_create", "rr_ledger_destroy", "rr_anchor_route", "rr_relay_layer",
              "rr_full_route"):
        assert f in names


def test_library_exports_every_declared_symbol():
    rr = _rr()
    lib = ctypes.CDLL(rr.LIB_PATH)
    for name in declared_functions():
        assert hasattr(lib, name), name
    assert set(rr.EXPORTED) == set(declared_functions())


def test_config_struct_layout():
    rr = _rr()
    assert ctypes.sizeof(rr._Config) == 88
    assert rr._Config.seed.offset == 48 and rr._Config.gamma.offset == 40
    assert rr._Config.n_sink.offset == 56 and rr._Config.reserved.offset == 68
    assert rr._Config.gamma_rows.offset == 72 and rr._Config.k_rows.offset == 80


def test_status_strings():
    rr = _rr()
    for s in range(-5, 1):
        assert rr.lib.rr_status_string(s)
    assert rr.lib.rr_last_error() is not None


def _cfg(**kw):
    rr = _rr()
    base = dict(n_heads=2, n_kv_heads=1, n_q=64, n_k=64, d=64, k=8, m=4, r=4)
    base.update(kw)
    return rr.Config(**base)


@pytest.mark.parametrize("kw,status", [
    (dict(k=0), -1), (dict(k=65), -1), (dict(m=-1), -1), (dict(n_kv_heads=3), -1),
    (dict(n_q=0), -1), (dict(causal=True, n_q=32), -1), (dict(gamma=math.nan), -1),
    (dict(d=48), -5), (dict(d=256), -5), (dict(k=60, m=70), -5), (dict(n_k=9000, n_q=9000), -5),
    (dict(k=64, m=64, r=200, n_k=4096), -5),
    (dict(n_sink=-1), -1), (dict(n_recent=-2), -1), (dict(min_reuse=-1), -1),
    (dict(k=32, m=32, r=160, n_sink=16, n_recent=17, n_k=4096, n_q=4096), -5),
])
def test_invalid_configs_rejected_before_any_launch(kw, status):
    rr = _rr()
    cfg = _cfg(**kw)
    h = ctypes.c_void_p()
    got = rr.lib.rr_ledger_create(ctypes.byref(cfg.c()), ctypes.byref(h))
    assert got == status, rr.lib.rr_last_error()
    assert not h.value
    assert rr.lib.rr_last_error()
    # the stateless path validates the same way (m and r are ignored there)
    if not set(kw) & {"m", "r", "n_sink", "n_recent", "min_reuse"}:
        fake = ctypes.c_void_p(0x1000)
        got = rr.lib.rr_full_route(ctypes.byref(cfg.c()), fake, fake, fake, None, None, None)
        assert got == status


@pytest.mark.parametrize("options", [3, 4, 0x80000000])
def test_invalid_options_rejected(options):
    """rr_config.options: the two relay schedules exclude each other; other
    bits are unknown."""
    rr = _rr()
    c = _cfg().c()
    c.options = options
    h = ctypes.c_void_p()
    assert rr.lib.rr_ledger_create(ctypes.byref(c), ctypes.byref(h)) == -1
    assert not h.value


def test_one_pass_relay_beyond_lds_rejected():
    """RR_OPT_ONE_PASS_RELAY where a tile's ledger bitmaps exceed its LDS
    (n_k = 8192) is refused before anything is allocated."""
    rr = _rr()
    h = ctypes.c_void_p()
    c = _cfg(n_q=8192, n_k=8192, d=128, k=32, m=16, r=16).c()
    c.options = rr.RR_OPT_ONE_PASS_RELAY
    assert rr.lib.rr_ledger_create(ctypes.byref(c), ctypes.byref(h)) == -5
    assert b"one-pass" in rr.lib.rr_last_error()
    assert not h.value


def test_kernel_kinds_match_binding():
    """The binding sizes its profile arrays from the header's kernel kinds."""
    rr = _rr()
    src = open(HEADER).read()
    kinds = dict((n, int(v)) for n, v in re.findall(r"RR_KERNEL_([A-Z]+)\s*=\s*(\d+)", src))
    n = kinds.pop("KINDS")
    assert len(rr.KERNEL_KINDS) == n
    for name, v in kinds.items():
        assert rr.KERNEL_KINDS[v] == name.lower()


def test_null_arguments():
    rr = _rr()
    assert rr.lib.rr_ledger_destroy(None) == 0
    assert rr.lib.rr_anchor_route(None, 0, None, None, None, None, None) == -1
    assert rr.lib.rr_relay_layer(None, 0, None, None, None, None, None, None, None) == -1
    cfg = _cfg()
    assert rr.lib.rr_full_route(ctypes.byref(cfg.c()), None, None, None, None, None, None) == -1
    assert rr.lib.rr_ledger_create(None, None) == -1
    assert rr.lib.rr_ledger_routes(None) is None


def test_reserved_config_field_must_be_zero():
    rr = _rr()
    c = _cfg().c()
    c.reserved = 1
    h = ctypes.c_void_p()
    assert rr.lib.rr_ledger_create(ctypes.byref(c), ctypes.byref(h)) == -1
    assert not h.value


def test_ledger_index_bytes_counts_mandatory_slots():
    rr = _rr()
    cfg = rr.Config(1, 1, 1024, 1024, 128, 32, 16, 16, n_sink=2, n_recent=6)
    assert rr.index_bytes(cfg) == 1024 * (64 + 8) * 4


def test_ledger_index_bytes_paper_figure():
    """Sec. 4.4: n_q = 1024 rows with c = k+m+r = 64 int32 ids take 256 KB."""
    rr = _rr()
    cfg = rr.Config(1, 1, 1024, 1024, 128, 32, 16, 16)
    assert rr.index_bytes(cfg) == 256 * 1024


def test_profile_stop_rejects_short_arrays():
    """rr_profile_stop takes the length of its output arrays: a length below
    RR_KERNEL_KINDS is refused before anything is written (an earlier
    signature without the length let a binding sized for fewer kinds overrun
    its arrays)."""
    rr = _rr()
    n = len(rr.KERNEL_KINDS)
    ms = (ctypes.c_double * (n + 2))(*([-7.0] * (n + 2)))
    cnt = (ctypes.c_int64 * (n + 2))(*([-7] * (n + 2)))
    assert rr.lib.rr_profile_start() == 0
    assert rr.lib.rr_profile_stop(ms, cnt, n - 1) == -1
    assert b"RR_KERNEL_KINDS" in rr.lib.rr_last_error()
    assert list(ms) == [-7.0] * (n + 2) and list(cnt) == [-7] * (n + 2)
    # the full length succeeds and writes exactly RR_KERNEL_KINDS entries
    # (nothing was launched, so every kind reads zero)
    assert rr.lib.rr_profile_stop(ms, cnt, n + 2) == 0
    assert list(ms[:n]) == [0.0] * n and list(cnt[:n]) == [0] * n
    assert list(ms[n:]) == [-7.0, -7.0] and list(cnt[n:]) == [-7, -7]
    # NULL arrays need no length
    assert rr.lib.rr_profile_stop(None, None, 0) == 0


def test_sweep_cap_hook_validates():
    rr = _rr()
    assert rr.lib.rr_set_sweep_cap(-1) == -1
    assert rr.lib.rr_set_sweep_cap(0) == 0
    assert rr.lib.rr_unconverged_rows(None) == -1


def test_attention_config_layout():
    rr = _rr()
    assert ctypes.sizeof(rr._AttnConfig) == 40
    assert rr._AttnConfig.scale.offset == 32 and rr._AttnConfig.reserved.offset == 36


def _attn_cfg(rr, **kw):
    base = dict(n_heads=4, n_kv_heads=2, n_tokens=512, d=128, chunk=64, k=4, causal=1, dtype=rr.RR_BF16,
                scale=0.0, reserved=0)
    base.update(kw)
    return rr._AttnConfig(*base.values())


# pointers that are never dereferenced: every call below is refused by the
# host-side checks before any launch
FAKE = ctypes.c_void_p(0x1000)


@pytest.mark.parametrize("kw,status", [
    ({"n_heads": 3}, -1), ({"n_tokens": 0}, -1), ({"chunk": 0}, -1), ({"k": 0}, -1), ({"k": 257}, -1),
    ({"causal": 2}, -1), ({"reserved": 1}, -1), ({"scale": -1.0}, -1), ({"scale": float("inf")}, -1),
    ({"dtype": 7}, -1), ({"dtype": 0}, -5), ({"d": 96}, -5), ({"d": 256}, -5),
])
def test_sparse_attention_rejects_bad_configs(kw, status):
    rr = _rr()
    c = _attn_cfg(rr, **kw)
    assert rr.lib.rr_sparse_attention(ctypes.byref(c), FAKE, FAKE, FAKE, FAKE, FAKE, None) == status


def test_consumer_calls_reject_null_and_bad_sizes():
    rr = _rr()
    c = _attn_cfg(rr)
    assert rr.lib.rr_sparse_attention(None, FAKE, FAKE, FAKE, FAKE, FAKE, None) == -1
    assert rr.lib.rr_sparse_attention(ctypes.byref(c), FAKE, None, FAKE, FAKE, FAKE, None) == -1
    assert rr.lib.rr_pool_chunks(None, 1, 64, 128, 8, rr.RR_BF16, FAKE, None) == -1
    for h, n, d, ch, dt in ((0, 64, 128, 8, 1), (1, 0, 128, 8, 1), (1, 64, 12, 8, 1), (1, 64, 2048, 8, 1),
                            (1, 64, 128, 0, 1), (1, 64, 128, 8, 5)):
        assert rr.lib.rr_pool_chunks(FAKE, h, n, d, ch, dt, FAKE, None) == -1
    assert rr.lib.rr_expand_tokens(None, 1, 4, 8, 64, FAKE, None) == -1
    for rows, k, ch, n in ((0, 4, 8, 64), (1, 0, 8, 64), (1, 4, 0, 64), (1, 4, 8, 0), (1, 70000, 70000, 64)):
        assert rr.lib.rr_expand_tokens(FAKE, rows, k, ch, n, FAKE, None) == -1
    assert b"" != rr.lib.rr_last_error()
