"""GPU parity of the steps either side of route maintenance, through the C
ABI, against the oracle: chunk pooling and token expansion (Sec. 2.1) and
sparse attention over the routed chunks' tokens (Sec. 2.2 Eq. (3)).

Tolerances, from the arithmetic: pooling sums in binary32 (error at most
len * 2^-24 * mean|x| per feature) and rounds bf16 outputs to nearest even
(2^-8 relative).  Attention takes exact bf16 products with binary32 sums,
rounds each softmax weight to bf16 before the value product (relative error
at most 2^-8, so the output moves by at most 2^-8 * sum_u w_u |v_u|, which
the oracle computes by attending over |V|), and rounds the output to bf16
(2^-8 relative)."""
import sys

import numpy as np
import pytest
import torch

from oracle import consumer as oc
from paper_2609_07306_amd import synth

pytestmark = pytest.mark.gpu
U8 = 2.0 ** -8


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


def _bf16(rng, *shape, scale=1.0):
    """(bf16 bits as a device tensor, the same values widened to binary32)."""
    x = (rng.standard_normal(shape) * scale).astype(np.float32)
    bits = synth.bf16_round(x)
    return torch.from_numpy(bits.view(np.int16)).to("cuda").view(torch.bfloat16), synth.bf16_widen(bits)


def _to_f32(t):
    return t.float().cpu().numpy()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("n,chunk,d", [(100, 7, 16), (512, 64, 128), (1000, 256, 128), (37, 1, 8), (50, 64, 64),
                                       (300, 128, 136)])
def test_pool_parity(dtype, n, chunk, d):
    rr = rrmod()
    rng = np.random.default_rng(n * 7 + d)
    note(f"pool {dtype} n={n} chunk={chunk} d={d}")
    H = 3
    if dtype == "bf16":
        X, Xf = _bf16(rng, H, n, d)
    else:
        Xf = rng.standard_normal((H, n, d)).astype(np.float32)
        X = torch.from_numpy(Xf).to("cuda")
    got = _to_f32(rr.pool_chunks(X, chunk))
    torch.cuda.synchronize()
    exact = oc.pool_chunks(Xf, chunk)
    nc = exact.shape[1]
    lens = np.array([min((j + 1) * chunk, n) - j * chunk for j in range(nc)], np.float64)
    mean_abs = oc.pool_chunks(np.abs(Xf), chunk)
    tol = (lens[None, :, None] + 2) * 2.0 ** -24 * mean_abs + 2.0 ** -24 * np.abs(exact)
    if dtype == "bf16":
        tol = tol + U8 * np.abs(exact)
    err = np.abs(got - exact)
    assert np.all(err <= tol + 1e-30), f"max excess {np.max(err - tol)}"


def test_expand_parity():
    rr = rrmod()
    rng = np.random.default_rng(5)
    n, chunk, k = 1000, 48, 7
    nc = oc.n_chunks(n, chunk)
    routes = rng.integers(-1, nc + 3, size=(300, k)).astype(np.int32)
    routes[0] = [nc - 1, -1, 0, nc, nc + 2, 3, -1]  # the short last chunk, empty and out-of-range slots
    note("token expansion")
    got = rr.expand_tokens(torch.from_numpy(routes).to("cuda"), chunk, n).cpu().numpy()
    np.testing.assert_array_equal(got, oc.expand_tokens(routes, chunk, n))


def _routes(rng, H, nc, k, causal):
    """Distinct admissible chunks per row (for causal rows j <= i), with -1
    padding where fewer exist, plus an occasional inadmissible slot (a chunk
    after i, an out-of-range id) that must be skipped."""
    R = np.full((H * nc, k), -1, np.int32)
    for h in range(H):
        for i in range(nc):
            pool = np.arange(i + 1) if causal else np.arange(nc)
            take = rng.permutation(pool)[:k]
            R[h * nc + i, :len(take)] = take
            if len(take) < k and rng.random() < 0.5:
                R[h * nc + i, len(take)] = nc + 1 if not causal or i + 1 >= nc else rng.integers(i + 1, nc)
    return R


def _check_attention(rr, H, Hkv, n, chunk, d, k, causal, seed, routes=None):
    rng = np.random.default_rng(seed)
    Q, Qf = _bf16(rng, H, n, d)
    K, Kf = _bf16(rng, Hkv, n, d)
    V, Vf = _bf16(rng, Hkv, n, d)
    nc = oc.n_chunks(n, chunk)
    if routes is None:
        routes = _routes(rng, H, nc, k, causal)
    O = rr.sparse_attention(Q, K, V, torch.from_numpy(routes).to("cuda"), chunk, causal)
    got = _to_f32(O)
    torch.cuda.synchronize()
    exact = oc.sparse_attention(Qf, Kf, Vf, routes, chunk, causal)
    wabs = oc.sparse_attention(Qf, Kf, np.abs(Vf), routes, chunk, causal)
    tol = 1.05 * U8 * (wabs + np.abs(exact)) + 1e-6
    err = np.abs(got - exact)
    bad = np.argwhere(err > tol)
    assert len(bad) == 0, f"{len(bad)} outputs beyond tolerance, first {bad[:4].tolist()}: " \
                          f"{got[tuple(bad[0])]} vs {exact[tuple(bad[0])]} (tol {tol[tuple(bad[0])]})"
    return got, exact


ATTN_CASES = [
    # name, H, H_kv, n_tokens, chunk, d, k, causal
    ("d128_c64", 4, 2, 640, 64, 128, 6, False),
    ("d128_c64_causal", 4, 2, 640, 64, 128, 6, True),
    ("d64_c32_ragged_causal", 2, 1, 333, 32, 64, 5, True),
    ("d128_c100_ragged_causal", 2, 2, 450, 100, 128, 3, True),
    ("d128_c256_causal", 2, 1, 1024, 256, 128, 3, True),
    ("d128_c300_two_tiles", 2, 1, 900, 300, 128, 2, False),
    ("d128_c300_two_tiles_causal", 2, 1, 900, 300, 128, 3, True),
    ("d64_one_token_chunks", 1, 1, 100, 1, 64, 7, False),
    ("d128_every_chunk", 2, 2, 256, 64, 128, 4, True),
    ("d64_short_sequence", 2, 2, 20, 64, 64, 2, True),
]


@pytest.mark.parametrize("case", ATTN_CASES, ids=[c[0] for c in ATTN_CASES])
def test_attention_parity(case):
    rr = rrmod()
    name, H, Hkv, n, chunk, d, k, causal = case
    note(f"sparse attention parity: {case}")
    _check_attention(rr, H, Hkv, n, chunk, d, k, causal, seed=len(name) * 31 + n)


def test_attention_empty_and_inadmissible_routes_give_zero():
    rr = rrmod()
    H, n, chunk, d, k = 2, 200, 32, 128, 3
    nc = oc.n_chunks(n, chunk)
    R = np.full((H * nc, k), -1, np.int32)
    R[1] = [5, nc + 4, -1]  # chunk 1 (causal) routes only to a later chunk and an invalid id
    note("empty routes")
    got, exact = _check_attention(rr, H, H, n, chunk, d, k, True, seed=3, routes=R)
    assert not got.any() and not exact.any()


def test_attention_on_library_routes_full_size_sampled():
    """The causal GQA prefill shape (131072 tokens in 256-token chunks, 32
    query heads on 8 key heads, d = 128, top-32 routes from the library's own
    full routing of the pooled chunk representations): 96 sampled query
    tokens against the oracle."""
    rr = rrmod()
    H, Hkv, n, chunk, d, k = 32, 8, 131072, 256, 128, 32
    nc = n // chunk
    gen = torch.Generator(device="cuda").manual_seed(11)
    note("full-size attention: generating tokens")
    # tokens of a chunk scatter around a chunk centre, so that routing on the
    # pooled representations has structure
    def tokens(heads):
        c = torch.randn((heads, nc, 1, d), generator=gen, device="cuda")
        x = c + 0.5 * torch.randn((heads, nc, chunk, d), generator=gen, device="cuda")
        return (x.reshape(heads, n, d) / d ** 0.5).to(torch.bfloat16)
    Q, K, V = tokens(H), tokens(Hkv), tokens(Hkv)
    Qc, Kc = rr.pool_chunks(Q, chunk), rr.pool_chunks(K, chunk)
    cfg = rr.Config(H, Hkv, nc, nc, d, k, 0, 0, "bf16", True)
    routes = torch.empty((H * nc, k), dtype=torch.int32, device="cuda")
    rr.full_route(cfg, Qc, Kc, routes)
    O = rr.sparse_attention(Q, K, V, routes, chunk, True)
    torch.cuda.synchronize()
    note("full-size attention: oracle on sampled rows")
    rng = np.random.default_rng(12)
    rows = [(int(h), int(t)) for h, t in zip(rng.integers(0, H, 96), rng.integers(0, n, 96))]
    rows += [(0, 0), (H - 1, n - 1), (5, 255), (5, 256)]
    Rn = routes.cpu().numpy()
    Kf, Vf = _to_f32(K), _to_f32(V)
    Qrows = np.stack([_to_f32(Q[h, t]) for h, t in rows])
    got = np.stack([_to_f32(O[h, t]) for h, t in rows])
    for idx, (h, t) in enumerate(rows):
        # a one-row problem holding the sampled query and its route row
        i = t // chunk
        g = h // (H // Hkv)
        Q1 = np.zeros((1, n, d), np.float32)
        Q1[0, t] = Qrows[idx]
        R1 = np.full((nc, k), -1, np.int32)
        R1[i] = Rn[h * nc + i]
        ex = oc.sparse_attention(Q1, Kf[g:g + 1], Vf[g:g + 1], R1, chunk, True, rows=[(0, t)])[0]
        wa = oc.sparse_attention(Q1, Kf[g:g + 1], np.abs(Vf[g:g + 1]), R1, chunk, True, rows=[(0, t)])[0]
        tol = 1.05 * U8 * (wa + np.abs(ex)) + 1e-6
        assert np.all(np.abs(got[idx] - ex) <= tol), f"row {(h, t)}: max err {np.max(np.abs(got[idx] - ex))}"
