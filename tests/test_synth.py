"""The seeded input generator: shapes, determinism, bf16 rounding against
torch's own conversion, the AR(1) drift statistics and near-tie duplicates."""
import numpy as np
import pytest
import torch

from paper_2609_07306_amd import synth


def test_bf16_round_matches_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(100000).astype(np.float32) * 10.0 ** rng.integers(-8, 8, 100000),
                        np.array([0.0, -0.0, 1.0, -1.0, 3.0e38, 1.00390625, 1.01171875], np.float32)])
    x = x.astype(np.float32)
    ours = synth.bf16_round(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(ours, ref)
    back = torch.from_numpy(ref.view(np.int16)).view(torch.bfloat16).float().numpy()
    np.testing.assert_array_equal(synth.bf16_widen(ours), back)


@pytest.mark.parametrize("name", ["tiny", "drift", "scale", "gqa", "longctx"])
def test_presets_shapes(name):
    w = synth.preset(name)
    small = w.with_(n=min(w.n, 64), n_layers=2)
    out = list(synth.Generator(small))
    assert len(out) == 2
    _, Qf, Kf, Qd, Kd = out[0]
    assert Qf.shape == (w.n_heads, small.n, w.d) and Kf.shape == (w.n_kv_heads, small.n, w.d)
    assert Qf.dtype == np.float32
    assert Qd.dtype == (np.uint16 if w.dtype == "bf16" else np.float32)
    if w.dtype == "bf16":
        np.testing.assert_array_equal(synth.bf16_widen(Qd), Qf)


def test_deterministic_and_seeded():
    w = synth.preset("tiny", n_layers=3)
    a = synth.layers(w)
    b = synth.layers(w)
    c = synth.layers(w.with_(seed=1))
    for x, y in zip(a, b):
        np.testing.assert_array_equal(x[0], y[0])
        np.testing.assert_array_equal(x[1], y[1])
    assert not np.array_equal(a[0][0], c[0][0])


def test_drift_correlation():
    rho = 0.3
    w = synth.preset("tiny", n_layers=2, rho=rho, n=512, d=128)
    (_, Q0, K0, _, _), (_, Q1, K1, _, _) = list(synth.Generator(w))
    # the innovation has variance rho^2/d per element and is independent of X^l
    dq = Q1 - np.sqrt(1 - rho ** 2) * Q0
    assert np.var(dq) == pytest.approx(rho ** 2 / w.d, rel=0.03)
    assert abs(np.mean(dq * Q0)) < 5 * np.std(dq * Q0) / np.sqrt(dq.size)


def test_near_tie_duplicates():
    w = synth.preset("longctx", n=256, n_layers=2, n_heads=2, n_kv_heads=2)
    for _, Qf, Kf, _, _ in synth.Generator(w):
        for g in range(2):
            D = np.linalg.norm(Kf[g][:, None, :] - Kf[g][None, :, :], axis=-1)
            np.fill_diagonal(D, np.inf)
            close = (D.min(1) < 0.05).sum()
            assert close >= 256 // 4
