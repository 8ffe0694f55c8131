"""rr_relay_layer_static, the relay entry point that allocates nothing (its
scratch is the library's static device area), against rr_relay_layer on the
same ledger state: routes, sentinels, build layers, ages, mask, score pairs
and rerouted-row counts must be identical, call after call, including a
second configuration smaller than the first that reuses the same area."""
import dataclasses

import numpy as np
import pytest
import torch

from paper_2609_07306_amd import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    torch.cuda.set_device(0)
    yield


def _compare(w, relay, n_layers):
    from paper_2609_07306_amd import routerelay as rr
    dev = torch.device("cuda", 0)
    cfg = dataclasses.replace(rr.Config.of(w), relay=relay)
    led = rr.Ledger(cfg)
    lay = synth.layers(w.with_(n_layers=n_layers))
    Q0, K0 = rr.to_device(lay[0][2], w.dtype, dev), rr.to_device(lay[0][3], w.dtype, dev)
    led.anchor(0, Q0, K0)
    own = led.export()  # the caller's ledger, allocated before the calls under test
    outs = [dict(routes=torch.full((cfg.rows, cfg.k), -7, dtype=torch.int32, device=dev),
                 mask=torch.full((cfg.rows,), 7, dtype=torch.uint8, device=dev),
                 pairs=torch.zeros(1, dtype=torch.int64, device=dev),
                 n_rerouted=torch.zeros(1, dtype=torch.int32, device=dev)) for _ in range(2)]
    total = 0
    for layer in range(1, n_layers):
        Q, K = rr.to_device(lay[layer][2], w.dtype, dev), rr.to_device(lay[layer][3], w.dtype, dev)
        led.relay(layer, Q, K, **outs[0])
        rr.relay_static(cfg, layer, Q, K, own, **outs[1])
        torch.cuda.synchronize()
        for key in ("routes", "mask", "pairs", "n_rerouted"):
            assert torch.equal(outs[0][key], outs[1][key]), f"{w.name} {relay} layer {layer}: {key} differs"
        ref = led.export()
        torch.cuda.synchronize()
        for key in ("routes", "sent", "build", "age"):
            assert torch.equal(ref[key], own[key]), f"{w.name} {relay} layer {layer}: ledger {key} differs"
        total += int(outs[0]["n_rerouted"].item())
    led.close()
    return total


@pytest.mark.parametrize("relay", ["split", "one_pass"])
def test_static_relay_matches_ledger_relay(relay):
    # a larger configuration, then a smaller one on the same static area
    big = synth.preset("scale", n_heads=64, n_kv_heads=64, n=256, rho=0.05)
    small = synth.preset("gqa", n_heads=8, n_kv_heads=2, n=160, rho=0.05)
    rerouted = _compare(big, relay, 4) + _compare(small, relay, 4)
    assert rerouted > 0


def test_static_relay_refuses_beyond_its_area():
    from paper_2609_07306_amd import routerelay as rr
    cfg = rr.Config(64, 64, 8192, 8192, 128, 32, 16, 16, "bf16")
    with pytest.raises(rr.RRError) as e:
        rr.relay_static(cfg, 1, torch.empty((64, 8192, 128), dtype=torch.bfloat16, device="cuda"),
                        torch.empty((64, 8192, 128), dtype=torch.bfloat16, device="cuda"),
                        {"routes": torch.empty((cfg.rows, 32), dtype=torch.int32, device="cuda"),
                         "sent": torch.empty((cfg.rows, 32), dtype=torch.int32, device="cuda"),
                         "build": torch.empty(cfg.rows, dtype=torch.int32, device="cuda"),
                         "age": torch.empty(cfg.rows, dtype=torch.int32, device="cuda")})
    assert e.value.status == rr.RR_ERR_UNSUPPORTED
