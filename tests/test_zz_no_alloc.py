"""unif_moe_layer_forward_static (the forward without a caller workspace,
for callers that cannot allocate) against unif_moe_layer_forward: the same
bits for Y and the routing record, on two calls in a row on one GPU, the
second with a smaller layer (the static scratch keeps the first call's
contents). Both calls go through the C ABI."""
import numpy as np
import pytest
import torch

from paper_2608_10392_amd import _lib
from paper_2608_10392_amd.layer import DeviceLayer
from synth import generate, get_config, layer_config

pytestmark = pytest.mark.gpu

CASES = [  # (label, config overrides), called in this order
    ("larger", dict(n_tokens=3001, d_model=256, n_experts=6, n_blocks=8, block_width=64, max_shared=8)),
    ("smaller", dict(n_tokens=517, d_model=128, n_experts=4, n_blocks=4, block_width=128, max_shared=4)),
]


def _layer(over):
    g = generate(get_config("vit_s16", **over))
    cfg = layer_config(g["cfg"])
    assert _lib.layer_forward_workspace_size(cfg) <= _lib.STATIC_WORKSPACE_BYTES
    return cfg, DeviceLayer(cfg, g["X"], g["valid"], g["W_router"], g["prototypes"], g["W_up"],
                            g["W_down"], device="cuda:0")


def test_static_forward_matches_workspace_forward():
    for label, over in CASES:
        cfg, dev = _layer(over)
        print(f"[gpu] static forward {label}: N={cfg['n_tokens']} d={cfg['d_model']} "
              f"K={cfg['n_experts']} B={cfg['n_blocks']} M={cfg['block_width']}", flush=True)
        dev.forward()
        torch.cuda.synchronize()
        y_ref, r_ref = dev.output_numpy(), dev.routing_numpy()
        dev.Y.fill_(float("nan"))
        for v in dev.routing.values():
            v.fill_(-7)
        _lib.layer_forward_static(cfg, dev.X, dev.valid, dev.W_router, dev.prototypes, dev.W_up,
                                  dev.W_down, dev.Y, routing=dev.routing)
        torch.cuda.synchronize()
        y, r = dev.output_numpy(), dev.routing_numpy()
        assert np.array_equal(y, y_ref), f"{label}: Y differs"
        for k in r_ref:
            assert np.array_equal(r[k], r_ref[k]), f"{label}: record {k} differs"


def test_static_forward_rejects_large_layer():
    cfg = layer_config(get_config("vit_b16"))
    assert _lib.layer_forward_workspace_size(cfg) > _lib.STATIC_WORKSPACE_BYTES
    with pytest.raises(_lib.UnifMoeError) as e:
        _lib.layer_forward_static(cfg, 1, None, 1, 1, 1, 1, 1)
    assert e.value.status == _lib.EWORKSPACE
