"""The forward's pair capacity (cfg max_pairs) through the C ABI.

A workspace sized for exactly the (token, expert) pairs the routing needs
gives the same bits as the worst-case workspace; one pair short, the call
still writes the routing record, writes Y = 0, runs no expert FFN (nothing
is touched past the smaller buffers) and unif_moe_forward_status reports
UNIF_ECAPACITY with the number of pairs needed. Layer (bf16 with and
without padding, fp32), block and allocation-free forwards."""
import numpy as np
import pytest
import torch

from paper_2608_10392_amd import _lib
from paper_2608_10392_amd.layer import DeviceLayer, to_device
from synth import block_inputs, generate, get_config, layer_config

pytestmark = pytest.mark.gpu

LAYERS = [  # (label, workload, overrides)
    ("bf16 vit_s16 shape", "vit_s16", dict(n_tokens=3001)),
    ("bf16 padded BERT-base shape", "bert_base_padded", dict(n_tokens=1024)),
    ("bf16 small, split down-projection", "vit_s16", dict(n_tokens=600, d_model=256, n_experts=6,
                                                           n_blocks=8, block_width=64, max_shared=8)),
    ("fp32 tiny", "tiny_f32", dict()),
]


def _pairs(dev):
    r = dev.routing_numpy()
    valid = r["n_res"] > 0
    return int(valid.sum() + r["n_res"][valid].sum())


def _layer(name, over):
    g = generate(get_config(name, **over))
    cfg = layer_config(g["cfg"])
    return g, cfg, DeviceLayer(cfg, g["X"], g["valid"], g["W_router"], g["prototypes"], g["W_up"],
                               g["W_down"], device="cuda:0")


@pytest.mark.parametrize("label,name,over", LAYERS, ids=[l[0] for l in LAYERS])
def test_exact_capacity_and_one_pair_short(label, name, over):
    g, cfg, dev = _layer(name, over)
    print(f"[gpu] capacity {label}: N={cfg['n_tokens']} d={cfg['d_model']} K={cfg['n_experts']} "
          f"B={cfg['n_blocks']} M={cfg['block_width']} {cfg['dtype']}", flush=True)
    dev.forward()
    torch.cuda.synchronize()
    y_ref, r_ref = dev.output_numpy(), dev.routing_numpy()
    status, pairs = _lib.forward_status(cfg, dev.ws_forward)
    assert status == _lib.OK and pairs == _pairs(dev)
    worst = cfg["n_tokens"] * (cfg["n_experts"] + 1)
    assert pairs < worst

    exact = dict(cfg, max_pairs=pairs)
    ws = _lib.alloc_workspace(_lib.layer_forward_workspace_size(exact))
    assert ws.numel() < dev.ws_forward.numel()
    dev.Y.fill_(float("nan"))
    _lib.layer_forward(exact, dev.X, dev.valid, dev.W_router, dev.prototypes, dev.W_up, dev.W_down,
                       dev.Y, ws, routing=dev.routing)
    assert _lib.forward_status(exact, ws) == (_lib.OK, pairs)
    assert np.array_equal(dev.output_numpy(), y_ref), f"{label}: Y differs at the exact capacity"

    short = dict(cfg, max_pairs=pairs - 1)
    ws = _lib.alloc_workspace(_lib.layer_forward_workspace_size(short))
    dev.Y.fill_(float("nan"))
    for v in dev.routing.values():
        v.fill_(-7)
    _lib.layer_forward(short, dev.X, dev.valid, dev.W_router, dev.prototypes, dev.W_up, dev.W_down,
                       dev.Y, ws, routing=dev.routing)
    assert _lib.forward_status(short, ws) == (_lib.ECAPACITY, pairs)
    assert not dev.Y.any().item() and not dev.Y.isnan().any().item(), f"{label}: Y not zero past the capacity"
    r = dev.routing_numpy()
    for k in r_ref:
        assert np.array_equal(r[k], r_ref[k]), f"{label}: record {k} differs past the capacity"

    # the same workspace, a later call within the capacity: OK again
    _lib.layer_forward(dict(cfg, max_pairs=pairs), dev.X, dev.valid, dev.W_router, dev.prototypes,
                       dev.W_up, dev.W_down, dev.Y, _lib.alloc_workspace(
                           _lib.layer_forward_workspace_size(dict(cfg, max_pairs=pairs))), routing=dev.routing)
    torch.cuda.synchronize()
    assert np.array_equal(dev.output_numpy(), y_ref)


def test_block_forward_past_the_capacity():
    g, cfg, dev = _layer("vit_s16", dict(n_tokens=1000))
    blk, X = block_inputs(g, "post", residual=True, eps=1e-6)
    dev.block_forward(blk, X=X)
    torch.cuda.synchronize()
    y_ref = dev.output_numpy()
    pairs = _pairs(dev)
    b = dict(norm="post", residual=True, ln_eps=blk["ln_eps"])
    for k in ("ln_gamma", "ln_beta", "b_up", "b_down"):
        b[k] = to_device(np.asarray(blk[k], np.float32), "f32", dev.device)
    Xd = to_device(X, "bf16", dev.device)
    for cap, expect in ((pairs, _lib.OK), (pairs - 1, _lib.ECAPACITY)):
        c = dict(cfg, max_pairs=cap)
        ws = _lib.alloc_workspace(_lib.block_forward_workspace_size(c, b))
        dev.Y.fill_(float("nan"))
        _lib.block_forward(c, b, Xd, dev.valid, dev.W_router, dev.prototypes, dev.W_up, dev.W_down,
                           dev.Y, ws, routing=dev.routing)
        assert _lib.forward_status(c, ws) == (expect, pairs)
        if expect == _lib.OK:
            assert np.array_equal(dev.output_numpy(), y_ref)
        else:
            assert not dev.Y.any().item() and not dev.Y.isnan().any().item()


def test_static_forward_with_capacity():
    """A layer whose worst-case scratch exceeds the static array runs there
    with a capacity that fits, and matches the workspace forward bit for
    bit."""
    g, cfg, dev = _layer("vit_s16", dict(n_tokens=3001))
    assert _lib.layer_forward_workspace_size(cfg) > _lib.STATIC_WORKSPACE_BYTES
    dev.forward()
    torch.cuda.synchronize()
    y_ref = dev.output_numpy()
    c = dict(cfg, max_pairs=_pairs(dev) + 100)
    assert _lib.layer_forward_workspace_size(c) <= _lib.STATIC_WORKSPACE_BYTES
    dev.Y.fill_(float("nan"))
    _lib.layer_forward_static(c, dev.X, dev.valid, dev.W_router, dev.prototypes, dev.W_up, dev.W_down,
                              dev.Y, routing=dev.routing)
    torch.cuda.synchronize()
    assert np.array_equal(dev.output_numpy(), y_ref)
