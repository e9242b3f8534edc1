"""Workspace discipline of every entry point that takes one (MI355X only).

Each call gets a workspace of exactly the reported size inside a larger
buffer whose guard bands before and after hold a known byte pattern, and
whose own bytes start as either zeros or a pattern (0xA5 and NaN-like
0xFF bytes). Checked:
  * no byte of either guard band changes (nothing is written outside the
    reported size);
  * the outputs are bitwise the same whatever the workspace held before the
    call (no result depends on uninitialised workspace memory), and the
    workspace may start at any byte offset (the size covers the library's
    own alignment).
"""
import numpy as np
import pytest

from synth import generate, get_config, layer_config, upstream_grad

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

GUARD = 4096


def fenced(nbytes, fill, offset, dev):
    """A workspace view of nbytes at byte offset `offset` past a guard band,
    inside a buffer with a guard band after it."""
    buf = torch.empty(GUARD + offset + nbytes + GUARD, dtype=torch.uint8, device=dev)
    buf.fill_(0x5A)
    ws = buf[GUARD + offset: GUARD + offset + nbytes]
    ws.fill_(fill)
    return buf, ws


def guards_intact(buf, offset, nbytes):
    lo = buf[:GUARD + offset]
    hi = buf[GUARD + offset + nbytes:]
    return bool((lo == 0x5A).all()) and bool((hi == 0x5A).all())


def run_fenced(call, nbytes, dev):
    outs = []
    for fill, offset in ((0x00, 0), (0xA5, 3), (0xFF, 200)):
        buf, ws = fenced(nbytes, fill, offset, dev)
        got = call(ws)
        torch.cuda.synchronize()
        assert guards_intact(buf, offset, nbytes), f"guard band changed (fill {fill:#x}, offset {offset})"
        outs.append({k: v.clone() for k, v in got.items()})
    for o in outs[1:]:
        for k in o:
            assert torch.equal(o[k].view(torch.uint8), outs[0][k].view(torch.uint8)), \
                f"{k} depends on the workspace's prior contents"


CASES = {
    "bf16": get_config("vit_s16", n_tokens=1500, d_model=384, n_experts=8, n_blocks=8, block_width=192,
                       max_shared=8),
    "f32": get_config("tiny_f32", n_tokens=300, d_model=96, n_experts=5, n_blocks=3, block_width=40,
                      max_shared=3),
}


@pytest.mark.parametrize("name", list(CASES))
def test_workspace_guards_and_independence(name):
    from paper_2608_10392_amd import _lib
    from paper_2608_10392_amd.layer import DeviceLayer
    g = generate(CASES[name])
    cfg = layer_config(g["cfg"])
    print(f"\n[gpu] workspace canaries {name}", flush=True)
    dev = DeviceLayer(cfg, g["X"], g["valid"], g["W_router"], g["prototypes"], g["W_up"], g["W_down"])
    d0 = dev.device
    N, K = cfg["n_tokens"], cfg["n_experts"]

    def fwd(ws):
        _lib.layer_forward(cfg, dev.X, dev.valid, dev.W_router, dev.prototypes, dev.W_up, dev.W_down,
                           dev.Y, ws)
        return {"Y": dev.Y}
    run_fenced(fwd, _lib.layer_forward_workspace_size(cfg), d0)

    def route(ws):
        out = _lib.alloc_routing(N, K, d0)
        _lib.route(cfg, dev.X, dev.valid, dev.W_router, dev.prototypes, out, ws)
        return out
    run_fenced(route, _lib.route_workspace_size(cfg), d0)

    def stats(ws):
        st = _lib.stats(cfg, dev.routing, dev.valid, ws)
        return {"hist_k": torch.tensor(st["hist_k"]), "blocks": torch.tensor([st["activated_blocks"]])}
    dev.forward()
    run_fenced(stats, _lib.stats_workspace_size(cfg), d0)

    blk = dict(norm="pre", residual=True, ln_eps=1e-6,
               ln_gamma=torch.ones(cfg["d_model"], dtype=torch.float32, device=d0),
               ln_beta=torch.zeros(cfg["d_model"], dtype=torch.float32, device=d0), b_up=None, b_down=None)

    def block(ws):
        _lib.block_forward(cfg, blk, dev.X, dev.valid, dev.W_router, dev.prototypes, dev.W_up, dev.W_down,
                           dev.Y, ws)
        return {"Y": dev.Y}
    run_fenced(block, _lib.block_forward_workspace_size(cfg, blk), d0)

    dY = upstream_grad(g)
    from paper_2608_10392_amd.layer import to_device
    dYd = to_device(dY, cfg["dtype"], d0)
    H = cfg["n_blocks"] * cfg["block_width"]
    f = dict(dtype=torch.float32, device=d0)
    gr = dict(dX=torch.empty((N, cfg["d_model"]), **f), dW_up=torch.empty((K + 1, H, cfg["d_model"]), **f),
              dW_down=torch.empty((K + 1, cfg["d_model"], H), **f),
              dW_router=torch.empty((K + 1, cfg["d_model"]), **f))

    def bwd(ws):
        _lib.layer_backward(cfg, dev.X, dev.valid, dev.W_router, dev.prototypes, dev.W_up, dev.W_down, dYd,
                            gr["dX"], gr["dW_up"], gr["dW_down"], gr["dW_router"], ws)
        return gr
    run_fenced(bwd, _lib.layer_backward_workspace_size(cfg), d0)

    loss = torch.zeros(1, **f)

    def div(ws):
        dW = torch.zeros((K + 1, cfg["d_model"]), **f)
        _lib.diversity_loss(cfg, dev.W_router, 0.5, loss, dW, ws)
        return {"loss": loss, "dW": dW}
    run_fenced(div, _lib.diversity_loss_workspace_size(cfg), d0)
    del dev
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
