"""Parity of the backward pass (unif_moe_layer_backward) and of the Gram
diversity loss (unif_moe_diversity_loss) with the CPU oracle (MI355X only).

The gradients of sum(dY * Y) are compared tensor by tensor as max |g_gpu -
g_ref| / max |g_ref|:
  * fp32 layers: <= 1e-4 (fp32 arithmetic on inputs exact in fp32; the
    oracle in fp64);
  * bf16 layers: <= 1e-2. The matrix-core path rounds d loss / da and
    w GELU(a) to bf16 (relative step 2^-8, so at most 2^-9 = 1.95e-3 per
    value) before the products that give dx, dW_up and dW_down, and the
    pre-activation a to fp16; each gradient element is a sum of such terms,
    whose error is at most 2^-9 of the sum of their magnitudes. The bound
    allows that sum to reach five times the largest gradient element.
The decisions are held fixed, so tokens whose routing margin is below 1e-4
(where the two sides may take different decisions) are marked padded in the
input; padded tokens must get dX = 0.
"""
import numpy as np
import pytest

import oracle.unif_moe_oracle as O
from synth import generate, get_config, layer_config, upstream_grad
from tests import parity

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

TOL = {"f32": 1e-4, "bf16": 1e-2}


def run_backward(g, label):
    cfg = g["cfg"]
    N = cfg["n_tokens"]
    rec0 = O.route(cfg, g["X"], g["valid"], g["W_router"], g["prototypes"])
    m, _ = O.margins(cfg, rec0)
    valid = np.ones(N, np.uint8) if g["valid"] is None else g["valid"].copy()
    valid[m < parity.MARGIN] = 0
    dY = upstream_grad(g)
    print(f"\n[gpu] backward {label}: N={N} ({int(valid.sum())} valid) d={cfg['d_model']} "
          f"K={cfg['n_experts']} B={cfg['n_blocks']} M={cfg['block_width']} {cfg['dtype']}", flush=True)
    from paper_2608_10392_amd.layer import DeviceLayer
    dev = DeviceLayer(layer_config(cfg), g["X"], valid, g["W_router"], g["prototypes"],
                      g["W_up"], g["W_down"])
    got = {k: v.cpu().numpy().astype(np.float64) for k, v in dev.backward(dY).items()}
    dYf = O._as_f32(dY, cfg["dtype"]).astype(np.float64)
    ref = O.backward(cfg, g["X"], valid, g["W_router"], g["prototypes"], g["W_up"], g["W_down"], dYf)
    errs = {}
    for k in ("dX", "dW_up", "dW_down", "dW_router"):
        scale = float(np.abs(ref[k]).max())
        err = float(np.abs(got[k] - ref[k]).max()) / scale
        errs[k] = err
        assert err <= TOL[cfg["dtype"]], f"{k}: error {err:.2e} x max |ref| ({scale:.3e})"
    assert np.all(got["dX"][valid == 0] == 0)
    print(f"[gpu] backward {label}: " + ", ".join(f"{k} {v:.1e}" for k, v in errs.items())
          + " x max |ref|", flush=True)
    del dev
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


CASES = {
    "bf16_m64": ("vit_s16", dict(n_tokens=300, d_model=128, n_experts=4, n_blocks=4,
                                 block_width=64, max_shared=4)),
    "bf16_m192": ("vit_s16", dict(n_tokens=600, d_model=384, n_experts=8, n_blocks=8,
                                  block_width=192, max_shared=8)),
    "bf16_fixed_alpha_top2": ("vit_s16", dict(n_tokens=300, d_model=128, n_experts=5, n_blocks=4,
                                              block_width=64, max_shared=4, alpha_mode="fixed",
                                              alpha_fixed=0.4, mass_mode="topk", fixed_k=2)),
    "bf16_padded": ("bert_base_padded", dict(n_tokens=384, d_model=256, n_experts=6, n_blocks=8,
                                             block_width=64, max_shared=8)),
    "f32": ("tiny_f32", dict(n_tokens=200, d_model=64, n_experts=4, n_blocks=4, block_width=32,
                             max_shared=4)),
    # a block width that is not a multiple of the fp32 kernels' 16-channel
    # steps: a step then spans two blocks
    "f32_m24": ("tiny_f32", dict(n_tokens=200, d_model=64, n_experts=4, n_blocks=4, block_width=24,
                                 max_shared=4)),
    # edge shapes: one token; two blocks of the widest kernel; 64 experts x 64 blocks
    "n1": ("vit_s16", dict(n_tokens=1, d_model=128, n_experts=4, n_blocks=4, block_width=64,
                           max_shared=4)),
    "b2_m256": ("vit_s16", dict(n_tokens=260, d_model=256, n_experts=3, n_blocks=2,
                                block_width=256, max_shared=2)),
    "m128_d512": ("vit_s16", dict(n_tokens=450, d_model=512, n_experts=5, n_blocks=4,
                                  block_width=128, max_shared=4)),
    # d = 640: five 128-column n tiles of the weight gradients, the down
    # projection's 256 x 128 tiles
    "m192_d640": ("vit_s16", dict(n_tokens=500, d_model=640, n_experts=4, n_blocks=4,
                                  block_width=192, max_shared=4)),
    "k64_b64": ("vit_s16", dict(n_tokens=200, d_model=128, n_experts=64, n_blocks=64,
                                block_width=64, max_shared=64, mass_threshold=0.9)),
}


@pytest.mark.parametrize("name", list(CASES))
def test_backward(name):
    base, over = CASES[name]
    run_backward(generate(get_config(base, **over)), name)


@pytest.mark.parametrize("name", ["vit_b16", "bert_base_padded", "zipf_stress"])
def test_backward_full_size_properties(name):
    """At the full workload sizes, where the oracle's gradient sums are out of
    reach: every gradient is linear in dY, and scaling dY by 2 scales every
    intermediate the backward rounds (to bf16 or fp16, away from the
    formats' range limits) by exactly 2, so backward(2 dY) equals
    2 backward(dY) bit for bit, for all four gradients, since every sum runs
    in a fixed order. A repeated call gives the same bits. Padded tokens get
    dX = 0; all gradients are finite."""
    g = generate(name)
    cfg = g["cfg"]
    print(f"\n[gpu] backward properties {name}: N={cfg['n_tokens']}", flush=True)
    from paper_2608_10392_amd.layer import DeviceLayer
    dev = DeviceLayer(layer_config(cfg), g["X"], g["valid"], g["W_router"], g["prototypes"],
                      g["W_up"], g["W_down"])
    dY = upstream_grad(g)
    g1 = dev.backward(dY)
    dY2 = O._as_f32(dY, cfg["dtype"]) * np.float32(2.0)
    dY2 = (dY2.view(np.uint32) >> 16).astype(np.uint16) if cfg["dtype"] == "bf16" else dY2
    g2 = dev.backward(dY2)
    g3 = dev.backward(dY)
    for k in g1:
        a, b = g1[k], g2[k]
        assert bool(torch.isfinite(a).all()), k
        assert torch.equal(g3[k], a), f"{k}: a repeated backward differs"
        assert torch.equal(b, 2.0 * a), f"{k}: backward(2 dY) != 2 backward(dY)"
    if g["valid"] is not None:
        pad = torch.from_numpy(g["valid"] == 0).to(g1["dX"].device)
        assert bool((g1["dX"][pad] == 0).all())
    del dev, g1, g2, g3
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def test_backward_all_padded():
    """No valid token: no pairs, and every gradient is exactly zero."""
    g = generate(get_config("vit_s16", n_tokens=200, d_model=128, n_experts=4, n_blocks=4,
                            block_width=64, max_shared=4))
    from paper_2608_10392_amd.layer import DeviceLayer
    dev = DeviceLayer(layer_config(g["cfg"]), g["X"], np.zeros(200, np.uint8), g["W_router"],
                      g["prototypes"], g["W_up"], g["W_down"])
    grads = dev.backward(upstream_grad(g))
    for k, v in grads.items():
        assert bool((v == 0).all()), k


@pytest.mark.parametrize("shape", [(17, 768), (65, 128), (2, 40), (7, 384)])
def test_diversity_loss(shape):
    """L_div (Eq. diversity-loss) and lambda times its gradient added to
    dW_router, against oracle.diversity_loss (fp64): the loss to 1e-6
    relative, the update to 1e-6 of its largest element; a zero lambda
    leaves dW_router untouched, and a repeated call gives the same bits."""
    from paper_2608_10392_amd import _lib
    K1, d = shape
    cfg = layer_config(get_config("tiny_f32", n_experts=K1 - 1, d_model=d, fixed_k=1))
    rng = np.random.default_rng(K1 * 1000 + d)
    W = (rng.standard_normal((K1, d)) / np.sqrt(d)).astype(np.float32)
    print(f"\n[gpu] diversity loss K+1={K1} d={d}", flush=True)
    L_ref, g_ref = O.diversity_loss(W)
    dev = torch.device("cuda:0")
    Wd = torch.from_numpy(W).to(dev)
    loss = torch.zeros(1, dtype=torch.float32, device=dev)
    base = torch.from_numpy(rng.standard_normal((K1, d)).astype(np.float32)).to(dev)
    ws = _lib.alloc_workspace(_lib.diversity_loss_workspace_size(cfg), dev)
    lam = 0.25
    dW = base.clone()
    _lib.diversity_loss(cfg, Wd, lam, loss, dW, ws)
    torch.cuda.synchronize()
    assert abs(float(loss.item()) - L_ref) <= 1e-6 * L_ref
    upd = (dW.double() - base.double()).cpu().numpy()
    scale = float(np.abs(lam * g_ref).max())
    assert np.abs(upd - lam * g_ref).max() <= 1e-6 * scale + 2.0 ** -23 * float(base.abs().max())
    dW2 = base.clone()
    _lib.diversity_loss(cfg, Wd, lam, loss, dW2, ws)
    dW0 = base.clone()
    _lib.diversity_loss(cfg, Wd, 0.0, loss, dW0, ws)
    torch.cuda.synchronize()
    assert torch.equal(dW2, dW) and torch.equal(dW0, base)
