"""Parity of the block forward (unif_moe_block_forward: pre-/post-LN, FFN
biases, residual add) with the CPU oracle's block_forward (MI355X only).

Routing is compared on the FFN input as in tests/parity.py; tokens whose
pre-LN input has an element that may round either way (within 1e-11 of a
rounding midpoint; the two sides compute LN in fp64) are checked like
near-ties. Outputs: the layer's bound, 2e-2 x RMS (bf16) or 1e-4 x RMS (fp32)
beyond the output format's half ulp. Cases without the residual add test the
FFN part on its own; the residual stream would otherwise dominate the RMS.
"""
import numpy as np
import pytest

import oracle.unif_moe_oracle as O
from synth import block_inputs, generate, get_config, layer_config
from tests import parity

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def run_block(g, blk, X, label, n_sample=None):
    cfg = g["cfg"]
    print(f"\n[gpu] block {label}: norm={blk['norm']} residual={blk['residual']} "
          f"biases={blk['b_up'] is not None} N={cfg['n_tokens']} d={cfg['d_model']} "
          f"K={cfg['n_experts']} B={cfg['n_blocks']} M={cfg['block_width']} {cfg['dtype']}",
          flush=True)
    from paper_2608_10392_amd.layer import DeviceLayer
    dev = DeviceLayer(layer_config(cfg), X, g["valid"], g["W_router"], g["prototypes"],
                      g["W_up"], g["W_down"])
    dev.block_forward(blk)
    torch.cuda.synchronize()
    grec, Y = dev.routing_numpy(), dev.output_numpy()
    Xin = O.block_input(cfg, blk, X)
    orec = O.route(cfg, Xin, g["valid"], g["W_router"], g["prototypes"])
    loose = parity.block_loose_tokens(cfg, blk, X)
    summary = parity.check_routing(cfg, orec, grec, loose=loose)
    tokens = (np.arange(cfg["n_tokens"]) if n_sample is None
              else parity.sample_tokens(orec, cfg, n_sample))
    inputs = dict(g, X=X)
    raw, excess = parity.check_block_outputs(cfg, blk, inputs, Xin, orec, grec, Y, tokens)
    print(f"[gpu] block {label}: checked {summary['n_checked']}/{summary['n_valid']} decisions, "
          f"loose {int(loose.sum())}, near-ties {summary['n_near']} (differing "
          f"{summary['n_near_differ']}), output err raw {raw:.2e} x RMS, "
          f"beyond half-ulp {excess:.2e} over {len(tokens)} tokens", flush=True)
    del dev
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return grec, Y


SMALL = dict(n_tokens=1000, d_model=384, n_experts=8, n_blocks=8, block_width=192, max_shared=8)


@pytest.mark.parametrize("norm", ["pre", "post", "none"])
@pytest.mark.parametrize("residual", [False, True])
def test_block_bf16(norm, residual):
    g = generate(get_config("vit_s16", **SMALL))
    blk, X = block_inputs(g, norm, residual=residual, eps=1e-6)
    run_block(g, blk, X, "bf16 small")


@pytest.mark.parametrize("M", [64, 128, 256])
def test_block_bf16_block_widths(M):
    """The up-projection's bias epilogue in each block-width kernel."""
    g = generate(get_config("vit_s16", n_tokens=700, d_model=256, n_experts=5, n_blocks=4,
                            block_width=M, max_shared=4))
    blk, X = block_inputs(g, "pre", residual=False)
    run_block(g, blk, X, f"bf16 M={M}")


def test_block_bias_only():
    """Zero expert weights: the output is the bias terms alone,
    alpha (b/B) b2_shr + sum_i p_i ((B-b)/B) b2_{q_i}."""
    g = generate(get_config("vit_s16", n_tokens=513, d_model=256, n_experts=6, n_blocks=8,
                            block_width=64, max_shared=8))
    g["W_up"][:] = 0
    g["W_down"][:] = 0
    blk, X = block_inputs(g, "none", residual=False)
    run_block(g, blk, X, "zero weights")


def test_block_post_ln_padded_wide():
    """Post-LN (BERT-like) with padded tokens, d = 1024."""
    g = generate(get_config("bert_base_padded", n_tokens=1024, d_model=1024, n_experts=8,
                            n_blocks=16, block_width=128))
    blk, X = block_inputs(g, "post", residual=True, eps=1e-12)
    run_block(g, blk, X, "post-LN padded")


@pytest.mark.parametrize("norm", ["pre", "post"])
def test_block_fp32(norm):
    g = generate(get_config("tiny_f32", n_tokens=301, d_model=96, n_experts=5, n_blocks=3,
                            block_width=40, max_shared=3))
    g["valid"] = (np.arange(301) % 6 != 1).astype(np.uint8)
    blk, X = block_inputs(g, norm, residual=(norm == "post"))
    run_block(g, blk, X, "fp32")


@pytest.mark.parametrize("name, norm, eps", [("paper_vision", "pre", 1e-6),
                                              ("paper_language", "post", 1e-12)])
def test_block_paper_configs(name, norm, eps):
    """The paper's operating points at full size in their backbones' block
    form (DeiT-S: pre-LN; BERT-large: post-LN), sampled outputs."""
    g = generate(name)
    blk, X = block_inputs(g, norm, residual=True, eps=eps)
    run_block(g, blk, X, name, n_sample=384)


def test_block_matches_layer_without_block_terms():
    """No LN, no biases, no residual: the block forward is the layer forward,
    bit for bit in the routing record and in Y (the block's merge sums the
    same bf16 expert rows in fp32 in the same order and rounds once, like the
    layer's)."""
    g = generate(get_config("vit_s16", **SMALL))
    blk, X = block_inputs(g, "none", residual=False, biases=False)
    from paper_2608_10392_amd.layer import DeviceLayer
    dev = DeviceLayer(layer_config(g["cfg"]), X, g["valid"], g["W_router"], g["prototypes"],
                      g["W_up"], g["W_down"])
    dev.forward()
    torch.cuda.synchronize()
    y_layer, rec_layer = dev.output_numpy().copy(), dev.routing_numpy()
    dev.block_forward(blk)
    torch.cuda.synchronize()
    y_block, rec_block = dev.output_numpy(), dev.routing_numpy()
    for k in rec_layer:
        assert np.array_equal(rec_layer[k], rec_block[k]), k
    a = parity.gpu_output_f64(y_layer, "bf16")
    b = parity.gpu_output_f64(y_block, "bf16")
    # Both sum the same bf16 expert rows in fp32 in the same order.
    assert np.array_equal(a, b)


def test_block_all_padded():
    """Every token padded: the FFN term is zero, so the pre-LN block returns
    x exactly and the post-LN block LN(x) (checked against the oracle)."""
    g = generate(get_config("vit_s16", n_tokens=300, d_model=256, n_experts=4, n_blocks=4,
                            block_width=64, max_shared=4))
    g["valid"] = np.zeros(300, np.uint8)
    blk, X = block_inputs(g, "pre", residual=True)
    grec, Y = run_block(g, blk, X, "all padded, pre-LN")
    assert np.array_equal(Y, X)
    blk, X = block_inputs(g, "post", residual=True)
    run_block(g, blk, X, "all padded, post-LN")
