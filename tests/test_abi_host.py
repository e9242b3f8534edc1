"""Host-side checks of the C ABI (no GPU needed): the library loads and
exports every function include/unif_moe.h declares, the ctypes structures
match the C layout, and invalid arguments are rejected before any HIP call.
"""
import ctypes
import math
import os
import re
import subprocess

import pytest

from paper_2608_10392_amd import _lib
from synth import config_names, get_config, layer_config

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "unif_moe.h")


@pytest.fixture(scope="module")
def L():
    return _lib.lib()


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:int32_t|const char\*)\s+(unif_moe_\w+)\s*\(", text, re.M)))


def test_every_declared_symbol_is_exported(L):
    names = declared_functions()
    assert len(names) == 17, names
    assert set(names) == set(_lib.EXPORTS)
    out = subprocess.run(["nm", "-D", "--defined-only", _lib.LIB_PATH], capture_output=True, text=True).stdout
    for n in names:
        assert re.search(rf"\bT {n}$", out, re.M), n
        assert getattr(L, n) is not None


def test_struct_layout_matches_header(tmp_path):
    src = tmp_path / "layout.c"
    src.write_text(
        '#include <stdio.h>\n#include <stddef.h>\n#include "unif_moe.h"\n'
        "#define F(T, m) printf(#T \".\" #m \" %zu\\n\", offsetof(T, m))\n"
        "int main(void) {\n"
        ' printf("config %zu\\nrouting %zu\\nstats %zu\\nblock %zu\\nwork %zu\\n", sizeof(unif_moe_config),'
        " sizeof(unif_moe_routing), sizeof(unif_moe_stats_t), sizeof(unif_moe_block), sizeof(unif_moe_work_t));\n"
        " F(unif_moe_config, tau); F(unif_moe_config, select_mode); F(unif_moe_config, max_pairs);"
        " F(unif_moe_routing, weights); F(unif_moe_stats_t, expert_tokens);"
        " F(unif_moe_stats_t, activated_blocks); F(unif_moe_stats_t, routing_flops);\n"
        " F(unif_moe_block, ln_eps); F(unif_moe_block, ln_gamma); F(unif_moe_block, b_down);\n"
        " F(unif_moe_work_t, down_mfma_flops); F(unif_moe_work_t, down_queued);\n"
        " return 0; }\n")
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-I", os.path.dirname(HEADER), str(src), "-o", str(exe)], check=True)
    got = dict(l.rsplit(" ", 1) for l in subprocess.run([str(exe)], capture_output=True, text=True).stdout.splitlines())
    assert int(got["config"]) == ctypes.sizeof(_lib.Config)
    assert int(got["routing"]) == ctypes.sizeof(_lib.Routing)
    assert int(got["stats"]) == ctypes.sizeof(_lib.Stats)
    assert int(got["unif_moe_config.tau"]) == _lib.Config.tau.offset
    assert int(got["unif_moe_config.select_mode"]) == _lib.Config.select_mode.offset
    assert int(got["unif_moe_config.max_pairs"]) == _lib.Config.max_pairs.offset
    assert int(got["unif_moe_routing.weights"]) == _lib.Routing.weights.offset
    assert int(got["unif_moe_stats_t.expert_tokens"]) == _lib.Stats.expert_tokens.offset
    assert int(got["unif_moe_stats_t.activated_blocks"]) == _lib.Stats.activated_blocks.offset
    assert int(got["unif_moe_stats_t.routing_flops"]) == _lib.Stats.routing_flops.offset
    assert int(got["block"]) == ctypes.sizeof(_lib.Block)
    assert int(got["unif_moe_block.ln_eps"]) == _lib.Block.ln_eps.offset
    assert int(got["unif_moe_block.ln_gamma"]) == _lib.Block.ln_gamma.offset
    assert int(got["unif_moe_block.b_down"]) == _lib.Block.b_down.offset
    assert int(got["work"]) == ctypes.sizeof(_lib.Work)
    assert int(got["unif_moe_work_t.down_mfma_flops"]) == _lib.Work.down_mfma_flops.offset
    assert int(got["unif_moe_work_t.down_queued"]) == _lib.Work.down_queued.offset


def test_status_strings(L):
    assert _lib.status_string(0) == "ok"
    assert _lib.status_string(-2) == "workspace too small"
    assert _lib.status_string(_lib.ECAPACITY) == "routing needs more pairs than the capacity"
    assert _lib.status_string(12345) == "unknown status"


def base_cfg(**kw):
    c = layer_config(get_config("vit_b16"))
    c.update(kw)
    return c


@pytest.mark.parametrize("bad", [
    dict(n_tokens=-1), dict(d_model=0), dict(n_experts=0), dict(n_blocks=0), dict(block_width=0),
    dict(mass_threshold=0.0), dict(mass_threshold=1.5), dict(mass_threshold=math.nan),
    dict(max_shared=-1), dict(max_shared=17), dict(n_blocks=1, max_shared=1),
    dict(alpha_mode="fixed", alpha_fixed=1.5), dict(mass_mode="topk", fixed_k=0),
    dict(mass_mode="topk", fixed_k=17), dict(tau=0.5), dict(tau=-0.1), dict(max_pairs=-1),
])
def test_invalid_config_rejected(bad):
    with pytest.raises(_lib.UnifMoeError) as e:
        _lib.layer_forward_workspace_size(base_cfg(**bad))
    assert e.value.status == _lib.EINVAL


@pytest.mark.parametrize("bad", [
    dict(n_blocks=65, max_shared=65), dict(n_experts=65), dict(d_model=200),
    dict(block_width=96), dict(block_width=320), dict(n_tokens=2 ** 30),
])
def test_unsupported_shapes(bad):
    with pytest.raises(_lib.UnifMoeError) as e:
        _lib.layer_forward_workspace_size(base_cfg(**bad))
    assert e.value.status == _lib.EUNSUPPORTED


def test_fixed_alpha_allows_one_block():
    assert _lib.route_workspace_size(base_cfg(n_blocks=1, max_shared=1, alpha_mode="fixed",
                                              block_width=3072)) > 0


@pytest.mark.parametrize("name", config_names())
def test_workspace_sizes_cover_worst_case(name):
    c = layer_config(get_config(name))
    N, d, K, H = c["n_tokens"], c["d_model"], c["n_experts"], c["n_blocks"] * c["block_width"]
    es = 2 if c["dtype"] == "bf16" else 4
    ws = _lib.layer_forward_workspace_size(c)
    pairs = N * (K + 1)
    assert ws >= pairs * d * es                      # per-expert outputs
    if c["dtype"] == "bf16":
        assert ws >= pairs * (H * 2 + d * 2)         # activations + outputs
    assert _lib.stats_workspace_size(c) >= 199 * 8


def test_calls_fail_before_touching_the_device(L):
    """Each rejected call returns its status without any HIP call, so these
    run on a host with no GPU."""
    c = _lib.make_config(base_cfg(n_tokens=4))
    r = _lib.Routing(*([1] * 6))
    # NULL token matrix
    assert L.unif_moe_route(ctypes.byref(c), None, None, 1, 1, ctypes.byref(r), 1, 1 << 30, None) == _lib.EINVAL
    # incomplete record
    r0 = _lib.Routing(1, 1, 1, None, 1, 1)
    assert L.unif_moe_route(ctypes.byref(c), 1, None, 1, 1, ctypes.byref(r0), 1, 1 << 30, None) == _lib.EINVAL
    # workspace too small / missing
    assert L.unif_moe_route(ctypes.byref(c), 1, None, 1, 1, ctypes.byref(r), 1, 16, None) == _lib.EWORKSPACE
    assert L.unif_moe_layer_forward(ctypes.byref(c), 1, None, 1, 1, 1, 1, 1, None, None, 0, None) == _lib.EWORKSPACE
    assert L.unif_moe_layer_forward(ctypes.byref(c), 1, None, 1, 1, None, 1, 1, None, 1, 1 << 40, None) == _lib.EINVAL
    assert L.unif_moe_layer_forward(ctypes.byref(c), 1, None, 1, 1, 1, 1, 1, ctypes.byref(r0), 1, 1 << 40, None) == _lib.EINVAL
    s = _lib.Stats()
    assert L.unif_moe_stats(ctypes.byref(c), ctypes.byref(r), None, None, 1, 4096, None) == _lib.EINVAL
    assert L.unif_moe_stats(ctypes.byref(c), ctypes.byref(r), None, ctypes.byref(s), None, 0, None) == _lib.EWORKSPACE
    assert L.unif_moe_layer_forward(None, 1, None, 1, 1, 1, 1, 1, None, 1, 1, None) == _lib.EINVAL
    n = ctypes.c_size_t(0)
    assert L.unif_moe_layer_forward_workspace_size(ctypes.byref(c), None) == _lib.EINVAL
    assert L.unif_moe_layer_forward_workspace_size(ctypes.byref(c), ctypes.byref(n)) == 0 and n.value > 0


def test_empty_batch_is_a_no_op(L):
    """N = 0 with a large enough workspace returns OK without launching."""
    c = _lib.make_config(base_cfg(n_tokens=0))
    n = ctypes.c_size_t(0)
    assert L.unif_moe_layer_forward_workspace_size(ctypes.byref(c), ctypes.byref(n)) == 0
    assert L.unif_moe_layer_forward(ctypes.byref(c), None, None, None, None, None, None, None,
                                    None, 1, n.value, None) == 0


def _blk(**kw):
    b = dict(norm="pre", residual=True, ln_eps=1e-6, ln_gamma=1, ln_beta=1, b_up=None, b_down=None)
    b.update(kw)
    return b


def test_block_workspace_adds_the_normalised_input():
    c = base_cfg(n_tokens=1000)
    layer = _lib.layer_forward_workspace_size(c)
    assert _lib.block_forward_workspace_size(c, _blk(norm="none")) == layer
    assert _lib.block_forward_workspace_size(c, _blk(norm="post")) == layer
    pre = _lib.block_forward_workspace_size(c, _blk(norm="pre"))
    assert layer + 1000 * 768 * 2 <= pre <= layer + 1000 * 768 * 2 + 256


@pytest.mark.parametrize("bad, status", [
    (dict(norm="pre", ln_eps=0.0), _lib.EINVAL), (dict(norm="post", ln_eps=-1.0), _lib.EINVAL),
    (dict(norm="pre", ln_eps=math.inf), _lib.EINVAL), (dict(norm="post", ln_eps=math.nan), _lib.EINVAL),
])
def test_block_invalid_rejected(bad, status):
    with pytest.raises(_lib.UnifMoeError) as e:
        _lib.block_forward_workspace_size(base_cfg(), _blk(**bad))
    assert e.value.status == status


def test_block_calls_fail_before_touching_the_device(L):
    c = _lib.make_config(base_cfg(n_tokens=4))
    n = ctypes.c_size_t(0)
    good = _lib.make_block(_blk())
    assert L.unif_moe_block_forward_workspace_size(ctypes.byref(c), None, ctypes.byref(n)) == _lib.EINVAL
    assert L.unif_moe_block_forward_workspace_size(ctypes.byref(c), ctypes.byref(good), ctypes.byref(n)) == 0
    big = 1 << 40
    args = (1, None, 1, 1, 1, 1, 1, None, 1, big, None)
    assert L.unif_moe_block_forward(ctypes.byref(c), None, *args) == _lib.EINVAL
    bad_norm = _lib.Block(norm=7, residual=1, ln_eps=1e-6, ln_gamma=1, ln_beta=1)
    assert L.unif_moe_block_forward(ctypes.byref(c), ctypes.byref(bad_norm), *args) == _lib.EINVAL
    no_gamma = _lib.make_block(_blk(ln_gamma=None))
    assert L.unif_moe_block_forward(ctypes.byref(c), ctypes.byref(no_gamma), *args) == _lib.EINVAL
    odd_bias = _lib.make_block(_blk(b_up=4))          # bf16 layers read b1 and b2 in 16-byte pieces
    assert L.unif_moe_block_forward(ctypes.byref(c), ctypes.byref(odd_bias), *args) == _lib.EINVAL
    odd_bias = _lib.make_block(_blk(b_down=20))
    assert L.unif_moe_block_forward(ctypes.byref(c), ctypes.byref(odd_bias), *args) == _lib.EINVAL
    no_ln = _lib.make_block(_blk(norm="none", ln_gamma=None, ln_beta=None, ln_eps=0.0))
    assert L.unif_moe_block_forward(ctypes.byref(c), ctypes.byref(no_ln), 1, None, 1, 1, 1, 1, 1, None,
                                    None, 0, None) == _lib.EWORKSPACE
    post_wide = _lib.make_config(base_cfg(n_tokens=4, d_model=40960 + 128))
    post = _lib.make_block(_blk(norm="post"))
    assert L.unif_moe_block_forward_workspace_size(ctypes.byref(post_wide), ctypes.byref(post),
                                                   ctypes.byref(n)) == _lib.EUNSUPPORTED


def test_backward_workspace_and_validation(L):
    c = base_cfg(n_tokens=1000)
    N, d, K, H = 1000, 768, 16, 3072
    B = 16
    ws = _lib.layer_backward_workspace_size(c)
    # bf16: a second H buffer (bf16), the transposed W_down, the per-block partial sums
    assert ws >= (_lib.layer_forward_workspace_size(c) + 2 * (N * (K + 1) + 1) * H + 2 * (K + 1) * d * H
                  + 8 * B * N * (K + 1))
    # fp32: the per-pair fp32 intermediates
    cf = base_cfg(n_tokens=1000, dtype="f32")
    assert (_lib.layer_backward_workspace_size(cf)
            >= _lib.layer_forward_workspace_size(cf) + 4 * 2 * H * N * (K + 1))
    cc = _lib.make_config(c)
    big = 1 << 45
    # NULL dY, NULL gradient outputs, small workspace: rejected before any HIP call
    assert L.unif_moe_layer_backward(ctypes.byref(cc), 1, None, 1, 1, 1, 1, None, 1, 1, 1, 1, 1, big, None) == _lib.EINVAL
    assert L.unif_moe_layer_backward(ctypes.byref(cc), 1, None, 1, 1, 1, 1, 1, 1, None, 1, 1, 1, big, None) == _lib.EINVAL
    assert L.unif_moe_layer_backward(ctypes.byref(cc), 1, None, 1, 1, 1, 1, 1, 1, 1, 1, 1, 1, 16, None) == _lib.EWORKSPACE
    # fp32 layers: pair tiles of an expert segment index grid dimension y
    # (at most 65535 tiles of 128); bf16 layers have no such limit
    assert _lib.layer_backward_workspace_size(base_cfg(n_tokens=128 * 65535, dtype="f32")) > 0
    with pytest.raises(_lib.UnifMoeError) as e:
        _lib.layer_backward_workspace_size(base_cfg(n_tokens=128 * 65535 + 1, dtype="f32"))
    assert e.value.status == _lib.EUNSUPPORTED
    assert _lib.layer_backward_workspace_size(base_cfg(n_tokens=128 * 65535 + 1)) > 0


def test_static_forward_rejects_layers_beyond_its_scratch(L):
    """The forward without a workspace rejects, on the host before any HIP
    call, a layer that needs more than the static scratch."""
    c = _lib.make_config(layer_config(get_config("vit_b16")))
    assert _lib.layer_forward_workspace_size(c) > _lib.STATIC_WORKSPACE_BYTES
    assert L.unif_moe_layer_forward_static(ctypes.byref(c), 1, None, 1, 1, 1, 1, 1, None, None) == _lib.EWORKSPACE
    assert L.unif_moe_layer_forward_static(None, 1, None, 1, 1, 1, 1, 1, None, None) == _lib.EINVAL


def test_diversity_loss_rejects_bad_arguments(L):
    """unif_moe_diversity_loss validates before any device call: the
    pointers below are never dereferenced."""
    cfg = layer_config(get_config("vit_b16"))
    c = _lib.make_config(cfg)
    n = ctypes.c_size_t(0)
    assert L.unif_moe_diversity_loss_workspace_size(ctypes.byref(c), ctypes.byref(n)) == 0
    K1 = cfg["n_experts"] + 1
    assert n.value >= 8 * (K1 * K1 + 1)
    assert L.unif_moe_diversity_loss_workspace_size(ctypes.byref(c), None) == _lib.EINVAL
    p = ctypes.c_void_p(4096)
    args = dict(W=p, lam=1.0, loss=p, dW=p, ws=p, nbytes=n.value)

    def call(**over):
        a = dict(args, **over)
        return L.unif_moe_diversity_loss(ctypes.byref(c), a["W"], a["lam"], a["loss"], a["dW"], a["ws"],
                                          a["nbytes"], None)
    assert call(W=None) == _lib.EINVAL
    assert call(loss=None) == _lib.EINVAL
    assert call(dW=None) == _lib.EINVAL
    assert call(lam=float("nan")) == _lib.EINVAL
    assert call(lam=float("inf")) == _lib.EINVAL
    assert call(ws=None) == _lib.EWORKSPACE
    assert call(nbytes=n.value - 1) == _lib.EWORKSPACE
    bad = _lib.make_config(dict(cfg, n_experts=0))
    assert L.unif_moe_diversity_loss(ctypes.byref(bad), p, 1.0, p, p, p, n.value, None) == _lib.EINVAL


def test_backward_needs_whole_column_groups():
    """The backward's per-token and router kernels take 8 columns at a time:
    an fp32 layer with d % 8 != 0 is rejected by the size query."""
    ok = layer_config(get_config("tiny_f32", d_model=64))
    assert _lib.layer_backward_workspace_size(ok) > 0
    with pytest.raises(_lib.UnifMoeError) as e:
        _lib.layer_backward_workspace_size(dict(ok, d_model=60))
    assert e.value.status == _lib.EUNSUPPORTED
    assert _lib.layer_forward_workspace_size(dict(ok, d_model=60)) > 0


@pytest.mark.parametrize("name", ["vit_b16", "zipf_stress", "tiny_f32"])
def test_capacity_sizes_the_forward_workspace(name):
    """max_pairs sizes the pair-indexed buffers: the workspace shrinks with
    the capacity (by the activations and per-expert rows of the pairs left
    out), equals the worst case at or above N (K+1), and the backward's
    workspace ignores it."""
    c = layer_config(get_config(name))
    N, d, K, H = c["n_tokens"], c["d_model"], c["n_experts"], c["n_blocks"] * c["block_width"]
    worst = N * (K + 1)
    full = _lib.layer_forward_workspace_size(c)
    assert _lib.layer_forward_workspace_size(dict(c, max_pairs=worst)) == full
    assert _lib.layer_forward_workspace_size(dict(c, max_pairs=worst + 12345)) == full
    per_pair = d * 4 + (H * 2 if c["dtype"] == "bf16" else 0)   # per-expert row (+ fp16 activations)
    sizes = [_lib.layer_forward_workspace_size(dict(c, max_pairs=p)) for p in (worst // 2, worst // 4, worst // 8)]
    assert full > sizes[0] > sizes[1] > sizes[2]
    assert full - sizes[0] >= (worst - worst // 2) * per_pair
    if d % 8 == 0:   # a shape the backward takes
        assert _lib.layer_backward_workspace_size(dict(c, max_pairs=1000)) == _lib.layer_backward_workspace_size(c)
