"""Seeded generator for the synthetic layer workloads.

Every tensor comes from its own stream,
``numpy.random.Generator(PCG64(SeedSequence([seed, tag])))``, so the same
bytes are produced no matter which subset of tensors is requested, and the
first n token rows of a workload do not depend on the total token count.

Stream tags: 0 token draws, 1 base up-projection, 2 base down-projection,
3 router, 4 block prototypes, 5 padding lengths, 6 skewed-router directions,
7 bimodal token signs, 10 + e expert e's perturbation (up, then down);
for the transformer block around the layer: 200 LayerNorm gain, 201 LayerNorm
shift, 202 up-projection biases, 203 down-projection biases, 204 residual-
stream scales and offsets; 205 the upstream gradient dY of a training step.

Values are drawn in float64. Router and prototypes are cast to float32;
tokens and expert weights to float32 (fp32 workloads) or to bfloat16 with
round-to-nearest-even through float32 (bf16 workloads). bfloat16 arrays are
returned as their uint16 bit patterns.

Weight layout (one row-major array per tensor, expert 0 is the shared expert):
  W_up   [K+1, H, d]: row h of expert e is the key K_e[:, h];
  W_down [K+1, d, H]: V_e stored column-major, i.e. row j of expert e holds
                      V_e[:, j]; this is the [out, in] weight of the FFN's
                      second linear layer.
  W_router [K+1, d]: row 0 is W_shr, row j is W_j (the transpose of the
                     augmented router W_g* of Eq. augmented-router).
  prototypes [B, d]: row c is the block prototype mu_c (Eq. block-prototype).
"""
import json
import math
import os

import numpy as np

from .configs import get_config

_CAL_PATH = os.path.join(os.path.dirname(__file__), "calibration.json")
_CHUNK = 16384


def _rng(seed, tag):
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, tag])))


def f32_to_bf16_bits(a):
    """float32 -> bfloat16 bit patterns, round to nearest even (finite input)."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    bits = a.view(np.uint32)
    bias = ((bits >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((bits + bias) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(u):
    """bfloat16 bit patterns -> float32 (exact)."""
    u = np.ascontiguousarray(u, dtype=np.uint16)
    return (u.astype(np.uint32) << 16).view(np.float32)


def _cast(a64, dtype):
    a32 = a64.astype(np.float32)
    return f32_to_bf16_bits(a32) if dtype == "bf16" else a32


def load_calibration():
    if not os.path.exists(_CAL_PATH):
        return {}
    with open(_CAL_PATH) as f:
        return json.load(f)


def _layernorm_rows(x, eps=1e-5):
    mean = x.mean(axis=1, keepdims=True)
    var = ((x - mean) ** 2).mean(axis=1, keepdims=True)
    return (x - mean) / np.sqrt(var + eps)


def _skew_directions(cfg):
    """Unit vector v and K unit vectors orthogonal to it (tag 6)."""
    d, K = cfg["d_model"], cfg["n_experts"]
    r = _rng(cfg["seed"], 6)
    v = r.standard_normal(d)
    v /= np.linalg.norm(v)
    U = r.standard_normal((K, d))
    U -= np.outer(U @ v, v)
    U /= np.linalg.norm(U, axis=1, keepdims=True)
    return v, U


def _tokens(cfg, n):
    d = cfg["d_model"]
    r = _rng(cfg["seed"], 0)
    if cfg["tokens"] == "bimodal":
        v, _ = _skew_directions(cfg)
        sign = _rng(cfg["seed"], 7).integers(0, 2, size=n) * 2 - 1
    out = np.empty((n, d), dtype=np.uint16 if cfg["dtype"] == "bf16" else np.float32)
    for s in range(0, n, _CHUNK):
        e = min(n, s + _CHUNK)
        x = r.standard_normal((e - s, d))
        if cfg["tokens"] == "normal_ln":
            x = _layernorm_rows(x)
        elif cfg["tokens"] == "bimodal":
            x = x + 3.0 * sign[s:e, None] * v[None, :]
        out[s:e] = _cast(x, cfg["dtype"])
    return out


def _valid(cfg, n):
    p = cfg["padding"]
    if p is None:
        return None
    n_seq = -(-n // p["seq_len"])
    lengths = _rng(cfg["seed"], 5).integers(p["lo"], p["hi"] + 1, size=p["n_seq"])
    if n_seq > p["n_seq"]:
        raise ValueError("token count exceeds the padded batch")
    pos = np.arange(n) % p["seq_len"]
    seq = np.arange(n) // p["seq_len"]
    return (pos < lengths[seq]).astype(np.uint8)


def _router(cfg, router_scales=None):
    d, K = cfg["d_model"], cfg["n_experts"]
    cal = load_calibration().get(cfg["name"], {})
    if cfg["router"] == "zipf_bimodal":
        v, U = _skew_directions(cfg)
        c = router_scales if router_scales is not None else cal.get("residual_scales")
        if c is None:
            raise RuntimeError(f"{cfg['name']}: residual scales not calibrated")
        W = np.vstack([2.0 * v[None, :], np.asarray(c, dtype=np.float64)[:, None] * U])
        return W.astype(np.float32)
    W = _rng(cfg["seed"], 3).standard_normal((K + 1, d)) / math.sqrt(d)
    if cfg["router"] == "scaled_residual":
        s = router_scales if router_scales is not None else cal.get("residual_scale")
        if s is None:
            raise RuntimeError(f"{cfg['name']}: residual scale not calibrated")
        W[1:] *= float(s)
    return W.astype(np.float32)


def _prototypes(cfg):
    B, d = cfg["n_blocks"], cfg["d_model"]
    return (_rng(cfg["seed"], 4).standard_normal((B, d)) / math.sqrt(d)).astype(np.float32)


def _experts(cfg):
    K, d = cfg["n_experts"], cfg["d_model"]
    H = cfg["n_blocks"] * cfg["block_width"]
    sb, sp = cfg["sigma_base"], cfg["sigma_pert"]
    base_up = _rng(cfg["seed"], 1).standard_normal((H, d)) * sb
    base_down = _rng(cfg["seed"], 2).standard_normal((d, H)) * sb
    dt = np.uint16 if cfg["dtype"] == "bf16" else np.float32
    W_up = np.empty((K + 1, H, d), dtype=dt)
    W_down = np.empty((K + 1, d, H), dtype=dt)
    for e in range(K + 1):
        r = _rng(cfg["seed"], 10 + e)
        W_up[e] = _cast(base_up + sp * r.standard_normal((H, d)), cfg["dtype"])
        W_down[e] = _cast(base_down + sp * r.standard_normal((d, H)), cfg["dtype"])
    return W_up, W_down


def generate(name_or_cfg, n_tokens=None, weights=True, router_scales=None, **overrides):
    """Inputs of a workload.

    ``n_tokens`` keeps the first n token rows (same values as the full
    workload). ``weights=False`` skips the expert weights. ``overrides``
    change config fields (e.g. ``sigma_pert=0`` for identical experts, or a
    routing mode for the reduction tests).
    """
    cfg = get_config(name_or_cfg, **overrides) if isinstance(name_or_cfg, str) else dict(name_or_cfg)
    n = cfg["n_tokens"] if n_tokens is None else int(n_tokens)
    cfg["n_tokens"] = n
    out = dict(cfg=cfg, X=_tokens(cfg, n), valid=_valid(cfg, n),
               W_router=_router(cfg, router_scales), prototypes=_prototypes(cfg))
    if weights:
        out["W_up"], out["W_down"] = _experts(cfg)
    return out


def as_f32(a, dtype):
    """Array of a workload (bf16 bits or float32) as float32 values."""
    return bf16_bits_to_f32(a) if dtype == "bf16" else np.asarray(a, dtype=np.float32)


def block_inputs(gen, norm, residual=True, biases=True, eps=1e-5):
    """Parameters of the transformer block around a generated layer, and its
    residual-stream input.

    Returns (blk, X): ``blk`` holds norm ("none", "pre" or "post"), residual,
    ln_eps, ln_gamma [d] ~ 1 + 0.2 N(0, 1), ln_beta [d] ~ 0.1 N(0, 1),
    b_up [K+1, H] ~ 0.3 N(0, 1) and b_down [K+1, d] ~ 0.05 N(0, 1) (float32;
    None without biases). X is the block input in the layer's format: for
    "pre", the workload's tokens with a per-token scale U(0.5, 2.5) and a
    per-feature offset 0.3 N(0, 1) (the un-normalised residual stream that
    the pre-FFN LayerNorm sees); otherwise the workload's tokens as they are
    (in a post-LN block the FFN input is the previous LayerNorm's output).
    """
    cfg = gen["cfg"]
    d, K = cfg["d_model"], cfg["n_experts"]
    H = cfg["n_blocks"] * cfg["block_width"]
    n = gen["X"].shape[0]
    seed = cfg["seed"]
    blk = dict(norm=norm, residual=bool(residual), ln_eps=np.float32(eps),
               ln_gamma=(1.0 + 0.2 * _rng(seed, 200).standard_normal(d)).astype(np.float32),
               ln_beta=(0.1 * _rng(seed, 201).standard_normal(d)).astype(np.float32),
               b_up=None, b_down=None)
    if biases:
        blk["b_up"] = (0.3 * _rng(seed, 202).standard_normal((K + 1, H))).astype(np.float32)
        blk["b_down"] = (0.05 * _rng(seed, 203).standard_normal((K + 1, d))).astype(np.float32)
    if norm != "pre":
        return blk, gen["X"].copy()
    r = _rng(seed, 204)
    offset = 0.3 * r.standard_normal(d)
    scale = r.uniform(0.5, 2.5, size=n)
    x = as_f32(gen["X"], cfg["dtype"]).astype(np.float64) * scale[:, None] + offset[None, :]
    return blk, _cast(x, cfg["dtype"])


def upstream_grad(gen):
    """Seeded upstream gradient dY [N, d] ~ N(0, 1) of a generated layer, in
    the layer's format (tag 205)."""
    cfg = gen["cfg"]
    n, d = gen["X"].shape
    return _cast(_rng(cfg["seed"], 205).standard_normal((n, d)), cfg["dtype"])
