"""Parity protocol between the HIP library and the CPU oracle.

Routing: every valid token whose decision margin (oracle.margins) is at least
1e-4 must get exactly the oracle's discrete decisions (b, I_shr, k and the
set {q_1..q_k}); the order of q is compared wherever neighbouring affinities
differ by at least 1e-4. Tokens below the margin are counted; where their
decisions differ, each differing decision must lie within 1e-4 of its
boundary, and their outputs are checked against the oracle evaluated under
the GPU's decisions (oracle.forced_forward).

Outputs, over the checked tokens and all features, against y_ref, the
float64 oracle output:
  raw     max |y_gpu - y_ref| / RMS(y_ref) <= TOL (2e-2 bf16, 1e-4 fp32), the
          bound as stated;
  excess  max (|y_gpu - y_ref| - ulp_out(y_ref) / 2) / RMS(y_ref) <= KERNEL_TOL,
          the error the computation adds beyond rounding y_ref once to the
          output format (ulp_out: the format's spacing at y_ref), so that the
          kernels' own error cannot grow unseen below the raw bound.
Only where rounding y_ref once to nearest (RNE) already exceeds TOL (bf16
outputs of 8 x RMS and more) is the raw bound replaced by RNE + KERNEL_TOL,
and the message says so; every message carries the raw, RNE and excess
figures.
"""
import numpy as np

import oracle.unif_moe_oracle as O
from synth.generate import bf16_bits_to_f32

MARGIN = 1e-4
TOL = {"bf16": 2e-2, "f32": 1e-4}
KERNEL_TOL = {"bf16": 5e-3, "f32": 5e-5}


def _decision_parts(rec, t, B):
    m = int(rec["shared_mask"][t])
    k = int(rec["n_res"][t])
    return (int(rec["n_shared"][t]), m, k, frozenset(int(j) for j in rec["expert_ids"][t, :k]))


def check_routing(cfg, orec, grec, loose=None):
    """Compare records; returns a summary dict, raises AssertionError.

    ``loose`` marks tokens whose routing input itself may differ between the
    two sides (see block_loose_tokens): they are checked like near-ties,
    without the boundary condition."""
    K, B = cfg["n_experts"], cfg["n_blocks"]
    m, parts = O.margins(cfg, orec)
    v = orec["valid"]
    N = len(v)
    if loose is None:
        loose = np.zeros(N, bool)
    # padded tokens: exact record
    pad = ~v
    assert np.all(grec["n_res"][pad] == 0) and np.all(grec["n_shared"][pad] == 0)
    assert np.all(grec["shared_mask"][pad] == 0) and np.all(grec["alpha"][pad] == 0)
    assert np.all(grec["expert_ids"][pad] == -1) and np.all(grec["weights"][pad] == 0)

    sure = v & (m >= MARGIN) & ~loose
    idx = np.nonzero(sure)[0]
    bad = idx[grec["n_shared"][idx] != orec["n_shared"][idx]]
    assert bad.size == 0, f"b differs on {bad.size} tokens with margin >= {MARGIN}, e.g. {bad[:5]}"
    bad = idx[grec["shared_mask"][idx] != orec["shared_mask"][idx]]
    assert bad.size == 0, f"I_shr differs on {bad.size} tokens, e.g. {bad[:5]}"
    bad = idx[grec["n_res"][idx] != orec["n_res"][idx]]
    assert bad.size == 0, f"k differs on {bad.size} tokens, e.g. {bad[:5]}"
    # expert sets {q_1..q_k}
    kk = orec["n_res"]
    pos = np.arange(K)[None, :]
    sel_o = np.zeros((N, K + 1), bool)
    sel_g = np.zeros((N, K + 1), bool)
    rows = np.repeat(np.arange(N)[:, None], K, 1)
    live = (pos < kk[:, None]) & v[:, None]
    np.logical_or.at(sel_o, (rows[live], orec["expert_ids"][live]), True)
    live_g = (pos < grec["n_res"][:, None]) & v[:, None]
    np.logical_or.at(sel_g, (rows[live_g], np.clip(grec["expert_ids"][live_g], 0, K)), True)
    bad = idx[np.any(sel_o[idx] != sel_g[idx], axis=1)]
    assert bad.size == 0, f"expert set differs on {bad.size} tokens, e.g. {bad[:5]}"
    # order of q where neighbouring affinities are separated
    p = orec["weights"].astype(np.float64)
    gap = np.full((N, K + 1), np.inf)
    gap[:, 1:K] = p[:, :-1] - p[:, 1:]
    sep = (gap[:, :K] >= MARGIN) & (gap[:, 1:] >= MARGIN)
    chk = sure[:, None] & sep
    bad = np.nonzero(np.any(chk & (grec["expert_ids"] != orec["expert_ids"]), axis=1))[0]
    assert bad.size == 0, f"expert order differs on {bad.size} tokens, e.g. {bad[:5]}"
    # continuous values (diagnostics)
    vs = v & ~loose
    da = float(np.abs(grec["alpha"][vs].astype(np.float64) - orec["alpha"][vs]).max(initial=0.0))
    dp = float(np.abs(np.sort(grec["weights"][vs], axis=1).astype(np.float64)
                      - np.sort(orec["weights"][vs], axis=1)).max(initial=0.0))
    # Logits differ from the correctly rounded ones by the fp32 accumulation
    # order: about sqrt(d) ulp of the partial sums, <= 1e-5 for |z| <= 30 and
    # d <= 1024; alpha and p move by at most 1/4 of that (sigmoid and softmax
    # slopes are <= 1/4 per unit logit).
    assert da <= 1e-5, f"alpha differs by {da}"
    assert dp <= 1e-5, f"affinities differ by {dp}"

    near = np.nonzero(v & ((m < MARGIN) | loose))[0]
    differ = []
    for t in near:
        go, oo = _decision_parts(grec, t, B), _decision_parts(orec, t, B)
        if go == oo:
            continue
        differ.append(int(t))
        if loose[t]:
            continue
        if go[0] != oo[0]:
            assert parts["m_b"][t] < MARGIN, ("b differs away from its boundary", t)
        elif go[1] != oo[1]:
            assert parts["m_sel"][t] < MARGIN, ("I_shr differs away from its boundary", t)
        if go[2] != oo[2]:
            assert parts["m_k"][t] < MARGIN, ("k differs away from its boundary", t)
        elif go[3] != oo[3]:
            assert parts["m_set"][t] < MARGIN, ("expert set differs away from its boundary", t)
    return dict(n_valid=int(v.sum()), n_checked=int(sure.sum()), n_near=int(near.size),
                n_near_differ=len(differ), near_differ=differ, max_alpha_err=da, max_p_err=dp)


def sample_tokens(orec, cfg, n_sample, seed=1234, near_cap=256):
    """Seeded sample of valid tokens, plus near-tie tokens (capped) and
    tokens with the extreme b and k."""
    v = np.nonzero(orec["valid"])[0]
    rng = np.random.default_rng(seed)
    pick = set(rng.choice(v, size=min(n_sample, v.size), replace=False).tolist())
    m, _ = O.margins(cfg, orec)
    near = np.nonzero(orec["valid"] & (m < MARGIN))[0]
    if near.size > near_cap:
        near = rng.choice(near, size=near_cap, replace=False)
    pick.update(near.tolist())
    for key in ("n_shared", "n_res"):
        vals = orec[key][v]
        for target in (vals.min(), vals.max()):
            pick.update(v[vals == target][:4].tolist())
    return np.array(sorted(pick))


def half_ulp(y, dtype):
    """Half the spacing of the output format (bf16: 8 significant bits,
    fp32: 24) at |y|, for normal numbers."""
    bits = 8 if dtype == "bf16" else 24
    e = np.floor(np.log2(np.maximum(np.abs(y), 1e-300)))
    return np.where(y == 0, 0.0, 2.0 ** (e - bits))


def gpu_output_f64(Y, dtype):
    return (bf16_bits_to_f32(Y) if dtype == "bf16" else np.asarray(Y, np.float32)).astype(np.float64)


def rne_format(y, dtype):
    """y (float64) rounded once to the output format, to nearest even."""
    if dtype == "f32":
        return np.asarray(y, np.float64).astype(np.float32).astype(np.float64)
    return gpu_output_f64(O.to_format(y, "bf16"), "bf16")


def _output_error(cfg, Yg, ref):
    dt = cfg["dtype"]
    rms = float(np.sqrt(np.mean(ref ** 2)))
    scale = rms if rms > 0 else 1.0
    raw = float(np.abs(Yg - ref).max()) / scale
    rne = float(np.abs(rne_format(ref, dt) - ref).max()) / scale
    excess = float(np.maximum(np.abs(Yg - ref) - half_ulp(ref, dt), 0.0).max()) / scale
    bound = TOL[dt]
    note = ""
    if rne > TOL[dt]:
        bound = rne + KERNEL_TOL[dt]
        note = " (format-limited case: rounding y_ref once already exceeds the bound)"
    msg = (f"output error: raw {raw:.3e} x RMS (bound {bound:.1e}{note}), rounding y_ref once "
           f"{rne:.3e}, beyond the half ulp {excess:.3e} (bound {KERNEL_TOL[dt]:.0e}); RMS {rms:.3e}")
    print(msg)
    assert raw <= bound, msg
    assert excess <= KERNEL_TOL[dt], msg
    return raw, excess


# ------------------------------------------------ the block around it ---
# The two sides compute LN(x) in fp64 (sums of d terms in different orders:
# about 1e-14 apart at these sizes) and round it to the layer's format; an
# element within this distance of a rounding midpoint may round differently,
# and its token's routing input with it.
LN_SLACK = 1e-11


def block_loose_tokens(cfg, blk, X):
    """Tokens whose pre-LN FFN input has an element within LN_SLACK (x (1 +
    |v|)) of a rounding midpoint of the layer's format."""
    N = X.shape[0]
    if blk["norm"] != "pre":
        return np.zeros(N, bool)
    x = O._as_f32(X, cfg["dtype"]).astype(np.float64)
    v = O.layer_norm(x, blk["ln_gamma"], blk["ln_beta"], blk["ln_eps"])
    return np.any(O.rounding_slack(v, cfg["dtype"]) < LN_SLACK * (1.0 + np.abs(v)), axis=1)


def check_block_outputs(cfg, blk, inputs, Xin, orec, grec, Y_gpu, tokens, weights=None):
    """As check_outputs, for the block forward: the oracle's FFN part under
    the agreed (or the GPU's) decisions on the FFN input Xin, then the
    residual add and post-LN of oracle.block_finish."""
    if weights is None:
        weights = O.block_weights(cfg, blk, inputs["W_up"], inputs["W_down"])
    B = cfg["n_blocks"]
    Yg = gpu_output_f64(Y_gpu[tokens], cfg["dtype"])
    agree = [t for t in tokens if _decision_parts(grec, t, B) == _decision_parts(orec, t, B)]
    Fa, _ = O.forward(cfg, Xin, inputs["valid"], inputs["W_router"], inputs["prototypes"],
                      None, None, tokens=agree, rec=orec, weights=weights)
    F = np.zeros_like(Yg)
    for i, t in enumerate(tokens):
        if not orec["valid"][t]:
            continue
        if _decision_parts(grec, t, B) == _decision_parts(orec, t, B):
            F[i] = Fa[t]
        else:
            b, mask, k, experts = _decision_parts(grec, t, B)
            F[i] = O.forced_forward(cfg, Xin, orec, t, [c for c in range(B) if mask >> c & 1],
                                    sorted(experts), weights)
    ref = O.block_finish(cfg, blk, inputs["X"][tokens], F)
    return _output_error(cfg, Yg, ref)


def check_outputs(cfg, inputs, orec, grec, Y_gpu, tokens, weights=None):
    """Compare GPU rows against the oracle on ``tokens``; returns the
    relative error (max abs / RMS)."""
    if weights is None:
        weights = O.ExpertWeights(cfg, inputs["W_up"], inputs["W_down"])
    B = cfg["n_blocks"]
    Yg = gpu_output_f64(Y_gpu[tokens], cfg["dtype"])
    ref = np.zeros_like(Yg)
    agree = [t for t in tokens if _decision_parts(grec, t, B) == _decision_parts(orec, t, B)]
    Ya, _ = O.forward(cfg, inputs["X"], inputs["valid"], inputs["W_router"], inputs["prototypes"],
                      None, None, tokens=agree, rec=orec, weights=weights)
    for i, t in enumerate(tokens):
        if not orec["valid"][t]:
            continue
        if _decision_parts(grec, t, B) == _decision_parts(orec, t, B):
            ref[i] = Ya[t]
        else:
            b, mask, k, experts = _decision_parts(grec, t, B)
            ref[i] = O.forced_forward(cfg, inputs["X"], orec, t,
                                      [c for c in range(B) if mask >> c & 1], sorted(experts), weights)
    return _output_error(cfg, Yg, ref)
