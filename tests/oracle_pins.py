"""Checks that pin the CPU oracle to things other than itself.

Each ``pin_*`` function takes the oracle module and raises AssertionError
when the oracle disagrees with:
  * a worked example derived by hand from the equations of Sec. III
    (tests/golden/hand_example.json);
  * closed forms (GELU through the standard normal CDF, tau values, the
    round-half-even rule of Eq. block-count);
  * brute-force enumeration on tiny layers (every subset of blocks and of
    experts, the output as an explicit sum over channels, all in float64);
  * reductions to textbook layers: top-k MoE (Eq. vanilla-moe-output), the
    dense FFN (Eq. ffn-kv) and the soft MoE over all experts;
  * the identical-expert decomposition E = sum of its blocks (Sec. III-A);
  * the mixture-mass bound (Eq. mixture-mass-bound).
The implementations here are written independently of the oracle (pure
Python loops and math.erf). tests/test_oracle_mutations.py re-runs these pins
on deliberately broken copies of the oracle to show that each mistake is
caught.
"""
import itertools
import json
import math
import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ------------------------------------------------------------ textbook ---
def phi(a):
    """Standard normal CDF."""
    return 0.5 * (1.0 + math.erf(a / math.sqrt(2.0)))


def gelu_tb(a):
    return a * phi(a)


_gelu_vec = np.vectorize(gelu_tb, otypes=[np.float64])


def tb_ffn(x, w_up, w_down):
    """Dense FFN of Eq. ffn-kv for rows x: GELU(x K) V, with K = w_up^T and
    V = w_down^T (float64)."""
    return _gelu_vec(x @ w_up.T) @ w_down.T


def tb_softmax(l):
    e = np.exp(l - l.max(axis=-1, keepdims=True))
    return e / e.sum(axis=-1, keepdims=True)


def layer_cfg(d, K, B, M, **kw):
    cfg = dict(n_tokens=0, d_model=d, n_experts=K, n_blocks=B, block_width=M,
               dtype="f32", tau=None, mass_threshold=1.0, max_shared=B,
               alpha_mode="adaptive", alpha_fixed=0.0, mass_mode="coupled",
               fixed_k=1, select_mode="prototype")
    cfg.update(kw)
    return cfg


def random_layer(rng, N, d, K, B, M, weight_scale=1.0, logit_scale=1.0):
    H = B * M
    f = np.float32
    return dict(
        X=rng.standard_normal((N, d)).astype(f),
        W_router=(logit_scale * rng.standard_normal((K + 1, d)) / math.sqrt(d)).astype(f),
        prototypes=(rng.standard_normal((B, d)) / math.sqrt(d)).astype(f),
        W_up=(weight_scale * rng.standard_normal((K + 1, H, d))).astype(f),
        W_down=(weight_scale * rng.standard_normal((K + 1, d, H))).astype(f))


def _forward(O, cfg, L, valid=None):
    cfg = dict(cfg)
    cfg["n_tokens"] = L["X"].shape[0]
    return O.forward(cfg, L["X"], valid, L["W_router"], L["prototypes"], L["W_up"], L["W_down"])


def _close(a, b, rel, what):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    scale = max(1e-30, float(np.abs(b).max()))
    err = float(np.abs(a - b).max()) / scale
    assert err <= rel, f"{what}: relative error {err:.3e} > {rel:.1e}"


# ---------------------------------------------------------------- pins ---
def pin_hand_example(O):
    with open(os.path.join(GOLDEN, "hand_example.json")) as f:
        g = json.load(f)
    f32 = np.float32
    L = dict(X=np.array(g["X"], f32), W_router=np.array(g["W_router"], f32),
             prototypes=np.array(g["prototypes"], f32), W_up=np.array(g["W_up"], f32),
             W_down=np.array(g["W_down"], f32))
    Y, rec = _forward(O, g["config"], L)
    B = g["config"]["n_blocks"]
    for e in g["expected"]:
        t = e["token"]
        assert abs(float(rec["alpha"][t]) - e["alpha"]) < 1e-6, ("alpha", t)
        assert int(rec["n_shared"][t]) == e["n_shared"], ("b", t)
        m = int(rec["shared_mask"][t])
        assert [c for c in range(B) if m >> c & 1] == e["shared_blocks"], ("I_shr", t)
        assert int(rec["n_res"][t]) == e["n_res"], ("k", t)
        assert list(rec["expert_ids"][t]) == e["experts"], ("q", t)
        assert np.allclose(rec["weights"][t], e["weights"], atol=1e-6), ("p", t)
        bc = O.block_count(int(rec["n_shared"][t]), int(rec["n_res"][t]), B)
        assert bc == e["block_count"], ("C_B", t)
        assert np.allclose(Y[t], e["y"], rtol=1e-6, atol=1e-7), ("y", t, Y[t], e["y"])


def pin_gelu(O):
    a = np.linspace(-6.0, 6.0, 241)
    ref = np.array([gelu_tb(v) for v in a])
    assert np.allclose(O.gelu(a), ref, rtol=1e-12, atol=1e-15), "GELU vs a Phi(a)"
    # GELU(a) - GELU(-a) = a (erf is odd) and GELU(0) = 0.
    assert np.allclose(O.gelu(a) - O.gelu(-a), a, atol=1e-12), "GELU odd-part identity"
    assert O.gelu(np.array([0.0]))[0] == 0.0
    # Phi(1) and Phi(2) from the standard normal table.
    assert abs(O.gelu(np.array([1.0]))[0] - 0.8413447460685429) < 1e-12
    assert abs(O.gelu(np.array([2.0]))[0] - 2 * 0.9772498680518208) < 1e-12


def pin_tau(O):
    for B, num, den in ((2, 1, 4), (4, 3, 16), (8, 7, 64), (16, 15, 256), (32, 31, 1024)):
        assert float(O.shared_offset(dict(n_blocks=B, tau=None))) == num / den, B
        assert float(O.shared_offset(dict(n_blocks=B, tau=float("nan")))) == num / den, B
    # A given tau replaces (B-1)/B^2: with x W_shr = ln 3, sigma = 3/4 and
    # alpha = tau + (1 - 2 tau) 3/4 = 0.1 + 0.8 * 0.75 = 0.7 for tau = 0.1.
    assert O.shared_offset(dict(n_blocks=4, tau=0.1)) == np.float32(0.1)
    L = dict(X=np.array([[1.0, 0.0]], np.float32), prototypes=np.eye(2, dtype=np.float32),
             W_router=np.array([[math.log(3.0), 0.0], [0.0, 0.0], [0.0, 0.0]], np.float32),
             W_up=np.zeros((3, 2, 2), np.float32), W_down=np.zeros((3, 2, 2), np.float32))
    _, rec = _forward(O, layer_cfg(2, 2, 2, 1, tau=0.1), L)
    assert abs(float(rec["alpha"][0]) - 0.7) < 1e-6, float(rec["alpha"][0])


def pin_round_half_even(O):
    """Eq. block-count with a fixed alpha: B alpha on exact half-integers."""
    rng = np.random.default_rng(5)
    L = random_layer(rng, 1, 4, 2, 4, 1)
    for alpha, b_expected in ((0.125, 0), (0.375, 2), (0.625, 2), (0.875, 4), (0.3, 1), (0.4, 2)):
        cfg = layer_cfg(4, 2, 4, 1, alpha_mode="fixed", alpha_fixed=alpha)
        _, rec = _forward(O, cfg, L)
        assert int(rec["n_shared"][0]) == b_expected, (alpha, int(rec["n_shared"][0]))


def pin_alpha_range(O):
    """tau < alpha < 1 - tau and b in {1..B-1} (Sec. III-B), including
    saturated sigmoids where B alpha lands on B - 1/2 or 1/2 (B = 2)."""
    rng = np.random.default_rng(6)
    for B in (2, 3, 4, 8):
        d, K = 4, 3
        L = random_layer(rng, 64, d, K, B, 1)
        L["W_router"][0] *= np.float32(200.0)     # saturate sigma for most tokens
        cfg = layer_cfg(d, K, B, 1)
        _, rec = _forward(O, cfg, L)
        tau = (B - 1) / B ** 2
        a = rec["alpha"].astype(np.float64)
        assert np.all(a >= tau - 1e-7) and np.all(a <= 1 - tau + 1e-7), B
        b = rec["n_shared"]
        assert b.min() >= 1 and b.max() <= B - 1, (B, b.min(), b.max())
        if B == 2:
            assert np.all(b == 1)
    # z0 = 0 gives alpha = 1/2 exactly.
    L = random_layer(rng, 1, 4, 2, 4, 1)
    L["W_router"][0] = 0
    _, rec = _forward(O, layer_cfg(4, 2, 4, 1), L)
    assert float(rec["alpha"][0]) == 0.5


def pin_rank_order(O):
    """Order of Eq. sorted-affinity and TopK: decreasing, ties to the lower
    index; equals a stable argsort of the negated values."""
    rng = np.random.default_rng(7)
    v = rng.integers(0, 4, size=(200, 9)).astype(np.float32)   # many ties
    r = O._index_rank(v)
    order = np.argsort(-v, axis=1, kind="stable")
    expect = np.empty_like(order)
    np.put_along_axis(expect, order, np.arange(9)[None, :].repeat(200, 0), axis=1)
    assert np.array_equal(r, expect)


def pin_softmax_large_logits(O):
    """Router logits far beyond float32's exp range (|l| ~ 300): the
    affinities of Eq. residual-router-score stay finite and equal the
    float64 textbook softmax."""
    rng = np.random.default_rng(8)
    d, K, B, M, N = 4, 5, 2, 1, 40
    L = random_layer(rng, N, d, K, B, M, logit_scale=300.0)
    _, rec = _forward(O, layer_cfg(d, K, B, M), L)
    s = tb_softmax(L["X"].astype(float) @ L["W_router"][1:].astype(float).T)
    assert np.all(np.isfinite(rec["s"]))
    assert np.abs(rec["s"] - s).max() < 1e-5, np.abs(rec["s"] - s).max()


def _bf_token(x, L, cfg):
    """Brute-force float64 decisions and output of one token (tiny sizes)."""
    d, K, B, M = cfg["d_model"], cfg["n_experts"], cfg["n_blocks"], cfg["block_width"]
    Wr, Mu = L["W_router"].astype(float), L["prototypes"].astype(float)
    Wu, Wd = L["W_up"].astype(float), L["W_down"].astype(float)
    x = [float(v) for v in x]
    dot = lambda a, b: sum(p * q for p, q in zip(a, b))
    tau = (B - 1) / B ** 2
    alpha = tau + (1 - 2 * tau) / (1 + math.exp(-dot(x, Wr[0])))
    v = B * alpha
    b = min(range(B + 1), key=lambda i: (abs(v - i), i % 2))       # nearest, ties even
    b = min(max(b, 1), B - 1)
    b = min(b, cfg["max_shared"])
    u = [dot(x, Mu[c]) for c in range(B)]
    prefix = cfg.get("select_mode", "prototype") == "prefix"
    if prefix:
        S = tuple(range(b))
    else:
        S = max(itertools.combinations(range(B), b), key=lambda s: sum(u[c] for c in s))
    l = [dot(x, Wr[j]) for j in range(1, K + 1)]
    mx = max(l)
    e = [math.exp(t - mx) for t in l]
    s = [t / sum(e) for t in e]
    target = min(1 - alpha, cfg["mass_threshold"])
    for n in range(1, K + 1):
        best = max(itertools.combinations(range(K), n), key=lambda c: sum(s[j] for j in c))
        if sum(s[j] for j in best) >= target:
            break
    k = n
    y = [0.0] * d
    for c in range(B):
        for h in range(c * M, (c + 1) * M):
            if c in S:
                g = alpha * gelu_tb(dot(x, Wu[0][h]))
                for i in range(d):
                    y[i] += g * Wd[0][i][h]
            else:
                for j in best:
                    g = s[j] * gelu_tb(dot(x, Wu[j + 1][h]))
                    for i in range(d):
                        y[i] += g * Wd[j + 1][i][h]
    # Distances of the continuous quantities to the decision boundaries.
    us = sorted(u, reverse=True)
    ss = sorted(s, reverse=True)
    P = list(itertools.accumulate(ss))
    fb = lambda r: min(min(max(r, 1), B - 1), cfg["max_shared"])
    marg = [abs(v - (h + 0.5)) for h in range(-1, B + 1) if fb(h) != fb(h + 1)]
    margin_b = min(marg, default=math.inf)
    if 0 < b < B and not prefix:
        marg.append(us[b - 1] - us[b])
    if k < K:
        marg.append(ss[k - 1] - ss[k])
    marg.append(abs(P[k - 1] - target))
    if k > 1:
        marg.append(abs(target - P[k - 2]))
    return dict(alpha=alpha, b=b, S=tuple(sorted(S)), k=k, experts=set(j + 1 for j in best),
                order=[j + 1 for j in sorted(range(K), key=lambda j: (-s[j], j))],
                order_gap=min([ss[i] - ss[i + 1] for i in range(K - 1)], default=1.0),
                y=np.array(y), margin=min(marg), margin_b=margin_b)


def pin_bruteforce(O, n_layers=60, n_tok=6, seed=11):
    rng = np.random.default_rng(seed)
    checked = 0
    for i in range(n_layers):
        d = int(rng.integers(1, 5))
        K = int(rng.integers(1, 4))
        B = int(rng.integers(2, 5))
        M = int(rng.integers(1, 3))
        t = float(rng.choice([0.3, 0.6, 1.0]))
        S_max = int(rng.integers(1, B + 1))
        cfg = layer_cfg(d, K, B, M, mass_threshold=t, max_shared=S_max)
        L = random_layer(rng, n_tok, d, K, B, M, logit_scale=float(rng.choice([0.5, 2.0, 6.0])))
        Y, rec = _forward(O, cfg, L)
        for tkn in range(n_tok):
            ref = _bf_token(L["X"][tkn], L, cfg)
            if ref["margin"] < 1e-4:
                continue
            b, S, k, q = O.decisions(rec, tkn)
            assert abs(float(rec["alpha"][tkn]) - ref["alpha"]) < 1e-6, "alpha"
            assert b == ref["b"], ("b", b, ref["b"])
            assert S == ref["S"], ("I_shr", S, ref["S"])
            assert k == ref["k"], ("k", k, ref["k"])
            assert set(q) == ref["experts"], ("experts", q, ref["experts"])
            if ref["order_gap"] >= 1e-4:
                assert list(rec["expert_ids"][tkn]) == ref["order"], ("q", q, ref["order"])
            scale = max(1e-12, float(np.abs(ref["y"]).max()))
            err = float(np.abs(Y[tkn] - ref["y"]).max()) / scale
            assert err < 1e-5, ("y", err)
            checked += 1
    assert checked >= n_layers * n_tok // 2, checked


def pin_topk_moe(O):
    """No shared blocks and a fixed k: the layer is the top-k MoE of Eq.
    vanilla-moe-output over complete experts (affinities not renormalised)."""
    rng = np.random.default_rng(12)
    d, K, B, M, N = 8, 5, 4, 3, 40
    L = random_layer(rng, N, d, K, B, M, weight_scale=0.3, logit_scale=3.0)
    for kk in (1, 2, 5):
        cfg = layer_cfg(d, K, B, M, max_shared=0, mass_mode="topk", fixed_k=kk)
        Y, rec = _forward(O, cfg, L)
        x = L["X"].astype(float)
        s = tb_softmax(x @ L["W_router"][1:].astype(float).T)
        ref = np.zeros_like(Y)
        for j in range(K):
            Fj = tb_ffn(x, L["W_up"][j + 1].astype(float), L["W_down"][j + 1].astype(float))
            top = np.argsort(-s, axis=1, kind="stable")[:, :kk]
            sel = (top == j).any(axis=1)
            ref += (sel * s[:, j])[:, None] * Fj
        _close(Y, ref, 1e-5, f"top-{kk} MoE")
        assert np.all(rec["n_shared"] == 0)


def pin_dense_ffn(O):
    """alpha fixed at 1: every block is shared with weight 1 and the layer is
    the shared expert's dense FFN."""
    rng = np.random.default_rng(13)
    d, K, B, M, N = 6, 3, 4, 2, 30
    L = random_layer(rng, N, d, K, B, M, weight_scale=0.5)
    cfg = layer_cfg(d, K, B, M, alpha_mode="fixed", alpha_fixed=1.0)
    Y, rec = _forward(O, cfg, L)
    ref = tb_ffn(L["X"].astype(float), L["W_up"][0].astype(float), L["W_down"][0].astype(float))
    _close(Y, ref, 1e-9, "dense FFN")
    assert np.all(rec["n_shared"] == B)


def pin_soft_moe(O):
    """No shared blocks and a fixed target of 1: every residual expert is
    active with its affinity, sum_j s_j E_j(x)."""
    rng = np.random.default_rng(14)
    d, K, B, M, N = 6, 4, 2, 3, 30
    L = random_layer(rng, N, d, K, B, M, weight_scale=0.5)
    cfg = layer_cfg(d, K, B, M, max_shared=0, mass_mode="fixed", mass_threshold=1.0)
    Y, rec = _forward(O, cfg, L)
    x = L["X"].astype(float)
    s = tb_softmax(x @ L["W_router"][1:].astype(float).T)
    ref = sum(s[:, j:j + 1] * tb_ffn(x, L["W_up"][j + 1].astype(float), L["W_down"][j + 1].astype(float))
              for j in range(K))
    assert np.all(rec["n_res"] == K)
    _close(Y, ref, 1e-5, "soft MoE")


def pin_identical_experts(O):
    """With identical experts F, y = alpha F^{I_shr}(x) + P_k F^{I_res}(x),
    and the two block sums add up to the dense F(x) (Sec. III-A)."""
    rng = np.random.default_rng(15)
    d, K, B, M, N = 5, 4, 4, 2, 40
    L = random_layer(rng, N, d, K, B, M, weight_scale=0.5)
    L["W_up"][:] = L["W_up"][0]
    L["W_down"][:] = L["W_down"][0]
    cfg = layer_cfg(d, K, B, M, mass_threshold=1.0)
    Y, rec = _forward(O, cfg, L)
    x = L["X"].astype(float)
    hid = _gelu_vec(x @ L["W_up"][0].astype(float).T)           # [N, H]
    Vt = L["W_down"][0].astype(float)                            # [d, H]
    for t in range(N):
        m = int(rec["shared_mask"][t])
        cols = np.array([(m >> (h // M)) & 1 for h in range(B * M)], bool)
        Fs = Vt[:, cols] @ hid[t, cols]
        Fr = Vt[:, ~cols] @ hid[t, ~cols]
        assert np.allclose(Fs + Fr, Vt @ hid[t], atol=1e-9)
        Pk = float(np.sum(rec["weights"][t, : rec["n_res"][t]].astype(float)))
        ref = float(rec["alpha"][t]) * Fs + Pk * Fr
        assert np.allclose(Y[t], ref, rtol=1e-9, atol=1e-9), t


def pin_prefix_selection(O):
    """Prefix selection (ablation): I_shr = the first b blocks."""
    rng = np.random.default_rng(16)
    d, K, B, M, N = 4, 3, 6, 1, 50
    L = random_layer(rng, N, d, K, B, M)
    cfg = layer_cfg(d, K, B, M, select_mode="prefix")
    _, rec = _forward(O, cfg, L)
    for t in range(N):
        b = int(rec["n_shared"][t])
        assert int(rec["shared_mask"][t]) == (1 << b) - 1


def pin_mass_bound(O):
    """Eq. mixture-mass-bound with the paper's target (t = 1):
    beta <= P_k < beta + p_k and 1 <= alpha + P_k < 1 + p_k."""
    rng = np.random.default_rng(17)
    d, K, B, M, N = 16, 8, 8, 1, 500
    L = random_layer(rng, N, d, K, B, M, logit_scale=2.0)
    _, rec = _forward(O, layer_cfg(d, K, B, M, mass_threshold=1.0), L)
    a = rec["alpha"].astype(float)
    k = rec["n_res"]
    p = rec["weights"].astype(float)
    Pk = np.array([p[t, : k[t]].sum() for t in range(N)])
    pk = p[np.arange(N), k - 1]
    eps = 1e-6
    assert np.all(1 - a <= Pk + eps) and np.all(Pk < 1 - a + pk + eps)
    assert np.all(1 <= a + Pk + eps) and np.all(a + Pk < 1 + pk + eps)
    assert np.all((k >= 1) & (k <= K))
    assert np.all(np.diff(p, axis=1) <= 0)
    assert np.allclose(p.sum(axis=1), 1.0, atol=1e-5)
    for t in range(N):
        assert sorted(rec["expert_ids"][t]) == list(range(1, K + 1))


def pin_padding(O):
    rng = np.random.default_rng(18)
    d, K, B, M, N = 4, 3, 4, 2, 10
    L = random_layer(rng, N, d, K, B, M)
    valid = (np.arange(N) % 3 != 0).astype(np.uint8)
    Y, rec = _forward(O, layer_cfg(d, K, B, M), L, valid=valid)
    pad = valid == 0
    assert np.all(Y[pad] == 0) and np.all(rec["n_res"][pad] == 0) and np.all(rec["alpha"][pad] == 0)
    assert np.all(rec["expert_ids"][pad] == -1) and np.all(rec["shared_mask"][pad] == 0)
    assert np.any(Y[~pad] != 0)


def pin_stats(O):
    rng = np.random.default_rng(19)
    d, K, B, M, N = 8, 6, 4, 2, 300
    L = random_layer(rng, N, d, K, B, M, logit_scale=2.0)
    valid = (rng.random(N) < 0.8).astype(np.uint8)
    cfg = layer_cfg(d, K, B, M, mass_threshold=0.7)
    _, rec = _forward(O, cfg, L, valid=valid)
    st = O.stats(cfg, rec)
    v = valid.astype(bool)
    b, k = rec["n_shared"][v], rec["n_res"][v]
    assert st["n_valid"] == v.sum()
    assert st["hist_b"].sum() == v.sum() and st["hist_k"].sum() == v.sum()
    per_expert = np.zeros(K + 1, int)
    for t in np.nonzero(v)[0]:
        for j in rec["expert_ids"][t, : rec["n_res"][t]]:
            per_expert[j] += 1
    assert list(st["expert_tokens"][1:K + 1]) == list(per_expert[1:])
    assert st["expert_tokens"][0] == v.sum()
    cb = b + k * (B - b)
    assert st["activated_blocks"] == cb.sum() and np.all(cb >= B)
    assert st["activated_gemm_flops"] == 4 * d * M * cb.sum()
    for i in range(65):
        assert st["hist_b"][i] == int(np.sum(b == i)) and st["hist_k"][i] == int(np.sum(k == i)), i
    assert st["routing_flops"] == 2 * d * (1 + K + B) * v.sum()
    assert abs(st["mean_b"] - b.mean()) < 1e-12 and abs(st["mean_k"] - k.mean()) < 1e-12
    assert abs(st["mean_cb"] - cb.mean()) < 1e-12


def pin_margins(O):
    """Margins agree with the brute-force float64 distances on tiny layers."""
    rng = np.random.default_rng(20)
    for _ in range(20):
        d, K, B, M = 3, 3, 4, 1
        cfg = layer_cfg(d, K, B, M, mass_threshold=0.8)
        L = random_layer(rng, 8, d, K, B, M, logit_scale=2.0)
        _, rec = _forward(O, cfg, L)
        m, _ = O.margins(cfg, rec)
        for t in range(8):
            ref = _bf_token(L["X"][t], L, cfg)["margin"]
            assert abs(m[t] - ref) < 1e-5, (m[t], ref)


def pin_margins_capped(O):
    """Margins where the cap S_max binds below B - 1 (the breakpoints of b
    move or vanish) and in prefix mode (no selection margin), against the
    brute-force float64 distances; the b-margin is compared on its own."""
    rng = np.random.default_rng(21)
    cases = [(4, 0, "prototype"), (4, 1, "prototype"), (4, 2, "prototype"), (5, 2, "prototype"),
             (5, 3, "prototype"), (4, 4, "prefix"), (5, 2, "prefix")]
    for B, S_max, sel in cases:
        for _ in range(6):
            d, K, M = 3, 3, 1
            cfg = layer_cfg(d, K, B, M, mass_threshold=0.8, max_shared=S_max, select_mode=sel)
            L = random_layer(rng, 8, d, K, B, M, logit_scale=2.0)
            L["W_router"][0] *= np.float32(3.0)       # spread alpha over the whole range
            _, rec = _forward(O, cfg, L)
            m, parts = O.margins(cfg, rec)
            for t in range(8):
                ref = _bf_token(L["X"][t], L, cfg)
                assert abs(m[t] - ref["margin"]) < 1e-5, (B, S_max, sel, m[t], ref["margin"])
                mb, rb = float(parts["m_b"][t]), ref["margin_b"]
                assert (math.isinf(mb) and math.isinf(rb)) or abs(mb - rb) < 1e-5, (B, S_max, sel, mb, rb)
                if sel == "prefix":
                    assert math.isinf(float(parts["m_sel"][t]))


def pin_forced_hand(O):
    """Outputs under given decisions (the near-tie check of the parity
    tests): cases derived by hand from Eq. output and block-expert-output
    on the worked example (tests/golden/hand_example.json, "forced")."""
    with open(os.path.join(GOLDEN, "hand_example.json")) as f:
        g = json.load(f)
    f32 = np.float32
    cfg = dict(g["config"])
    X = np.array(g["X"], f32)
    L = dict(X=X, W_router=np.array(g["W_router"], f32), prototypes=np.array(g["prototypes"], f32),
             W_up=np.array(g["W_up"], f32), W_down=np.array(g["W_down"], f32))
    _, rec = _forward(O, cfg, L)
    W = O.ExpertWeights(cfg, L["W_up"], L["W_down"])
    for e in g["forced"]:
        y = O.forced_forward(cfg, X, rec, e["token"], e["shared_blocks"], e["experts"], W)
        assert np.allclose(y, e["y"], rtol=1e-6, atol=1e-9), ("forced", e["token"], y, e["y"])


def _bf16_bits(v):
    """bfloat16 bit pattern of a float that bfloat16 represents exactly."""
    import struct
    w = struct.unpack(">I", struct.pack(">f", v))[0]
    assert w & 0xFFFF == 0, v
    return w >> 16


def pin_bf16_inputs(O):
    """bf16 inputs: bit patterns of known value decode exactly, and a tiny
    bf16 layer (values rounded to bf16 by exact rational rounding, passed
    as bit patterns) matches the brute force on those values."""
    known = [(0x3F80, 1.0), (0xBF80, -1.0), (0x4049, 3.140625), (0x3F81, 1.0 + 2.0 ** -7),
             (0xC2F7, -123.5), (0x0080, 2.0 ** -126), (0x0001, 2.0 ** -133),
             (0x7F7F, (2.0 - 2.0 ** -7) * 2.0 ** 127), (0x0000, 0.0), (0x3E20, 0.15625)]
    got = O._as_f32(np.array([b for b, _ in known], np.uint16), "bf16")
    assert got.dtype == np.float32
    for (bits, val), gv in zip(known, got):
        assert float(gv) == val, (hex(bits), float(gv), val)
    rng = np.random.default_rng(22)
    checked = 0
    for _ in range(25):
        d, K, B, M = 3, 3, 4, 2
        cfg = layer_cfg(d, K, B, M, mass_threshold=0.7, dtype="bf16")
        L = random_layer(rng, 5, d, K, B, M, logit_scale=3.0)
        for key in ("X", "W_up", "W_down"):
            L[key] = np.vectorize(tb_bf16, otypes=[np.float64])(L[key].astype(np.float64)).astype(np.float32)
        Lb = dict(L)
        for key in ("X", "W_up", "W_down"):
            Lb[key] = np.vectorize(_bf16_bits, otypes=[np.uint16])(L[key].astype(np.float64))
        Y, rec = _forward(O, cfg, Lb)
        for t in range(5):
            ref = _bf_token(L["X"][t], L, cfg)
            if ref["margin"] < 1e-4:
                continue
            b, S, k, q = O.decisions(rec, t)
            assert (b, S, k, set(q)) == (ref["b"], ref["S"], ref["k"], ref["experts"]), "bf16 decisions"
            scale = max(1e-12, float(np.abs(ref["y"]).max()))
            assert float(np.abs(Y[t] - ref["y"]).max()) / scale < 1e-5, "bf16 output"
            checked += 1
    assert checked >= 60, checked


def pin_rounding_slack(O):
    """Distance to the nearest rounding midpoint of the format, at values a
    known dyadic offset from a midpoint (exact), and as a property: no
    midpoint lies within the slack, one lies just beyond it."""
    cases = [  # (value, format, exact slack)
        (1.0 + 2.0 ** -8, "bf16", 0.0),
        (1.0 + 2.0 ** -8 + 2.0 ** -30, "bf16", 2.0 ** -30),
        (1.0 + 3 * 2.0 ** -8 - 2.0 ** -20, "bf16", 2.0 ** -20),
        (-(3.0 + 2.0 ** -7 + 2.0 ** -25), "bf16", 2.0 ** -25),
        (2.0 ** -100 * (1.0 + 2.0 ** -8) + 2.0 ** -131, "bf16", 2.0 ** -131),
        (1.5 + 2.0 ** -24, "f32", 0.0),
        (1.0 + 2.0 ** -24 + 2.0 ** -50, "f32", 2.0 ** -50),
        (-(7.0 + 2.0 ** -22 - 2.0 ** -45), "f32", 2.0 ** -45),
    ]
    for v, fmt, want in cases:
        got = float(O.rounding_slack(np.array([v]), fmt)[0])
        assert got == want, (v, fmt, got, want)
    rng = np.random.default_rng(23)
    vals = rng.standard_normal(400) * 10.0 ** rng.integers(-5, 5, 400)
    for fmt, rel in (("bf16", 2.0 ** -8), ("f32", 2.0 ** -24)):
        sl = O.rounding_slack(vals, fmt)
        for v, dlt in zip(vals, sl):
            if not (0 < dlt < abs(v) * rel / 4):
                continue
            r = lambda z: O.to_format(np.array([z]), fmt)[0]
            assert r(v - 0.5 * dlt) == r(v + 0.5 * dlt), (fmt, v, dlt)
            assert r(v - 1.5 * dlt) != r(v + 1.5 * dlt), (fmt, v, dlt)


# ------------------------------------------------ the block around it ---
def tb_layer_norm_row(v, gamma, beta, eps):
    """LayerNorm of one row in plain Python floats (biased variance)."""
    n = len(v)
    mu = math.fsum(v) / n
    var = math.fsum((a - mu) ** 2 for a in v) / n
    r = 1.0 / math.sqrt(var + float(eps))
    return [(a - mu) * r * float(g) + float(b) for a, g, b in zip(v, gamma, beta)]


def tb_layer_norm(x, gamma, beta, eps):
    return np.array([tb_layer_norm_row(list(map(float, row)), gamma, beta, eps) for row in x])


def tb_bf16(v):
    """Nearest bfloat16 to v (ties to even), by exact rational arithmetic."""
    from fractions import Fraction
    if v == 0:
        return 0.0
    q = Fraction(v)
    e = math.floor(math.log2(abs(v)))
    while Fraction(2) ** e > abs(q):
        e -= 1
    while Fraction(2) ** (e + 1) <= abs(q):
        e += 1
    ulp = Fraction(2) ** (e - 7)
    lo = math.floor(q / ulp)
    rem = q / ulp - lo
    n = lo + 1 if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and lo % 2 == 1) else lo
    return float(n * ulp)


def _block(d, K, B, M, rng, norm, residual, biases=True, eps=1e-5):
    H = B * M
    f = np.float32
    return dict(norm=norm, residual=residual, ln_eps=f(eps),
                ln_gamma=(1.0 + 0.3 * rng.standard_normal(d)).astype(f),
                ln_beta=(0.2 * rng.standard_normal(d)).astype(f),
                b_up=(0.5 * rng.standard_normal((K + 1, H))).astype(f) if biases else None,
                b_down=(0.5 * rng.standard_normal((K + 1, d))).astype(f) if biases else None)


def _block_forward(O, cfg, blk, L, valid=None):
    cfg = dict(cfg)
    cfg["n_tokens"] = L["X"].shape[0]
    return O.block_forward(cfg, blk, L["X"], valid, L["W_router"], L["prototypes"],
                           L["W_up"], L["W_down"])


def pin_layer_norm(O):
    """A row worked by hand, and random rows against plain-Python LayerNorm."""
    x = np.array([[1.0, 2.0, 3.0, 4.0]])
    # mean 5/2, biased variance 5/4, eps 11/4: the scale is 1 / sqrt(4) = 1/2
    y = O.layer_norm(x, [1.0, 2.0, -1.0, 0.5], [0.0, 1.0, 0.0, -1.0], 2.75)
    assert np.array_equal(y, [[-0.75, 0.5, -0.25, -0.625]]), y
    rng = np.random.default_rng(30)
    x = 3.0 * rng.standard_normal((20, 7)) + 5.0
    g = (1 + rng.standard_normal(7)).astype(np.float32)
    b = rng.standard_normal(7).astype(np.float32)
    _close(O.layer_norm(x, g, b, np.float32(1e-3)), tb_layer_norm(x, g, b, np.float32(1e-3)), 1e-12,
           "LayerNorm")


def pin_bf16_rounding(O):
    """Rounding to bf16 against exact rational rounding, including ties and
    values just off a tie (where rounding through float32 first goes wrong)."""
    one = 1.0
    vals = [one, one + 2.0 ** -8, one + 3 * 2.0 ** -8, one + 2.0 ** -8 + 2.0 ** -40,
            -(one + 2.0 ** -8 + 2.0 ** -40), 3.0 * 2.0 ** -100, -7.99, 1e30, 0.0]
    rng = np.random.default_rng(31)
    vals += list(rng.standard_normal(200) * 10.0 ** rng.integers(-6, 6, 200))
    got = O.to_format(np.array(vals), "bf16")
    got_f = (got.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    for v, g in zip(vals, got_f):
        assert g == tb_bf16(v), (v, g, tb_bf16(v))
    assert np.array_equal(O.to_format(np.array(vals), "f32"), np.array(vals, np.float32))


def pin_block_dense(O):
    """alpha fixed at 1, pre-LN, biases and residual: the textbook pre-LN
    block x + GELU(LN(x) K + b1) V + b2 of the shared expert (LN(x) rounded
    to the layer's float32 format)."""
    rng = np.random.default_rng(32)
    d, K, B, M, N = 6, 3, 4, 2, 25
    L = random_layer(rng, N, d, K, B, M, weight_scale=0.5)
    L["X"] = (2.0 * L["X"] + 1.0).astype(np.float32)
    blk = _block(d, K, B, M, rng, "pre", True)
    cfg = layer_cfg(d, K, B, M, alpha_mode="fixed", alpha_fixed=1.0)
    Y, rec, Xin = _block_forward(O, cfg, blk, L)
    xn = tb_layer_norm(L["X"], blk["ln_gamma"], blk["ln_beta"], blk["ln_eps"]).astype(np.float32)
    a = xn.astype(float) @ L["W_up"][0].astype(float).T + blk["b_up"][0].astype(float)
    ref = L["X"].astype(float) + _gelu_vec(a) @ L["W_down"][0].astype(float).T + blk["b_down"][0]
    _close(Y, ref, 1e-9, "pre-LN dense block")
    assert np.array_equal(Xin, xn)


def pin_block_pre_ln_bf16(O):
    """bf16 pre-LN block: the FFN input is LN(x) rounded once to bf16
    (exact rational rounding of the plain-Python LayerNorm)."""
    rng = np.random.default_rng(36)
    d, K, B, M, N = 6, 3, 4, 2, 12
    cfg = layer_cfg(d, K, B, M, dtype="bf16", n_tokens=N)
    x = (3.0 * rng.standard_normal((N, d)) + 1.0)
    xr = np.vectorize(tb_bf16, otypes=[np.float64])(x)
    Xb = np.vectorize(_bf16_bits, otypes=[np.uint16])(xr)
    blk = _block(d, K, B, M, rng, "pre", True)
    got = O.block_input(cfg, blk, Xb)
    ref = tb_layer_norm(xr, blk["ln_gamma"], blk["ln_beta"], blk["ln_eps"])
    want = np.vectorize(lambda v: _bf16_bits(tb_bf16(v)), otypes=[np.uint16])(ref)
    assert got.dtype == np.uint16 and np.array_equal(got, want)


def pin_block_bias_split(O):
    """Zero expert weights leave only the biases: GELU(0 + b1) meets zero
    values, and expert j's b2 enters with its pathway's share of the blocks,
    alpha (b / B) b2_shr + sum_i p_i ((B - b) / B) b2_{q_i}."""
    rng = np.random.default_rng(33)
    d, K, B, M, N = 5, 4, 4, 2, 40
    L = random_layer(rng, N, d, K, B, M, logit_scale=2.0)
    L["W_up"][:] = 0
    L["W_down"][:] = 0
    blk = _block(d, K, B, M, rng, "none", False)
    cfg = layer_cfg(d, K, B, M, mass_threshold=0.8)
    Y, rec, _ = _block_forward(O, cfg, blk, L)
    b2 = blk["b_down"].astype(float)
    for t in range(N):
        b, k = int(rec["n_shared"][t]), int(rec["n_res"][t])
        ref = float(rec["alpha"][t]) * (b / B) * b2[0]
        for i in range(k):
            ref = ref + float(rec["weights"][t, i]) * ((B - b) / B) * b2[rec["expert_ids"][t, i]]
        _close(Y[t], ref, 1e-12, f"bias split, token {t}")


def pin_block_post_ln(O):
    """Post-LN block: LN(x + F(x)) with F the layer itself; and without the
    residual add, LN(F(x))."""
    rng = np.random.default_rng(34)
    d, K, B, M, N = 6, 3, 4, 2, 20
    L = random_layer(rng, N, d, K, B, M, weight_scale=0.5)
    for residual in (True, False):
        blk = _block(d, K, B, M, rng, "post", residual, biases=False)
        Y, _, Xin = _block_forward(O, layer_cfg(d, K, B, M), blk, L)
        F, _ = _forward(O, layer_cfg(d, K, B, M), L)
        z = F + L["X"].astype(float) if residual else F
        _close(Y, tb_layer_norm(z, blk["ln_gamma"], blk["ln_beta"], blk["ln_eps"]), 1e-12,
               "post-LN block")
        assert Xin is L["X"]


def pin_block_padding(O):
    """Padded tokens have no FFN term: pre-LN + residual gives x, post-LN +
    residual gives LN(x)."""
    rng = np.random.default_rng(35)
    d, K, B, M, N = 4, 3, 4, 2, 12
    L = random_layer(rng, N, d, K, B, M)
    valid = (np.arange(N) % 3 != 0).astype(np.uint8)
    pad = valid == 0
    for norm in ("pre", "post"):
        blk = _block(d, K, B, M, rng, norm, True)
        Y, _, _ = _block_forward(O, layer_cfg(d, K, B, M), blk, L, valid=valid)
        x = L["X"][pad].astype(float)
        ref = x if norm == "pre" else tb_layer_norm(x, blk["ln_gamma"], blk["ln_beta"], blk["ln_eps"])
        _close(Y[pad], ref, 1e-12, f"padded rows ({norm})")


# ------------------------------------------------------ backward pass ---
def _fixed_decision_forward(cfg, rec, X, Wr, Wup, Wdown):
    """Layer output in float64 with the record's discrete decisions held
    fixed and alpha, s recomputed in float64 from the parameters (pure
    Python over channels)."""
    N, d = X.shape
    K, B, M = cfg["n_experts"], cfg["n_blocks"], cfg["block_width"]
    tau = (B - 1) / (B * B) if cfg.get("tau") is None else cfg["tau"]
    Y = np.zeros((N, d))
    for t in range(N):
        x = X[t]
        z = Wr @ x
        if cfg["alpha_mode"] == "adaptive":
            alpha = tau + (1 - 2 * tau) / (1 + math.exp(-z[0]))
        else:
            alpha = cfg["alpha_fixed"]
        s = tb_softmax(z[1:])
        mask = int(rec["shared_mask"][t])
        shared = [c for c in range(B) if mask >> c & 1]
        resid = [c for c in range(B) if not mask >> c & 1]
        paths = [(0, shared, alpha)]
        for i in range(int(rec["n_res"][t])):
            j = int(rec["expert_ids"][t, i])
            paths.append((j, resid, s[j - 1]))
        for j, blocks, w in paths:
            for c in blocks:
                for h in range(c * M, (c + 1) * M):
                    Y[t] += w * gelu_tb(float(Wup[j, h] @ x)) * Wdown[j][:, h]
    return Y


def pin_backward_finite_differences(O):
    """Every gradient against central differences of sum(dY * Y) with the
    decisions fixed (float64 forward, step 1e-6)."""
    rng = np.random.default_rng(40)
    d, K, B, M, N = 4, 3, 4, 2, 6
    L = random_layer(rng, N, d, K, B, M, weight_scale=0.7, logit_scale=2.0)
    cfg = layer_cfg(d, K, B, M, mass_threshold=0.8, n_tokens=N)
    _, rec = _forward(O, cfg, L)
    dY = rng.standard_normal((N, d))
    G = O.backward(cfg, L["X"], None, L["W_router"], L["prototypes"], L["W_up"], L["W_down"], dY, rec=rec)
    P = {k: L[k].astype(np.float64) for k in ("X", "W_router", "W_up", "W_down")}
    names = dict(X="dX", W_router="dW_router", W_up="dW_up", W_down="dW_down")

    def loss():
        return float(np.sum(dY * _fixed_decision_forward(cfg, rec, P["X"], P["W_router"], P["W_up"], P["W_down"])))
    h = 1e-6
    for key, gname in names.items():
        fd = np.zeros_like(P[key])
        for idx in np.ndindex(P[key].shape):
            v = P[key][idx]
            P[key][idx] = v + h
            lp = loss()
            P[key][idx] = v - h
            lm = loss()
            P[key][idx] = v
            fd[idx] = (lp - lm) / (2 * h)
        _close(G[gname], fd, 2e-5, f"gradient {gname}")
        assert np.any(fd != 0), gname
    assert np.all(G["dprototypes"] == 0)


def pin_backward_dense_torch(O):
    """alpha fixed at 1: the gradients of the dense FFN, from torch autograd."""
    import torch
    rng = np.random.default_rng(41)
    d, K, B, M, N = 6, 3, 4, 2, 20
    L = random_layer(rng, N, d, K, B, M, weight_scale=0.5)
    cfg = layer_cfg(d, K, B, M, alpha_mode="fixed", alpha_fixed=1.0, n_tokens=N)
    dY = rng.standard_normal((N, d))
    G = O.backward(cfg, L["X"], None, L["W_router"], L["prototypes"], L["W_up"], L["W_down"], dY)
    x = torch.tensor(L["X"], dtype=torch.float64, requires_grad=True)
    wu = torch.tensor(L["W_up"][0], dtype=torch.float64, requires_grad=True)
    wd = torch.tensor(L["W_down"][0], dtype=torch.float64, requires_grad=True)
    y = torch.nn.functional.gelu(x @ wu.T) @ wd.T
    (y * torch.tensor(dY)).sum().backward()
    _close(G["dX"], x.grad.numpy(), 1e-10, "dense dX")
    _close(G["dW_up"][0], wu.grad.numpy(), 1e-10, "dense dW_up")
    _close(G["dW_down"][0], wd.grad.numpy(), 1e-10, "dense dW_down")
    assert np.all(G["dW_up"][1:] == 0) and np.all(G["dW_router"] == 0)


def pin_backward_soft_moe_torch(O):
    """No shared blocks and target 1: y = sum_j s_j E_j(x) with s the softmax
    of the router; every gradient (router included) from torch autograd."""
    import torch
    rng = np.random.default_rng(42)
    d, K, B, M, N = 6, 4, 2, 3, 16
    L = random_layer(rng, N, d, K, B, M, weight_scale=0.5)
    cfg = layer_cfg(d, K, B, M, max_shared=0, mass_mode="fixed", mass_threshold=1.0, n_tokens=N)
    _, rec = _forward(O, cfg, L)
    assert np.all(rec["n_res"] == K)
    dY = rng.standard_normal((N, d))
    G = O.backward(cfg, L["X"], None, L["W_router"], L["prototypes"], L["W_up"], L["W_down"], dY, rec=rec)
    x = torch.tensor(L["X"], dtype=torch.float64, requires_grad=True)
    wr = torch.tensor(L["W_router"], dtype=torch.float64, requires_grad=True)
    wu = torch.tensor(L["W_up"], dtype=torch.float64, requires_grad=True)
    wd = torch.tensor(L["W_down"], dtype=torch.float64, requires_grad=True)
    s = torch.softmax(x @ wr[1:].T, dim=1)
    y = sum(s[:, j - 1:j] * (torch.nn.functional.gelu(x @ wu[j].T) @ wd[j].T) for j in range(1, K + 1))
    (y * torch.tensor(dY)).sum().backward()
    # the oracle takes the softmax derivative at the float32 affinities
    _close(G["dX"], x.grad.numpy(), 1e-6, "soft MoE dX")
    _close(G["dW_router"], wr.grad.numpy(), 1e-6, "soft MoE dW_router")
    _close(G["dW_up"], wu.grad.numpy(), 1e-6, "soft MoE dW_up")
    _close(G["dW_down"], wd.grad.numpy(), 1e-6, "soft MoE dW_down")


def pin_diversity_loss(O):
    """L_div vanishes at orthonormal router columns (exactly, with the zero
    subgradient, for unit vectors); at a random router, its value and
    gradient against torch (Frobenius norm, autograd)."""
    import torch
    rng = np.random.default_rng(43)
    Q, _ = np.linalg.qr(rng.standard_normal((8, 5)))
    assert O.diversity_loss(Q.T)[0] < 1e-12
    L0, g0 = O.diversity_loss(np.eye(8)[:5])
    assert L0 == 0.0 and np.all(g0 == 0)
    # an orthogonal pair of norm 2 columns: G - I = 3 I, L = 3 sqrt(2)
    L2, g2 = O.diversity_loss(2.0 * np.eye(4)[:2])
    assert abs(L2 - 3.0 * math.sqrt(2.0)) < 1e-12
    _close(g2, (2.0 / L2) * 3.0 * 2.0 * np.eye(4)[:2], 1e-12, "L_div gradient, scaled pair")
    W = rng.standard_normal((5, 8))
    Lv, g = O.diversity_loss(W)
    w = torch.tensor(W, requires_grad=True)
    lt = torch.linalg.matrix_norm(w @ w.T - torch.eye(5, dtype=torch.float64), "fro")
    lt.backward()
    assert abs(Lv - lt.item()) < 1e-10 * lt.item()
    _close(g, w.grad.numpy(), 1e-10, "L_div gradient")


ALL_PINS = [pin_hand_example, pin_gelu, pin_tau, pin_round_half_even, pin_alpha_range,
            pin_rank_order, pin_softmax_large_logits, pin_bruteforce, pin_topk_moe, pin_dense_ffn, pin_soft_moe,
            pin_identical_experts, pin_prefix_selection, pin_mass_bound, pin_padding,
            pin_stats, pin_margins, pin_margins_capped, pin_forced_hand, pin_bf16_inputs,
            pin_rounding_slack, pin_layer_norm, pin_bf16_rounding, pin_block_dense,
            pin_block_pre_ln_bf16, pin_block_bias_split, pin_block_post_ln, pin_block_padding,
            pin_backward_finite_differences, pin_backward_dense_torch, pin_backward_soft_moe_torch,
            pin_diversity_loss]
