"""CPU oracle for the forward pass of one UniF-MoE feed-forward layer.

TEST INFRASTRUCTURE ONLY. Only the tests, the smoke check and the CPU-baseline
leg of the benchmark may import this module. It shares no code with the HIP
library and must never be used as a fallback for it.

It follows Sec. III of "Share First, Route What Remains" step by step, in the
paper's order and notation, for one token x (a row of X):

  Sec. III-B  alpha = tau + (1 - 2 tau) sigma(x W_shr), tau = (B-1)/B^2 (Eq. alpha)
              b = round(B alpha)                                   (Eq. block-count)
              u_c = x mu_c                                         (Eq. block-priority)
              I_shr = TopK(u, b), I_res = complement               (Eq. shared-indices,
                                                                    residual-indices)
  Sec. III-C  s = softmax(x W_g) over the K residual experts      (Eq. residual-router-score)
              q = experts by decreasing s, p_i = s_{q_i}          (Eq. sorted-affinity)
              beta = 1 - alpha                                     (Eq. beta)
              k = min{n : p_1 + ... + p_n >= beta}                 (Eq. expert-count)
  Sec. III-D  y = alpha E_shr^S(x) + sum_{i<=k} p_i E_{q_i}^R(x)   (Eq. output) with
              E_j^(c)(x) = sum_{h in block c} GELU(x K_j[:,h]) V_j[h,:]
                                                                   (Eq. block-expert-output)

Precision. Routing decisions turn floating point into integers (b, the
shared block set, the expert order and k), so they are taken in float32, the
precision of the routing kernel: each logit is the exact dot product rounded
once to float32 (computed in float64, then rounded), and every later routing
step is float32 arithmetic in the order written above. Expert outputs and the
final merge are computed in float64 from the float32 alpha and p.

Readings where the paper is silent (each is listed in the design notes):
  * round() is round-half-to-even; in adaptive mode b is kept in [1, B-1]
    (the range Sec. III-B guarantees), then capped at ``max_shared``.
  * TopK and the sort break ties toward the lower index.
  * softmax subtracts the maximum and sums in index order; the prefix sums
    P_n are sequential float32 sums in sorted order.
  * k falls back to K when no prefix reaches the target (a target of 1 whose
    float32 prefix sums stay below 1).
  * The workloads' cumulative-mass threshold t caps the target:
    min(beta, t) ("coupled"); t = 1 is the paper exactly. "fixed" uses t
    alone; "topk" uses a fixed k (the ablation's top-k residual activation).
  * GELU is the exact erf form; the layer itself has no biases.
  * The selected residual experts keep their raw affinities p_i.

The surrounding transformer block (the paper leaves biases out of its
equations and converts layers of pre-LN DeiT and post-LN BERT backbones) is
``block_forward``. Its readings:
  * b1 enters each channel before the GELU: GELU(x K_j[:, h] + b1_j[h]).
  * b2 of expert j is split over the blocks in proportion: a pathway that
    runs the set C of blocks of expert j adds (|C| / B) b2_j, so the shared
    and residual parts of one expert add up to its full FFN (bias included).
  * LayerNorm uses the biased variance over d and its eps inside the square
    root. Pre-LN: y = x + F(LN(x)), LN(x) rounded once to the layer's format
    (it is the FFN's input, routing included). Post-LN: y = LN(x + F(x)).
    The residual add can be switched off (then y = F(..) or LN(F(x))).
  * Padded tokens have F = 0 (no biases); the rest of the block applies.

The backward pass of the layer (``backward``, decisions held fixed) and the
Gram diversity loss of Eq. diversity-loss (``diversity_loss``) are here too,
for the training step.

Parity pins: every function here is checked by tests marked "not gpu"
against brute-force enumeration, closed forms, the textbook top-k MoE /
dense FFN / soft MoE reductions, the mixture-mass bound of Eq.
mixture-mass-bound, and a worked example derived by hand.
"""
import math

import numpy as np
from scipy.special import erf as _erf

F32 = np.float32
F64 = np.float64
_CHUNK = 8192

ALPHA_MODES = ("adaptive", "fixed")
MASS_MODES = ("coupled", "fixed", "topk")
SELECT_MODES = ("prototype", "prefix")


# ---------------------------------------------------------------- helpers ---
def _as_f32(a, dtype):
    """Exact float32 values of an input array (bf16 bit patterns or float32)."""
    if dtype == "bf16":
        a = np.ascontiguousarray(a, dtype=np.uint16)
        return (a.astype(np.uint32) << 16).view(np.float32)
    return np.asarray(a, dtype=np.float32)


def shared_offset(cfg):
    """tau of Eq. alpha as float32: (B-1)/B^2 unless the config sets it."""
    B = cfg["n_blocks"]
    t = cfg.get("tau")
    if t is None or (isinstance(t, float) and math.isnan(t)):
        t = (B - 1) / (B * B)
    return F32(t)


def gelu(a):
    """GELU(a) = a * Phi(a) = a/2 * (1 + erf(a / sqrt 2)), float64."""
    a = np.asarray(a, dtype=F64)
    return 0.5 * a * (1.0 + _erf(a / math.sqrt(2.0)))


def _index_rank(v):
    """rank[n, j] = #{j' : v[n,j'] > v[n,j] or (v[n,j'] == v[n,j] and j' < j)}.

    Position of entry j when the row is ordered by decreasing value, ties to
    the lower index (TopK of Eq. shared-indices, the order of Eq.
    sorted-affinity).
    """
    n, m = v.shape
    greater = v[:, None, :] > v[:, :, None]
    lower_tie = (v[:, None, :] == v[:, :, None]) & (np.arange(m)[None, :] < np.arange(m)[:, None])[None]
    return (greater | lower_tie).sum(axis=2)


# ---------------------------------------------------------------- routing ---
def route(cfg, X, valid, W_router, prototypes):
    """Per-token routing record (Sec. III-B and III-C).

    Returns a dict of arrays, one entry per token:
      alpha f32, n_shared (b) i32, shared_mask u64 (bit c <=> c in I_shr),
      n_res (k) i32, expert_ids i32 [N, K] (q_1..q_K, residual experts
      numbered 1..K, -1 for padded tokens), weights f32 [N, K] (p_1..p_K),
    and, for margins and diagnostics: z0, u [N, B], s [N, K], P [N, K]
    (prefix sums), target, valid.
    """
    N = X.shape[0]
    K, B = cfg["n_experts"], cfg["n_blocks"]
    if cfg["alpha_mode"] not in ALPHA_MODES or cfg["mass_mode"] not in MASS_MODES \
            or cfg["select_mode"] not in SELECT_MODES:
        raise ValueError("unknown routing mode")
    valid = np.ones(N, dtype=bool) if valid is None else np.asarray(valid).astype(bool)
    Wr = np.asarray(W_router, dtype=F32).astype(F64)
    Mu = np.asarray(prototypes, dtype=F32).astype(F64)
    tau = shared_offset(cfg)
    one_minus_2tau = F32(1) - F32(2) * tau
    t_mass = F32(cfg["mass_threshold"])

    rec = dict(
        alpha=np.zeros(N, F32), n_shared=np.zeros(N, np.int32),
        shared_mask=np.zeros(N, np.uint64), n_res=np.zeros(N, np.int32),
        expert_ids=np.full((N, K), -1, np.int32), weights=np.zeros((N, K), F32),
        z0=np.zeros(N, F32), u=np.zeros((N, B), F32), s=np.zeros((N, K), F32),
        P=np.zeros((N, K), F32), target=np.zeros(N, F32), valid=valid.copy())

    for c0 in range(0, N, _CHUNK):
        sl = slice(c0, min(N, c0 + _CHUNK))
        x = _as_f32(X[sl], cfg["dtype"]).astype(F64)
        # Router logits x W_g* (Eq. augmented-router) and block priorities
        # x mu_c (Eq. block-priority), each rounded once to float32.
        z = (x @ Wr.T).astype(F32)
        u = (x @ Mu.T).astype(F32)
        z0, l = z[:, 0], z[:, 1:]

        # Eq. alpha: shared demand.
        if cfg["alpha_mode"] == "adaptive":
            with np.errstate(over="ignore"):          # exp overflow gives sigma = 0
                sigma = F32(1) / (F32(1) + np.exp(-z0))
            alpha = tau + one_minus_2tau * sigma
        else:
            alpha = np.full(z0.shape, F32(cfg["alpha_fixed"]), F32)

        # Eq. block-count: b = round(B alpha), half to even.
        b = np.rint(F32(B) * alpha).astype(np.int64)
        if cfg["alpha_mode"] == "adaptive":
            b = np.clip(b, 1, B - 1)
        b = np.minimum(b, cfg["max_shared"])

        # Eq. shared-indices / residual-indices: the b blocks of largest u.
        if cfg["select_mode"] == "prototype":
            shared = _index_rank(u) < b[:, None]
        else:
            shared = np.arange(B)[None, :] < b[:, None]
        mask = np.zeros(shared.shape[0], np.uint64)
        for c in range(B):
            mask |= shared[:, c].astype(np.uint64) << np.uint64(c)

        # Eq. residual-router-score: softmax over the K residual experts.
        e = np.exp(l - l.max(axis=1, keepdims=True))
        s = e / np.cumsum(e, axis=1, dtype=F32)[:, -1:]

        # Eq. sorted-affinity: q by decreasing affinity, p_i = s_{q_i}.
        rank = _index_rank(s)
        q = np.empty_like(rank)
        np.put_along_axis(q, rank, np.arange(K)[None, :].repeat(rank.shape[0], 0), axis=1)
        p = np.take_along_axis(s, q, axis=1)

        # Eq. beta and the cumulative target.
        beta = F32(1) - alpha
        if cfg["mass_mode"] == "coupled":
            target = np.minimum(beta, t_mass)
        else:
            target = np.full(beta.shape, t_mass, F32)

        # Eq. expert-count: smallest prefix with P_n >= target (else K).
        P = np.cumsum(p, axis=1, dtype=F32)
        if cfg["mass_mode"] == "topk":
            k = np.full(P.shape[0], cfg["fixed_k"], np.int64)
        else:
            reached = P >= target[:, None]
            k = np.where(reached.any(axis=1), reached.argmax(axis=1) + 1, K)

        v = valid[sl]
        rec["alpha"][sl] = np.where(v, alpha, F32(0))
        rec["n_shared"][sl] = np.where(v, b, 0)
        rec["shared_mask"][sl] = np.where(v, mask, np.uint64(0))
        rec["n_res"][sl] = np.where(v, k, 0)
        rec["expert_ids"][sl] = np.where(v[:, None], q + 1, -1)
        rec["weights"][sl] = np.where(v[:, None], p, F32(0))
        rec["z0"][sl], rec["u"][sl], rec["s"][sl] = z0, u, s
        rec["P"][sl], rec["target"][sl] = P, target
    return rec


def decisions(rec, t):
    """Discrete decisions of token t: (b, I_shr as a sorted tuple, k, q_1..q_k)."""
    B = rec["u"].shape[1]
    m = int(rec["shared_mask"][t])
    k = int(rec["n_res"][t])
    return (int(rec["n_shared"][t]), tuple(c for c in range(B) if m >> c & 1),
            k, tuple(int(j) for j in rec["expert_ids"][t, :k]))


# ------------------------------------------------------- expert outputs ---
class ExpertWeights:
    """Expert weights as float64 (exact copies of the bf16 / fp32 inputs)."""

    def __init__(self, cfg, W_up, W_down, b_up=None, b_down=None):
        self.M = cfg["block_width"]
        self.B = cfg["n_blocks"]
        self.up = _as_f32(W_up, cfg["dtype"]).astype(F64)      # [K+1, H, d]
        self.down = _as_f32(W_down, cfg["dtype"]).astype(F64)  # [K+1, d, H]
        # Optional FFN biases (float32 inputs): b1 [K+1, H], b2 [K+1, d].
        self.b_up = None if b_up is None else np.asarray(b_up, F32).astype(F64)
        self.b_down = None if b_down is None else np.asarray(b_down, F32).astype(F64)

    def block_output(self, x, j, c):
        """E_j^(c)(x) of Eq. block-expert-output, float64 [d] (with b1 when
        the block has biases)."""
        h = slice(c * self.M, (c + 1) * self.M)
        a = self.up[j, h] @ x                 # x K_j[:, h] for the M channels
        if self.b_up is not None:
            a = a + self.b_up[j, h]
        return self.down[j][:, h] @ gelu(a)   # sum_h GELU(.) V_j[h, :]

    def selected_output(self, x, j, blocks):
        """Sum of E_j^(c)(x) over the given blocks (Eq. selected-shared-output,
        selected-residual-output), plus the blocks' share |blocks| / B of b2_j
        when the block has biases."""
        y = np.zeros(self.down.shape[1], F64)
        for c in blocks:
            y += self.block_output(x, j, c)
        if self.b_down is not None:
            y = y + (len(blocks) / self.B) * self.b_down[j]
        return y


def _token_output(W, x, alpha, shared_blocks, residual):
    """Eq. output: alpha E_shr^S(x) + sum_i w_i E_{j_i}^R(x), float64.

    ``residual`` lists (expert j, weight w) in the order they are summed.
    """
    res_blocks = [c for c in range(W.B) if c not in set(shared_blocks)]
    y = F64(alpha) * W.selected_output(x, 0, shared_blocks)
    for j, w in residual:
        y = y + F64(w) * W.selected_output(x, j, res_blocks)
    return y


def forward(cfg, X, valid, W_router, prototypes, W_up, W_down, tokens=None,
            rec=None, weights=None):
    """Layer output Y (float64 [N, d]) and the routing record.

    ``tokens`` restricts the expert evaluation to those token indices (the
    other rows stay zero); routing always covers every token.
    """
    if rec is None:
        rec = route(cfg, X, valid, W_router, prototypes)
    W = weights if weights is not None else ExpertWeights(cfg, W_up, W_down)
    N, d = X.shape
    Y = np.zeros((N, d), F64)
    idx = range(N) if tokens is None else tokens
    for t in idx:
        if not rec["valid"][t]:
            continue
        x = _as_f32(X[t], cfg["dtype"]).astype(F64)
        b, shared_blocks, k, q = decisions(rec, t)
        residual = [(q[i], rec["weights"][t, i]) for i in range(k)]
        Y[t] = _token_output(W, x, rec["alpha"][t], shared_blocks, residual)
    return Y, rec


def forced_forward(cfg, X, rec, t, shared_blocks, experts, weights):
    """Output of token t under given discrete decisions.

    The shared block set and the residual expert set are taken as inputs
    (for a near-tie token, the set another implementation chose); alpha and
    the affinities s_j are the oracle's own float32 values.
    """
    x = _as_f32(X[t], cfg["dtype"]).astype(F64)
    residual = [(j, rec["s"][t, j - 1]) for j in experts]
    return _token_output(weights, x, rec["alpha"][t], list(shared_blocks), residual)


# ----------------------------------------------------- transformer block ---
NORM_MODES = ("none", "pre", "post")


def layer_norm(v, gamma, beta, eps):
    """LayerNorm over the last axis, float64: (v - mean) / sqrt(var + eps)
    gamma + beta with the biased variance; gamma, beta and eps are float32
    inputs."""
    v = np.asarray(v, F64)
    mu = v.mean(axis=-1, keepdims=True)
    var = np.mean((v - mu) ** 2, axis=-1, keepdims=True)
    g = np.asarray(gamma, F32).astype(F64)
    b = np.asarray(beta, F32).astype(F64)
    return (v - mu) / np.sqrt(var + F64(F32(eps))) * g + b


def to_format(v, dtype):
    """float64 -> the layer's format, rounded once to nearest, ties to even:
    bf16 bit patterns (uint16) or float32. (bf16: exact for values in the
    normal range and zero.)"""
    v = np.asarray(v, F64)
    if dtype == "f32":
        return v.astype(F32)
    m, e = np.frexp(v)                                   # v = m 2^e, 1/2 <= |m| < 1
    r = np.ldexp(np.rint(np.ldexp(m, 8)), e - 8)         # 8 significant bits
    return (r.astype(F32).view(np.uint32) >> np.uint32(16)).astype(np.uint16)


def rounding_slack(v, dtype):
    """Distance (float64) of each value to the nearest point where its
    rounding to the layer's format changes (a midpoint between two
    neighbours). Midpoints are taken within the value's own binade, so the
    result is exact whenever it is below a quarter of the format's spacing
    at the value (the only range the near-tie checks use); larger results
    can overstate the distance to a midpoint just below a power of two."""
    v = np.asarray(v, F64)
    bits = 8 if dtype == "bf16" else 24
    m, e = np.frexp(v)
    s = np.ldexp(np.abs(m), bits)
    return np.ldexp(np.abs(s - (np.floor(s) + 0.5)), e - bits)


def block_weights(cfg, blk, W_up, W_down):
    return ExpertWeights(cfg, W_up, W_down, blk.get("b_up"), blk.get("b_down"))


def block_input(cfg, blk, X):
    """The FFN's input: LN(x) rounded to the layer's format (pre-LN), else X."""
    if blk["norm"] != "pre":
        return X
    x = _as_f32(X, cfg["dtype"]).astype(F64)
    return to_format(layer_norm(x, blk["ln_gamma"], blk["ln_beta"], blk["ln_eps"]), cfg["dtype"])


def block_finish(cfg, blk, X, F):
    """Residual add and post-LN around FFN outputs F (float64 rows of the
    tokens in X)."""
    z = F + _as_f32(X, cfg["dtype"]).astype(F64) if blk["residual"] else F
    if blk["norm"] == "post":
        z = layer_norm(z, blk["ln_gamma"], blk["ln_beta"], blk["ln_eps"])
    return z


def block_forward(cfg, blk, X, valid, W_router, prototypes, W_up, W_down, tokens=None,
                  weights=None):
    """Transformer-block output around the layer (float64 [N, d]), the
    routing record and the FFN input.

    ``blk``: norm ("none", "pre", "post"), residual (bool), ln_gamma and
    ln_beta [d] and ln_eps (float32), b_up [K+1, H] and b_down [K+1, d]
    (float32 or None). With ``tokens`` only those rows are block outputs.
    """
    if blk["norm"] not in NORM_MODES:
        raise ValueError("unknown norm mode")
    Xin = block_input(cfg, blk, X)
    W = weights if weights is not None else block_weights(cfg, blk, W_up, W_down)
    F, rec = forward(cfg, Xin, valid, W_router, prototypes, None, None, tokens=tokens,
                     weights=W)
    return block_finish(cfg, blk, X, F), rec, Xin


# ---------------------------------------------------------- backward pass ---
def gelu_grad(a):
    """d GELU / da = Phi(a) + a phi(a), float64."""
    a = np.asarray(a, dtype=F64)
    return 0.5 * (1.0 + _erf(a / math.sqrt(2.0))) + a * np.exp(-0.5 * a * a) / math.sqrt(2.0 * math.pi)


def backward(cfg, X, valid, W_router, prototypes, W_up, W_down, dY, rec=None, weights=None):
    """Gradients of sum(dY * Y) for the layer's forward (float64).

    Readings (the paper does not give gradients): the discrete decisions b,
    I_shr, the expert order q and k are held fixed (they are piecewise
    constant); gradients flow through alpha (Eq. alpha, to W_shr and x;
    none in fixed-alpha mode), through the affinities p_i of the selected
    experts (the softmax of Eq. residual-router-score, to W_1..W_K and x) and
    through the expert FFNs (Eq. block-expert-output). The prototypes mu get
    no gradient (they only enter TopK). alpha and the softmax derivatives are
    taken at the record's float32 values.

    Returns dict(dX [N, d], dW_up [K+1, H, d], dW_down [K+1, d, H],
    dW_router [K+1, d], dprototypes [B, d] (zeros)).
    """
    if rec is None:
        rec = route(cfg, X, valid, W_router, prototypes)
    W = weights if weights is not None else ExpertWeights(cfg, W_up, W_down)
    N, d = X.shape
    K, B, M = cfg["n_experts"], cfg["n_blocks"], cfg["block_width"]
    Wr = np.asarray(W_router, dtype=F32).astype(F64)
    dY = np.asarray(dY, dtype=F64)
    tau = F64(shared_offset(cfg))
    dX = np.zeros((N, d), F64)
    dWup = np.zeros_like(W.up)
    dWdown = np.zeros_like(W.down)
    dWr = np.zeros_like(Wr)
    for t in range(N):
        if not rec["valid"][t]:
            continue
        x = _as_f32(X[t], cfg["dtype"]).astype(F64)
        g = dY[t]
        b, shared_blocks, k, q = decisions(rec, t)
        res_blocks = [c for c in range(B) if c not in set(shared_blocks)]
        pathways = [(0, shared_blocks, F64(rec["alpha"][t]))]
        pathways += [(q[i], res_blocks, F64(rec["weights"][t, i])) for i in range(k)]
        dcoef = []
        for j, blocks, w in pathways:
            E = np.zeros(d, F64)
            dE = w * g                                   # gradient of the pathway output
            for c in blocks:
                h = slice(c * M, (c + 1) * M)
                a = W.up[j, h] @ x
                act = gelu(a)
                E += W.down[j][:, h] @ act
                dWdown[j][:, h] += np.outer(dE, act)
                da = (W.down[j][:, h].T @ dE) * gelu_grad(a)
                dWup[j, h] += np.outer(da, x)
                dX[t] += W.up[j, h].T @ da
            dcoef.append(g @ E)                          # d loss / d (pathway weight)
        # alpha = tau + (1 - 2 tau) sigma(z0), z0 = x W_shr
        if cfg["alpha_mode"] == "adaptive":
            sig = 1.0 / (1.0 + math.exp(-F64(rec["z0"][t])))
            dz0 = dcoef[0] * (1.0 - 2.0 * tau) * sig * (1.0 - sig)
            dWr[0] += dz0 * x
            dX[t] += dz0 * Wr[0]
        # p_i = s_{q_i}, s = softmax(l), l_j = x W_j: ds/dl = diag(s) - s s^T
        dp = np.zeros(K, F64)
        for i in range(k):
            dp[q[i] - 1] += dcoef[1 + i]
        sv = rec["s"][t].astype(F64)
        dl = sv * (dp - sv @ dp)
        dWr[1:] += np.outer(dl, x)
        dX[t] += dl @ Wr[1:]
    return dict(dX=dX, dW_up=dWup, dW_down=dWdown, dW_router=dWr,
                dprototypes=np.zeros((B, d), F64))


def diversity_loss(W_router):
    """L_div = || W* ^T W* - I_{K+1} ||_F (Eq. diversity-loss), W* = the
    augmented router with columns W_shr, W_1..W_K (rows of W_router), and
    its gradient with respect to W_router: (2 / L_div) (G - I) W_router with
    G = W_router W_router^T (zero where L_div = 0). float64."""
    Wr = np.asarray(W_router, dtype=F64)
    G = Wr @ Wr.T
    D = G - np.eye(Wr.shape[0])
    L = math.sqrt(float(np.sum(D * D)))
    grad = np.zeros_like(Wr) if L == 0.0 else (2.0 / L) * (D @ Wr)
    return L, grad


# ------------------------------------------------------------- margins ---
def margins(cfg, rec):
    """Per-token distance (float64) of each discrete decision to its boundary.

    m_b   : distance of B*alpha to the nearest half-integer at which the final
            (clamped, capped) b changes;
    m_sel : u_(b) - u_(b+1) over the sorted priorities (inf if b in {0, B}
            or in prefix mode);
    m_set : p_k - p_{k+1} (inf if k = K);
    m_k   : distance of the prefix sums P_k, P_{k-1} to the target (inf in
            top-k mode).
    Returns (m, dict of the four) where m is their minimum; padded tokens
    get inf.
    """
    K, B = cfg["n_experts"], cfg["n_blocks"]
    N = rec["alpha"].shape[0]
    inf = np.inf
    v = rec["valid"]

    # b as a function of B*alpha: its breakpoints are the half-integers
    # h + 1/2 where the clamped, capped value changes.
    def final_b(r):
        bb = r
        if cfg["alpha_mode"] == "adaptive":
            bb = min(max(bb, 1), B - 1)
        return min(bb, cfg["max_shared"])
    breaks = np.array([h + 0.5 for h in range(-1, B + 1) if final_b(h) != final_b(h + 1)], F64)
    Ba = F64(B) * rec["alpha"].astype(F64)
    if breaks.size:
        m_b = np.abs(Ba[:, None] - breaks[None, :]).min(axis=1)
    else:
        m_b = np.full(N, inf)

    b = rec["n_shared"].astype(np.int64)
    us = -np.sort(-rec["u"].astype(F64), axis=1)
    m_sel = np.full(N, inf)
    if cfg["select_mode"] == "prototype":
        inner = (b > 0) & (b < B)
        rows = np.nonzero(inner)[0]
        m_sel[rows] = us[rows, b[rows] - 1] - us[rows, b[rows]]

    k = rec["n_res"].astype(np.int64)
    p = rec["weights"].astype(F64)
    m_set = np.full(N, inf)
    rows = np.nonzero((k >= 1) & (k < K))[0]
    m_set[rows] = p[rows, k[rows] - 1] - p[rows, k[rows]]

    m_k = np.full(N, inf)
    if cfg["mass_mode"] != "topk":
        P = rec["P"].astype(F64)
        tg = rec["target"].astype(F64)
        rows = np.nonzero(k >= 1)[0]
        m_k[rows] = np.abs(P[rows, k[rows] - 1] - tg[rows])
        rows = np.nonzero(k >= 2)[0]
        m_k[rows] = np.minimum(m_k[rows], np.abs(tg[rows] - P[rows, k[rows] - 2]))

    parts = dict(m_b=m_b, m_sel=m_sel, m_set=m_set, m_k=m_k)
    m = np.minimum.reduce([m_b, m_sel, m_set, m_k])
    m = np.where(v, m, inf)
    return m, parts


# --------------------------------------------------------------- stats ---
def block_count(b, k, B):
    """C_B = b + k (B - b), blocks activated by a token (Eq. block-compute)."""
    return b + k * (B - b)


def stats(cfg, rec):
    """Counts over valid tokens: histograms of b and k, tokens per expert
    (index 0 = shared expert), mean b / k / C_B, activated blocks and the
    activated expert-GEMM FLOPs 4 d M C_B (up- and down-projection)."""
    K, B, d, M = cfg["n_experts"], cfg["n_blocks"], cfg["d_model"], cfg["block_width"]
    v = rec["valid"]
    b = rec["n_shared"][v].astype(np.int64)
    k = rec["n_res"][v].astype(np.int64)
    nv = int(v.sum())
    hist_b = np.bincount(b, minlength=65)[:65]
    hist_k = np.bincount(k, minlength=65)[:65]
    exp_tokens = np.zeros(65, np.int64)
    exp_tokens[0] = nv
    ids = rec["expert_ids"][v]
    for i in range(K):
        sel = k > i
        exp_tokens[: K + 1] += np.bincount(ids[sel, i], minlength=K + 1)[: K + 1]
    exp_tokens[0] = nv
    cb = block_count(b, k, B)
    total_cb = int(cb.sum())
    return dict(
        n_valid=nv, hist_b=hist_b, hist_k=hist_k, expert_tokens=exp_tokens,
        mean_b=float(b.mean()) if nv else 0.0, mean_k=float(k.mean()) if nv else 0.0,
        mean_cb=float(cb.mean()) if nv else 0.0, activated_blocks=total_cb,
        activated_gemm_flops=4.0 * d * M * total_cb,
        routing_flops=2.0 * d * (1 + K + B) * nv)
