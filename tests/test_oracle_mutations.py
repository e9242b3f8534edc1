"""Planted mistakes in a copy of the oracle must be caught by the pins.

Each mutant replaces one expression of the oracle's source (a dropped term,
a wrong sign, index or comparison, a skipped step), is loaded as a separate
module, and is run against every pin of tests/oracle_pins.py; at least one
pin has to fail. This shows the pins constrain each step of the oracle, not
only its overall shape. CPU only; the real oracle is untouched.
"""
import inspect
import types

import pytest

import oracle.unif_moe_oracle as O
from tests import oracle_pins as P

MUTANTS = {
    "sigmoid_sign": ("np.exp(-z0)", "np.exp(z0)"),
    "tau_dropped": ("alpha = tau + one_minus_2tau * sigma", "alpha = sigma"),
    "round_is_floor": ("np.rint(F32(B) * alpha)", "np.floor(F32(B) * alpha)"),
    "clamp_dropped": ("b = np.clip(b, 1, B - 1)", "b = np.clip(b, 0, B)"),
    "cap_dropped": ('b = np.minimum(b, cfg["max_shared"])', "b = b"),
    "smallest_priorities": ("shared = _index_rank(u) < b[:, None]", "shared = _index_rank(-u) < b[:, None]"),
    "softmax_unnormalised": ("s = e / np.cumsum(e, axis=1, dtype=F32)[:, -1:]", "s = e"),
    "ascending_sort": ("rank = _index_rank(s)", "rank = _index_rank(-s)"),
    "strict_mass_test": ("reached = P >= target[:, None]", "reached = P > target[:, None]"),
    "demand_is_alpha": ("target = np.minimum(beta, t_mass)", "target = np.minimum(alpha, t_mass)"),
    "k_off_by_one": ("reached.argmax(axis=1) + 1, K)", "np.minimum(reached.argmax(axis=1) + 2, K), K)"),
    "expert_ids_zero_based": ('np.where(v[:, None], q + 1, -1)', 'np.where(v[:, None], q, -1)'),
    "residual_on_shared_blocks": ("res_blocks = [c for c in range(W.B) if c not in set(shared_blocks)]",
                                  "res_blocks = list(shared_blocks)"),
    "shared_weight_dropped": ("y = F64(alpha) * W.selected_output(x, 0, shared_blocks)",
                              "y = W.selected_output(x, 0, shared_blocks)"),
    "gelu_dropped": ("return self.down[j][:, h] @ gelu(a)", "return self.down[j][:, h] @ a"),
    "gelu_tanh": ("return 0.5 * a * (1.0 + _erf(a / math.sqrt(2.0)))", "return 0.5 * a * (1.0 + np.tanh(a))"),
    "wrong_block_slice": ("h = slice(c * self.M, (c + 1) * self.M)", "h = slice(c, c + self.M)"),
    "value_rows_swapped": ("a = self.up[j, h] @ x", "a = self.up[(j + 1) % self.up.shape[0], h] @ x"),
    "margin_set_wrong": ("m_set[rows] = p[rows, k[rows] - 1] - p[rows, k[rows]]",
                         "m_set[rows] = p[rows, 0] - p[rows, k[rows]]"),
    "stats_cb_wrong": ("return b + k * (B - b)", "return b + k * B"),
    "b1_dropped": ("a = a + self.b_up[j, h]", "a = a"),
    "b2_unsplit": ("y = y + (len(blocks) / self.B) * self.b_down[j]", "y = y + self.b_down[j]"),
    "b2_on_shared_row": ("y = y + (len(blocks) / self.B) * self.b_down[j]",
                         "y = y + (len(blocks) / self.B) * self.b_down[0]"),
    "ln_unbiased_variance": ("var = np.mean((v - mu) ** 2, axis=-1, keepdims=True)",
                             "var = np.sum((v - mu) ** 2, axis=-1, keepdims=True) / (v.shape[-1] - 1)"),
    "ln_eps_outside_root": ("(v - mu) / np.sqrt(var + F64(F32(eps)))", "(v - mu) / (np.sqrt(var) + F64(F32(eps)))"),
    "ln_shift_dropped": ("* g + b\n", "* g\n"),
    "bf16_through_f32": ("r = np.ldexp(np.rint(np.ldexp(m, 8)), e - 8)",
                         "r = np.ldexp(np.rint(np.ldexp(m.astype(F32).astype(F64), 8)), e - 8)"),
    "bf16_truncated": ("np.rint(np.ldexp(m, 8))", "np.trunc(np.ldexp(m, 8))"),
    "pre_ln_on_output": ('if blk["norm"] == "post":', 'if blk["norm"] in ("pre", "post"):'),
    "residual_dropped": ('z = F + _as_f32(X, cfg["dtype"]).astype(F64) if blk["residual"] else F', "z = F"),
    "gelu_grad_missing_density": ("+ a * np.exp(-0.5 * a * a) / math.sqrt(2.0 * math.pi)", "+ 0.0"),
    "sigmoid_slope_dropped": ("dz0 = dcoef[0] * (1.0 - 2.0 * tau) * sig * (1.0 - sig)", "dz0 = dcoef[0] * sig"),
    "softmax_jacobian_sign": ("dl = sv * (dp - sv @ dp)", "dl = sv * (dp + sv @ dp)"),
    "router_dx_dropped": ("dX[t] += dl @ Wr[1:]", "dX[t] += 0.0 * (dl @ Wr[1:])"),
    "dWdown_from_preactivation": ("dWdown[j][:, h] += np.outer(dE, act)", "dWdown[j][:, h] += np.outer(dE, a)"),
    "pathway_weight_dropped": ("dE = w * g ", "dE = g "),
    "dWup_transposed_input": ("dWup[j, h] += np.outer(da, x)", "dWup[j, h] += np.outer(da, x[::-1])"),
    "div_grad_factor": ("(2.0 / L) * (D @ Wr)", "(1.0 / L) * (D @ Wr)"),
    "div_squared": ("L = math.sqrt(float(np.sum(D * D)))", "L = float(np.sum(D * D))"),
    "forced_weight_lookup": ('residual = [(j, rec["s"][t, j - 1]) for j in experts]',
                             'residual = [(j, rec["s"][t, j % rec["s"].shape[1]]) for j in experts]'),
    "bf16_decode_shift": ("(a.astype(np.uint32) << 16)", "(a.astype(np.uint32) << 15)"),
    "slack_bf16_7_bits": ('bits = 8 if dtype == "bf16" else 24', 'bits = 7 if dtype == "bf16" else 24'),
    "margins_cap_ignored": ('return min(bb, cfg["max_shared"])', "return bb"),
    "stats_hist_k_from_b": ("hist_k = np.bincount(k, minlength=65)[:65]", "hist_k = np.bincount(b, minlength=65)[:65]"),
    "routing_flops_no_shr": ("routing_flops=2.0 * d * (1 + K + B) * nv", "routing_flops=2.0 * d * (K + B) * nv"),
    "softmax_min_shift": ("e = np.exp(l - l.max(axis=1, keepdims=True))", "e = np.exp(l - l.min(axis=1, keepdims=True))"),
    "tau_ignored": ("    return F32(t)\n", "    return F32((B - 1) / (B * B))\n"),
    "pre_ln_input_unrounded": ('return to_format(layer_norm(x, blk["ln_gamma"], blk["ln_beta"], blk["ln_eps"]), cfg["dtype"])',
                               'return layer_norm(x, blk["ln_gamma"], blk["ln_beta"], blk["ln_eps"]).astype(F32)'),
}


def _mutant(name):
    old, new = MUTANTS[name]
    src = inspect.getsource(O)
    assert src.count(old) == 1, f"mutation site of {name} not unique"
    mod = types.ModuleType(f"oracle_mutant_{name}")
    exec(compile(src.replace(old, new), mod.__name__, "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name):
    mod = _mutant(name)
    for pin in P.ALL_PINS:
        try:
            pin(mod)
        except Exception:
            return
    pytest.fail(f"no pin catches mutant {name}")
