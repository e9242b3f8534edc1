"""Writes synth/calibration.json: router scales of two workloads, fitted
with the oracle's routing (test infrastructure; calls only oracle/ and the
input generator).

bert_base_padded: one scale s on the residual router rows, found by
  bisection so that the mean residual expert count k over the valid tokens is
  2.00 +- 0.02 at threshold 0.5.
zipf_stress: one scale c_j per residual router row; starting from 1, 60
  multiplicative steps c_j <- c_j (pi_j / f_j)^0.15 on the first 16384 tokens
  drive the top-1 expert frequency f_j toward pi_j ~ j^-1.2 (Zipf, s = 1.2).

Run: python -m oracle.calibrate
"""
import json
import os

import numpy as np

from synth.generate import _CAL_PATH, generate
from synth.configs import get_config
from oracle.unif_moe_oracle import route


def _mean_k(name, scale):
    g = generate(name, weights=False, router_scales=scale)
    rec = route(g["cfg"], g["X"], g["valid"], g["W_router"], g["prototypes"])
    return float(rec["n_res"][rec["valid"]].mean())


def calibrate_bert():
    lo, hi = 0.05, 8.0          # mean k decreases as the logits sharpen
    for _ in range(60):
        mid = 0.5 * (lo + hi)
        mk = _mean_k("bert_base_padded", mid)
        if abs(mk - 2.0) <= 0.005:
            break
        if mk > 2.0:
            lo = mid
        else:
            hi = mid
    return dict(residual_scale=mid, mean_k=mk)


def calibrate_zipf(n_cal=16384, steps=60, rate=0.15):
    cfg = get_config("zipf_stress")
    K = cfg["n_experts"]
    pi = np.arange(1, K + 1, dtype=np.float64) ** -1.2
    pi /= pi.sum()
    c = np.ones(K)
    for _ in range(steps):
        g = generate("zipf_stress", n_tokens=n_cal, weights=False, router_scales=c)
        rec = route(g["cfg"], g["X"], g["valid"], g["W_router"], g["prototypes"])
        top1 = rec["expert_ids"][:, 0]
        f = np.bincount(top1, minlength=K + 1)[1:] / n_cal
        c = c * (pi / np.maximum(f, 1.0 / n_cal)) ** rate
    return dict(residual_scales=[float(v) for v in c],
                top1_freq=[float(v) for v in f], target_freq=[float(v) for v in pi])


def main():
    out = {}
    if os.path.exists(_CAL_PATH):
        with open(_CAL_PATH) as fh:
            out = json.load(fh)
    out["bert_base_padded"] = calibrate_bert()
    print("bert_base_padded", out["bert_base_padded"])
    out["zipf_stress"] = calibrate_zipf()
    print("zipf_stress scales", np.round(out["zipf_stress"]["residual_scales"], 3))
    with open(_CAL_PATH, "w") as fh:
        json.dump(out, fh, indent=1)


if __name__ == "__main__":
    main()
