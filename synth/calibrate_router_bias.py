"""Fit the router bias that gives MoE workloads Zipf-skewed expert loads.

Input synthesis only: it shapes the distribution of routed tokens, it does
not compute anything the parity tests compare.

The synthetic router produces logits x . W_r with x ~ N(0, 1) and W_r ~
N(0, 1/H), i.e. about N(0, 1) per expert.  A Zipf law with exponent 1.1 over
128 experts cannot be met exactly under top-8 routing (rank 1 would need 22.6 %
of all pairs, but an expert is picked at most once per token), so the target
is the capped profile  pi_r = min(1, c * r^-1.1)  with sum_r pi_r = top_k,
where pi_r is the fraction of tokens routed to the expert of rank r and ranks
follow a seeded permutation.  The bias is fitted by the fixed-point iteration
b <- b + 0.5 * (log pi_target - log pi_observed) on 65,536 simulated tokens.

    python -m synth.calibrate_router_bias      (writes router_bias_e128_k8.json)
"""
from __future__ import annotations

import json
import os

import numpy as np

from . import gen

HERE = os.path.dirname(os.path.abspath(__file__))
OUT = os.path.join(HERE, "router_bias_e128_k8.json")


def capped_zipf(E: int, k: int, s: float = 1.1) -> np.ndarray:
    """pi_r = min(1, c r^-s), sum pi = k, by bisection on c."""
    r = np.arange(1, E + 1, dtype=np.float64)
    lo, hi = 0.0, float(k)
    for _ in range(200):
        c = 0.5 * (lo + hi)
        if np.minimum(1.0, c * r ** -s).sum() < k:
            lo = c
        else:
            hi = c
    return np.minimum(1.0, hi * r ** -s)


def fit(E: int = 128, k: int = 8, tokens: int = 65536, iters: int = 60, seed: int = 4242):
    rank_of = np.empty(E, np.int64)
    rank_of[gen.permutation(seed, 1, E)] = np.arange(E)   # expert -> rank (0 = most popular)
    target = capped_zipf(E, k)[rank_of]                   # per expert
    z = gen.normal(gen.stream_key(seed, 2, gen.KIND_MISC), tokens * E).reshape(tokens, E)
    b = np.zeros(E)
    for _ in range(iters):
        sel = np.argpartition(-(z + b), k - 1, axis=1)[:, :k]
        frac = np.bincount(sel.ravel(), minlength=E) / tokens
        b += 0.5 * (np.log(target) - np.log(np.maximum(frac, 0.5 / tokens)))
        b = np.clip(b - b.mean(), -8.0, 8.0)
    sel = np.argpartition(-(z + b), k - 1, axis=1)[:, :k]
    frac = np.bincount(sel.ravel(), minlength=E) / tokens
    return b, target, frac, rank_of


def main() -> None:
    b, target, frac, rank_of = fit()
    json.dump({"n_experts": 128, "top_k": 8, "zipf_exponent": 1.1, "calibration_tokens": 65536,
               "seed": 4242, "bias": [round(float(v), 6) for v in b],
               "target_load": [round(float(v), 6) for v in target],
               "fitted_load": [round(float(v), 6) for v in frac],
               "rank": [int(r) for r in rank_of]}, open(OUT, "w"), indent=1)
    print(f"wrote {OUT}; max relative load error {np.max(np.abs(frac - target) / target):.3f}")


def load_bias() -> np.ndarray:
    """The fitted fp32 bias of the 128-expert, top-8 workloads."""
    return np.asarray(json.load(open(OUT))["bias"], dtype=np.float32)


if __name__ == "__main__":
    main()
