"""Thresholds of the synthetic workloads, set from oracle values.

The paper's lambda in {-1, -1.5, -2, -3} and alpha = -0.8 are calibrated to real
models, whose turn means sit near -0.7 (Sec. 3.2, Observation 1).  Synthetic
N(0, 3) logits over V = 151936 put turn means near -11, so the thresholds are
set from the oracle's own values by fixed rules instead:

  tiny       lambda strictly between the planted rollout's cumulative value at
             its planted turn and the larger of (its value one turn earlier,
             the clean rollout's final value), at the midpoint, so exactly one
             stop occurs (on the planted turn); alpha halfway between the
             planted turn's mean and the lowest clean mean.
  agentic    lambda at the 30th percentile of the pooled turn-level cumulative
  multi      values, alpha at the 5th percentile of the non-planted turn means
             (multi: per domain, over that domain's rollouts).
  reasoning  lambda at the 30th percentile of the pooled token-level cumulative
             values; alpha = -inf (the paper disables the gate for single-turn
             math, Sec. 4.2 and Appendix A).
  fused      lambda = 5.5 x the closed-form expected turn mean
             -(log V + d sigma_h^2 sigma_W^2 / 2); alpha = -inf.

A percentile rule takes the midpoint of the two sorted values straddling rank
floor(q (M - 1)), so lambda never equals an oracle value.
"""
from __future__ import annotations

import math

import numpy as np


def midpoint_quantile(values: np.ndarray, q: float) -> float:
    v = np.sort(np.asarray(values, np.float64)[np.isfinite(values)])
    if v.size < 2:
        raise ValueError("need at least two finite values")
    k = int(math.floor(q * (v.size - 1)))
    k = min(k, v.size - 2)
    return float(0.5 * (v[k] + v[k + 1]))


def pooled_cum(unit_off: np.ndarray, values: np.ndarray) -> np.ndarray:
    """C_u per rollout with K0 = 0, concatenated."""
    out = []
    for r in range(unit_off.size - 1):
        out.append(np.cumsum(values[unit_off[r]:unit_off[r + 1]]))
    return np.concatenate(out) if out else np.zeros(0)


def tiny_thresholds(turn_mean: np.ndarray, rollout_turn_off: np.ndarray, planted: np.ndarray):
    r0 = int(np.nonzero(planted >= 0)[0][0])
    k = int(planted[r0])
    t0 = int(rollout_turn_off[r0])
    c0 = np.cumsum(turn_mean[t0:int(rollout_turn_off[r0 + 1])])
    upper = [c0[k - 1]] if k > 0 else [0.0]
    for r in range(rollout_turn_off.size - 1):
        if r != r0:
            c = np.cumsum(turn_mean[int(rollout_turn_off[r]):int(rollout_turn_off[r + 1])])
            upper.append(c[-1])
    hi = min(upper)
    lo = c0[k]
    if not lo < hi - 2e-3:
        raise ValueError(f"no single-stop threshold: {lo} vs {hi}")
    lam = 0.5 * (lo + hi)
    planted_mean = turn_mean[t0 + k]
    clean = np.delete(turn_mean, t0 + k)
    alpha = 0.5 * (planted_mean + clean.min())
    return [float(lam)], [float(alpha)]


def agentic_thresholds(turn_mean: np.ndarray, rollout_turn_off: np.ndarray, planted: np.ndarray,
                       domain: np.ndarray | None, n_dom: int):
    R = rollout_turn_off.size - 1
    dom = np.zeros(R, np.int64) if domain is None else np.asarray(domain, np.int64)
    lam, alpha = [], []
    for d in range(n_dom):
        rs = np.nonzero(dom == d)[0]
        cums, clean = [], []
        for r in rs:
            a, b = int(rollout_turn_off[r]), int(rollout_turn_off[r + 1])
            cums.append(np.cumsum(turn_mean[a:b]))
            keep = np.ones(b - a, bool)
            if planted is not None and planted[r] >= 0:
                keep[planted[r]] = False
            clean.append(turn_mean[a:b][keep])
        lam.append(midpoint_quantile(np.concatenate(cums), 0.30))
        alpha.append(midpoint_quantile(np.concatenate(clean), 0.05))
    return lam, alpha


def reasoning_thresholds(logp_t: np.ndarray, tok_off_of_rollout: np.ndarray):
    return [midpoint_quantile(pooled_cum(tok_off_of_rollout, logp_t), 0.30)], [-math.inf]


def fused_thresholds(vocab: int, d: int, sigma_h: float, sigma_w: float):
    mean = -(math.log(vocab) + d * sigma_h ** 2 * sigma_w ** 2 / 2.0)
    return [5.5 * mean], [-math.inf]
