"""Temperature calibration of the synthetic workloads (test infrastructure).

The paper fixes no temperature; the workloads scale the logits by 1/tau, with
tau chosen from the seed so that a stated share of the masked positions of the
first step exceeds the calibration threshold. For one row of unscaled logits,
the top softmax probability f(tau) = 1 / sum_v exp((z_v - max z) / tau) never
increases with tau, so the largest tau at which it still exceeds gamma is found
by bisection in log(tau). The pooled per-position values are sorted and tau is
placed between the k-th and (k+1)-th largest, k = round(share * n), so exactly k
positions exceed gamma at that tau when the values are distinct.
"""
from __future__ import annotations

import numpy as np


def top_prob(z: np.ndarray, tau: float) -> float:
    z = np.asarray(z, np.float64)
    return 1.0 / np.exp((z - z.max()) / tau).sum()


def tau_star(z: np.ndarray, gamma: float, lo: float = 1e-4, hi: float = 1e4,
             iters: int = 100) -> float:
    """sup{tau in [lo, hi] : top_prob(z, tau) > gamma} by bisection in log tau."""
    if top_prob(z, lo) <= gamma:
        return lo
    if top_prob(z, hi) > gamma:
        return hi
    a, b = np.log(lo), np.log(hi)      # f(e^a) > gamma >= f(e^b)
    for _ in range(iters):
        m = 0.5 * (a + b)
        if top_prob(z, np.exp(m)) > gamma:
            a = m
        else:
            b = m
    return float(np.exp(a))


def calibrate(raw_logits: np.ndarray, gamma: float = 0.9, share: float = 0.3):
    """Return (tau, inv_tau as float32, achieved share, k, n).

    raw_logits: [n, V] unscaled logits of the pooled masked positions."""
    taus = np.array([tau_star(z, gamma) for z in raw_logits])
    order = np.sort(taus)[::-1]
    n = len(order)
    k = int(round(share * n))
    k = min(max(k, 1), n - 1)
    tau = float(np.sqrt(order[k - 1] * order[k]))
    inv_tau = np.float32(1.0 / tau)
    achieved = float(np.mean([top_prob(z * float(inv_tau), 1.0) > gamma for z in raw_logits]))
    return tau, inv_tau, achieved, k, n
