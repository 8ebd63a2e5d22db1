"""CPU oracle of the per-request confidence statistics (the Step Predictor's
confidence and progress features).

TEST INFRASTRUCTURE. Only the tests, the smoke check and the benchmark's CPU
baseline may import this module; the product path never does.

What is computed (paper, "Step Prediction" and the appendix "Step Predictor
Features"): the predictor of remaining denoising steps reads, besides the
threshold and the output length, four progress fractions and five statistics
of the confidences of the request's output tokens - the minimum, the lower
quartile, the median, the mean and the upper quartile.

Readings (the paper does not define them further):

* the output tokens are the generation positions [prompt_len, seq_len) that
  are unmasked; the confidence of such a token is the confidence with which it
  was unmasked (its softmax probability at that step);
* quartiles and the median interpolate linearly between order statistics:
  with the n values sorted ascending as v[0..n-1], the p-quantile is
  v[j] + (h - j) (v[j+1] - v[j]) with h = (n - 1) p and j = floor(h)
  (v[j+1] read as v[j] when j = n - 1);
* with no unmasked output token every statistic is 0.

Statistic vector (the order of the library's output): count, min, q25,
median, mean, q75, max, unmasked positions of the active block.
"""
from __future__ import annotations

import math

import numpy as np

N_STATS = 8


def quantile_sorted(v: np.ndarray, p: float) -> float:
    """Linear-interpolation p-quantile of an ascending array (n >= 1)."""
    n = len(v)
    h = (n - 1) * p
    j = int(math.floor(h))
    nxt = v[j + 1] if j + 1 < n else v[j]
    return float(v[j]) + (h - j) * (float(nxt) - float(v[j]))


def confidence_stats(tok_conf: np.ndarray, mask: np.ndarray, prompt_len: int,
                     block_start: int, block_len: int) -> np.ndarray:
    """Statistics of one request after a step.

    tok_conf, mask: the request's positions [0, seq_len) (mask 1 = [MASK]);
    returns float64 [N_STATS]."""
    seq_len = len(mask)
    out = np.zeros(N_STATS)
    pos = np.arange(prompt_len, seq_len)
    vals = np.asarray(tok_conf, dtype=np.float64)[pos[mask[pos] == 0]]
    n = len(vals)
    out[0] = n
    if n > 0:
        v = np.sort(vals)
        out[1] = v[0]
        out[2] = quantile_sorted(v, 0.25)
        out[3] = quantile_sorted(v, 0.5)
        out[4] = math.fsum(v) / n
        out[5] = quantile_sorted(v, 0.75)
        out[6] = v[-1]
    blk = mask[block_start:block_start + block_len]
    out[7] = int(np.sum(blk == 0))
    return out


def predictor_features(gamma: float, gen_len: int, steps_done: int, block_index: int,
                       n_blocks: int, block_len: int, stats: np.ndarray) -> dict:
    """The eleven features of the appendix, from a statistic vector."""
    return {
        "confidence_threshold": gamma,
        "output_length": gen_len,
        "full_progress": steps_done / gen_len,
        "full_unmask_progress": stats[0] / gen_len,
        "block_progress": block_index / n_blocks,
        "block_unmask_progress": stats[7] / block_len,
        "output_min_confidence": stats[1],
        "output_q25_confidence": stats[2],
        "output_median_confidence": stats[3],
        "output_avg_confidence": stats[4],
        "output_q75_confidence": stats[5],
    }
