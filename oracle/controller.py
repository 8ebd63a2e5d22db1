"""CPU oracle of the confidence-threshold controller: SLO-aware threshold
selection and adaptive load control, without and with approximate KV caching.

TEST INFRASTRUCTURE. Only the tests may import this module; the controller
library (libdlmctl.so) shares no code with it.

What is computed (paper, "SLO-aware Confidence Threshold Adjustment",
Algorithm 1; "Adaptive Load Control", Algorithm 2; appendix "Algorithm for
Supporting Approximate KV Caching", Algorithms 5 and 6):

* the remaining time of a request under a threshold is its predicted
  remaining steps times the per-step latency of its instance at the
  instance's batch size (Alg. 1); with KV caching, remaining cache steps are
  priced at the latency of a batch of block-size x resident-requests tokens
  and remaining recompute steps at the latency of the instance's whole token
  count (Alg. 6);
* a request's threshold is the highest allowed candidate whose predicted
  remaining time fits its remaining SLO budget, else the lowest allowed one;
* a request's load is its predicted remaining steps times its token count
  (Alg. 2); with caching, cache steps count block-size tokens and recompute
  steps the whole request (Alg. 5);
* cluster capacity is, per instance, its best tokens-per-second over batch
  sizes times the SLO (Alg. 2); with caching, the throughput of a block made
  of block-size - 1 cache steps at the largest batch and one recompute step
  of an average request (Alg. 5);
* load control gives each request, in arrival order, the highest maximum
  threshold for which the worst-case aggregate load (earlier requests at
  their maxima, this one at the candidate, later ones at the lowest
  threshold) fits the capacity; the lowest threshold is always kept (Alg. 2).

Both choices are written from the prose of those sections as set
definitions (the highest fitting candidate, the largest feasible maximum),
not by transcribing the printed loops.

Readings (the paper gives the latency profile as a table over batch sizes):
the latency at a token count between measured points is linear between its
neighbours, flat below the first point and linear along the last segment
beyond the last point; cache-step latencies use the cache-step curve when one
was measured, else the single curve. Capacity's maximum over batch sizes is
taken over the measured points.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Sequence


@dataclass
class Curve:
    tokens: Sequence[float]      # ascending
    latency_s: Sequence[float]


@dataclass
class Profile:
    recompute: Curve
    cache: Optional[Curve] = None


@dataclass
class Params:
    gammas: Sequence[float]      # candidate thresholds, ascending
    cache_block: int = 0         # 0: no KV caching (Alg. 1 and 2)
    max_seqs_per_batch: int = 1
    slo_s: float = 1.0


@dataclass
class Req:
    num_tokens: float
    pred_steps_left: Sequence[float]     # per candidate threshold (ascending order)
    slo_left_s: float = 0.0
    recomp_steps_left: float = 0.0
    allowed: List[int] = field(default_factory=list)   # candidate indices
    gamma_idx: int = -1


@dataclass
class Instance:
    profile: Profile
    num_tokens: float            # tokens of the batch it runs
    num_reqs: int


def latency(curve: Curve, tokens: float) -> float:
    t, y = list(curve.tokens), list(curve.latency_s)
    if len(t) == 1 or tokens <= t[0]:
        return float(y[0])
    for i in range(1, len(t)):
        if tokens <= t[i]:
            w = (tokens - t[i - 1]) / (t[i] - t[i - 1])
            return float(y[i - 1] + w * (y[i] - y[i - 1]))
    w = (tokens - t[-2]) / (t[-1] - t[-2])
    return float(y[-2] + w * (y[-1] - y[-2]))


def predicted_time_left(p: Params, inst: Instance, req: Req, gi: int) -> float:
    steps = req.pred_steps_left[gi]
    if p.cache_block == 0:                                   # Alg. 1
        return steps * latency(inst.profile.recompute, inst.num_tokens)
    cache_left = steps - req.recomp_steps_left               # Alg. 6
    cache_curve = inst.profile.cache or inst.profile.recompute
    cache_lat = latency(cache_curve, p.cache_block * inst.num_reqs)
    recomp_lat = latency(inst.profile.recompute, inst.num_tokens)
    return cache_left * cache_lat + req.recomp_steps_left * recomp_lat


def update_conf_threshold(p: Params, inst: Instance, req: Req) -> int:
    """The threshold choice of "SLO-aware Confidence Threshold Adjustment":
    among the allowed candidates, the highest one whose predicted remaining
    time fits the request's remaining SLO budget; when none fits, the lowest
    allowed one (the paper's loop over the allowed candidates from the top
    ends there)."""
    fits = [gi for gi in req.allowed if predicted_time_left(p, inst, req, gi) <= req.slo_left_s]
    req.gamma_idx = max(fits) if fits else min(req.allowed)
    return req.gamma_idx


def req_load(p: Params, req: Req, gi: int) -> float:
    steps = req.pred_steps_left[gi]
    if p.cache_block == 0:                                   # Alg. 2
        return steps * req.num_tokens
    cache_steps = steps - req.recomp_steps_left              # Alg. 5
    return cache_steps * p.cache_block + req.recomp_steps_left * req.num_tokens


def cluster_capacity(p: Params, profiles: Sequence[Profile], tokens_per_req: float) -> float:
    total = 0.0
    for prof in profiles:
        if p.cache_block == 0:                               # Alg. 2
            c = prof.recompute
            best = max(b / l for b, l in zip(c.tokens, c.latency_s))
            total += best * p.slo_s
        else:                                                # Alg. 5
            load = p.cache_block * p.max_seqs_per_batch
            cache_lat = latency(prof.cache or prof.recompute, load)
            recomp_lat = latency(prof.recompute, tokens_per_req)
            nb = p.cache_block - 1
            tput = (load * nb + tokens_per_req) / (cache_lat * nb + recomp_lat)
            total += tput * p.slo_s
    return total


def update_allowed(p: Params, reqs: List[Req], capacity: float) -> None:
    """Load control of "Adaptive Load Control", requests in arrival order (the
    list order): each request gets the highest maximum threshold for which
    the worst-case aggregate load fits the capacity, the worst case being
    every earlier request at the maximum it was given, this request at the
    candidate and every later request at the lowest threshold. The lowest
    threshold stays allowed even when it does not fit. A request's allowed
    set is every candidate up to its maximum."""
    maxima: List[int] = []
    for i, req in enumerate(reqs):
        earlier = sum(req_load(p, reqs[j], maxima[j]) for j in range(i))
        later = sum(req_load(p, reqs[j], 0) for j in range(i + 1, len(reqs)))
        fits = [gi for gi in range(len(p.gammas))
                if earlier + req_load(p, req, gi) + later <= capacity]
        top = max(fits) if fits else 0
        maxima.append(top)
        req.allowed = list(range(top + 1))
