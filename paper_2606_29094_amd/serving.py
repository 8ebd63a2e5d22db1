"""Single-GPU continuous batching with per-request dynamic thresholds.

The serving loop of one model instance (paper, "Request Scheduling",
Algorithm 3, reduced to one instance; "Dynamic Confidence Threshold
Adjustment and Scheduling"; "Supporting Approximate KV Caching", migration
granularity):

* every scheduling event (one per denoising step) considers the arrived
  requests that are not resident and the resident ones that just finished a
  step; a request's load for the next step is the tokens that step
  recomputes (the block for a cache step, the whole sequence for a recompute
  step), and a step runs at most `max_step_tokens` of them (Alg. 3's
  inst.batchSize + nTok <= inst.maxBatchSize);
* admission happens only at recompute steps (a new request's first step
  recomputes its whole sequence) and so does eviction: a request can leave
  the batch only when its next step is a recompute step, where its cache has
  to be rebuilt anyway, carrying only its tokens, mask and token confidences;
* cache steps of resident requests always run; recompute steps are granted
  in order of SLO slack (remaining budget minus predicted remaining time),
  and a resident request whose recompute step does not fit is evicted when a
  request with less slack is waiting for a slot;
* before each step the controller library sets every request's threshold:
  adaptive load control over all requests in arrival order (Alg. 2 / Alg. 5)
  every `control_every` steps, then the SLO-aware choice within the allowed
  set (Alg. 1 / Alg. 6), with remaining steps from the measured step table
  and step latencies from the measured latency profile.

Time is the GPU's: the clock advances by each step's measured wall time, and a
request arrives when the clock passes its arrival time (idle gaps jump to the
next arrival).
"""
from __future__ import annotations

import math
import time
from dataclasses import dataclass, field
from typing import Callable, Dict, List, Optional, Sequence

import numpy as np

from . import controller as ctl
from .engine import Request
from .profiling import StepTable


@dataclass
class Arrival:
    rid: int
    arrival_s: float
    prompt: np.ndarray
    gen_len: int
    slo_s: float
    # filled while serving
    req: Optional[Request] = None
    saved: Optional[tuple] = None
    first_step_s: Optional[float] = None
    finish_s: Optional[float] = None
    evictions: int = 0
    gammas: List[float] = field(default_factory=list)

    @property
    def seq_len(self):
        return len(self.prompt) + self.gen_len


@dataclass
class ServeConfig:
    gammas: Sequence[float]              # candidate thresholds, ascending
    block: int
    mode: str                            # "dual", "prefix" or "none"
    max_step_tokens: int
    control_every: int = 4


class Server:
    def __init__(self, eng, cfg: ServeConfig, profile: dict, table: StepTable, mask_id: int,
                 clock: Optional[Callable[[], float]] = None):
        """eng: an engine.Engine (or an object with the same admit / release /
        step / save_state / restore_state); profile: a measured latency
        profile ({"recompute": {...}, "cache": {...}})."""
        self.eng, self.cfg, self.table, self.mask_id = eng, cfg, table, mask_id
        self.gammas = list(cfg.gammas)
        rc, cc = profile["recompute"], profile.get("cache")
        self.profile = ctl.make_profile((rc["tokens"], rc["latency_s"]),
                                        (cc["tokens"], cc["latency_s"]) if cc else None)
        self.cache_block = 0 if cfg.mode == "none" else cfg.block
        self.clock = clock or time.perf_counter
        self.n_slots = eng.n_slots
        self.stats = {"steps": 0, "evictions": 0, "deferred": 0, "control_runs": 0,
                      "control_s": 0.0}

    # ---- controller inputs
    def _is_cache_step(self, a: Arrival) -> bool:
        """Resident, and its next step reads the cache of its last recompute."""
        r = a.req
        return (r is not None and r.slot >= 0 and self.cfg.mode != "none"
                and r.refreshed_block == r.block_start)

    def _next_tokens(self, a: Arrival) -> int:
        if not self._is_cache_step(a):
            return a.seq_len
        r = a.req
        return r.block_len if self.cfg.mode == "dual" else a.seq_len - r.block_start

    def _shadow(self, a: Arrival) -> Request:
        """The request's progress (a fresh one before its first admission)."""
        if a.req is not None:
            return a.req
        return Request(a.prompt, a.gen_len, self.cfg.block, self.gammas[-1],
                       masked_in_block=min(self.cfg.block, a.gen_len))

    def _ctl_req(self, a: Arrival, now: float, slo_s: float) -> ctl.Req:
        r = self._shadow(a)
        steps = self.table.pred_steps_left(r)
        recomp = min(self.table.recomp_steps_left(r, self.cfg.mode), min(steps)) \
            if self.cache_block else 0.0
        return ctl.make_req(a.seq_len, steps, slo_s - (now - a.arrival_s), recomp)

    def _control(self, active: List[Arrival], resident: List[Arrival], now: float,
                 run_alg2: bool) -> None:
        t0 = time.perf_counter()
        slo = max(a.slo_s for a in active)
        P = ctl.make_params(self.gammas, self.cache_block, self.n_slots, slo)
        reqs = [self._ctl_req(a, now, a.slo_s) for a in active]
        if run_alg2:
            tpr = float(np.mean([a.seq_len for a in active]))
            cap = ctl.capacity(P, [self.profile], tpr)
            ctl.update_allowed(P, reqs, cap)
            for a, q in zip(active, reqs):
                a._allowed = q.allowed
            self.stats["control_runs"] += 1
        n_tok = float(sum(a.seq_len for a in resident)) or float(active[0].seq_len)
        inst = ctl.make_instance(self.profile, n_tok, max(len(resident), 1))
        full = (1 << len(self.gammas)) - 1
        for a, q in zip(active, reqs):
            q.allowed = getattr(a, "_allowed", full)
            a._gamma_idx = ctl.update_threshold(P, inst, q)
            a._slack = q.slo_left_s - ctl.predicted_time_left(P, inst, q, a._gamma_idx)
        self.stats["control_s"] += time.perf_counter() - t0

    # ---- the loop
    def run(self, trace: List[Arrival], max_steps: int = 1 << 30) -> Dict:
        pending = sorted(trace, key=lambda a: a.arrival_s)
        queue: List[Arrival] = []          # arrived, not resident
        resident: List[Arrival] = []
        done: List[Arrival] = []
        now = 0.0
        steps = 0
        while (pending or queue or resident) and steps < max_steps:
            while pending and pending[0].arrival_s <= now:
                queue.append(pending.pop(0))
            if not queue and not resident:
                now = pending[0].arrival_s
                continue
            t_iter = self.clock()
            active = sorted(resident + queue, key=lambda a: a.arrival_s)
            self._control(active, resident, now, steps % self.cfg.control_every == 0)
            # cache steps of resident requests always run
            batch = [a for a in resident if self._is_cache_step(a)]
            budget = self.cfg.max_step_tokens - sum(self._next_tokens(a) for a in batch)
            # recompute steps (resident at a block boundary, or waiting) by slack
            want = sorted([a for a in resident if a not in batch] + queue, key=lambda a: a._slack)
            free = self.n_slots - len(resident)
            deferred: List[Arrival] = []
            for a in want:
                need = a.seq_len
                is_res = a in resident
                if need <= budget and (is_res or free > 0):
                    if not is_res:
                        self._admit(a)
                        resident.append(a)
                        queue.remove(a)
                        free -= 1
                    batch.append(a)
                    budget -= need
                elif is_res:
                    deferred.append(a)
            self.stats["deferred"] += len(deferred)
            # evict a deferred resident (its next step is a recompute) when a
            # waiting request with less slack has no slot
            waiting = [a for a in queue if a.arrival_s <= now]
            for a in sorted(deferred, key=lambda a: -a._slack):
                if free > 0 or not waiting:
                    break
                w = min(waiting, key=lambda x: x._slack)
                if w._slack < a._slack:
                    a.saved = self.eng.save_state(a.req)
                    self.eng.release(a.req)
                    resident.remove(a)
                    queue.append(a)
                    a.evictions += 1
                    self.stats["evictions"] += 1
                    free += 1
                    waiting.remove(w)
            if not batch:
                # nothing fits (a request longer than the step budget): run it alone
                a = min(resident + queue, key=lambda a: a._slack)
                if a not in resident:
                    self._admit(a)
                    resident.append(a)
                    queue.remove(a)
                batch = [a]
            for a in batch:
                a.req.threshold = self.gammas[a._gamma_idx]
                a.gammas.append(a.req.threshold)
                if a.first_step_s is None:
                    a.first_step_s = now
            self.eng.step([a.req for a in batch])
            now += self.clock() - t_iter          # controller, scheduling and the step
            steps += 1
            for a in batch:
                if a.req.done:
                    a.finish_s = now
                    self.eng.release(a.req)
                    resident.remove(a)
                    done.append(a)
        self.stats["steps"] = steps
        return self.report(done, trace, now)

    def _admit(self, a: Arrival) -> None:
        if a.req is None:
            a.req = Request(a.prompt, a.gen_len, self.cfg.block, self.gammas[-1])
        self.eng.admit(a.req, self.mask_id)
        if a.saved is not None:
            self.eng.restore_state(a.req, a.saved)
            a.saved = None

    def report(self, done: List[Arrival], trace: List[Arrival], end_s: float) -> Dict:
        lat = np.array([a.finish_s - a.arrival_s for a in done]) if done else np.zeros(1)
        ok = [a for a in done if a.finish_s - a.arrival_s <= a.slo_s]
        gam = [g for a in done for g in a.gammas]
        toks = sum(a.gen_len for a in done)
        return {
            "requests": len(trace), "completed": len(done),
            "slo_attainment": len(ok) / max(len(trace), 1),
            "latency_mean_s": float(lat.mean()), "latency_p50_s": float(np.median(lat)),
            "latency_p99_s": float(np.percentile(lat, 99)),
            "tokens_per_s": toks / end_s if end_s > 0 else 0.0,
            "mean_threshold": float(np.mean(gam)) if gam else None,
            "duration_s": end_s, **self.stats,
        }


def poisson_trace(rate_per_s: float, n: int, seed: int, prompt_range, gen_choices, slo_s: float,
                  vocab: int) -> List[Arrival]:
    """Synthetic arrivals: exponential gaps, uniform prompt lengths in
    prompt_range, output lengths drawn from gen_choices, uniform tokens."""
    rng = np.random.default_rng(seed)
    t = 0.0
    out = []
    for i in range(n):
        t += rng.exponential(1.0 / rate_per_s)
        P = int(rng.integers(prompt_range[0], prompt_range[1] + 1))
        G = int(rng.choice(gen_choices))
        out.append(Arrival(i, t, rng.integers(0, vocab - 1, P), G, slo_s))
    return out
