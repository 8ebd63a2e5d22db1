"""Host logic of the single-GPU serving loop (continuous batching with
admission and eviction only at recompute steps, per-request thresholds from
the controller library), driven by a stand-in engine on the CPU: the engine's
block bookkeeping is the real one (engine.advance), its unmasking is a
deterministic function of the threshold, and its step latency comes from a
latency profile through a virtual clock. No GPU."""
import math
import os

import numpy as np
import pytest

from paper_2606_29094_amd import controller as ctl
from paper_2606_29094_amd import engine, serving
from paper_2606_29094_amd.profiling import StepTable

PROFILE = {"recompute": {"tokens": [256, 1024, 4096, 16384],
                         "latency_s": [0.008, 0.017, 0.065, 0.276]},
           "cache": {"tokens": [32, 256, 2048], "latency_s": [0.0067, 0.0086, 0.039]}}
GAMMAS = [0.5, 0.7, 0.9]
TABLE = StepTable(GAMMAS, [3.7, 6.8, 16.6], 32)


@pytest.fixture(scope="module", autouse=True)
def built():
    if not os.path.exists(ctl.LIB_PATH):
        pytest.skip("libdlmctl.so not built")


class FakeEngine:
    """admit / release / step / save_state / restore_state with the real
    Request bookkeeping; a step unmasks a threshold-dependent number of the
    block's masked positions and advances the virtual clock by the profile's
    latency for the step's recomputed tokens."""

    def __init__(self, n_slots, mode):
        self.n_slots, self.mode = n_slots, mode
        self.free = list(range(n_slots))[::-1]
        self.t = 0.0
        self.log = []                       # (event, rid-ish, details)
        self.states = {}

    def clock(self):
        return self.t

    def admit(self, r, mask_id):
        assert self.free, "admitted without a free slot"
        r.slot = self.free.pop()
        r.k, r.masked_in_block, r.refreshed_block = 0, r.block_len, -1
        self.log.append(("admit", id(r)))

    def release(self, r):
        self.free.append(r.slot)
        r.slot = -1

    def save_state(self, r):
        # eviction is only allowed when the next step recomputes anyway
        assert self.mode == "none" or r.refreshed_block != r.block_start
        self.log.append(("evict", id(r)))
        return ("state", r.k, r.masked_in_block, r.steps, r.unmasked)

    def restore_state(self, r, st):
        _, r.k, r.masked_in_block, r.steps, r.unmasked = st

    def step(self, reqs):
        tokens = 0
        for r in reqs:
            assert r.slot >= 0
            refresh = self.mode == "none" or r.refreshed_block != r.block_start
            if refresh:
                tokens += r.seq_len
                r.refreshed_block = r.block_start
            else:
                tokens += r.block_len if self.mode == "dual" else r.seq_len - r.block_start
            self.log.append(("step", id(r), refresh, r.threshold))
        kind = "recompute" if tokens > 64 * len(reqs) else "cache"
        c = ctl.make_curve(PROFILE[kind]["tokens"], PROFILE[kind]["latency_s"])
        self.t += ctl.latency(c, tokens)
        self.log.append(("batch", tokens, len(reqs)))
        for r in reqs:
            n = max(1, int(round((1.0 - r.threshold) * 0.4 * r.block_len)))
            engine.advance(r, min(n, r.masked_in_block))


def _serve(rate, n, slo, mode="dual", slots=8, budget=8192, gammas=GAMMAS, seed=0):
    eng = FakeEngine(slots, mode)
    cfg = serving.ServeConfig(gammas, 32, mode, budget)
    srv = serving.Server(eng, cfg, PROFILE, StepTable(gammas, TABLE.steps_per_block, 32), 2047,
                         clock=eng.clock)
    trace = serving.poisson_trace(rate, n, seed, (128, 1024), (128, 256), slo, 2048)
    rep = srv.run(trace)
    return eng, trace, rep


@pytest.mark.parametrize("mode", ["dual", "prefix", "none"])
def test_every_request_completes(mode):
    eng, trace, rep = _serve(4.0, 40, 5.0, mode)
    assert rep["completed"] == len(trace)
    for a in trace:
        assert a.req.done and a.req.unmasked == a.gen_len
        assert set(a.gammas) <= set(GAMMAS)


def test_admission_and_eviction_only_at_recompute_steps():
    eng, trace, rep = _serve(20.0, 60, 3.0, "dual", slots=4, budget=3000)
    assert rep["completed"] == len(trace)
    # after every admit, the request's next step is a recompute step
    expect_refresh = set()
    for ev in eng.log:
        if ev[0] == "admit":
            expect_refresh.add(ev[1])
        elif ev[0] == "step" and ev[1] in expect_refresh:
            assert ev[2], "first step after admission must recompute"
            expect_refresh.discard(ev[1])
    assert rep["evictions"] == sum(1 for ev in eng.log if ev[0] == "evict")


def test_step_token_budget():
    eng, trace, rep = _serve(10.0, 50, 4.0, "dual", slots=8, budget=4096)
    for ev in eng.log:
        if ev[0] == "batch":
            tokens, n = ev[1], ev[2]
            assert tokens <= 4096 or n == 1


def test_threshold_follows_the_budget():
    _, _, loose = _serve(0.5, 20, 1e6)
    _, _, tight = _serve(0.5, 20, 0.05)
    assert loose["mean_threshold"] == pytest.approx(max(GAMMAS), abs=1e-12)
    assert tight["mean_threshold"] == pytest.approx(min(GAMMAS), abs=1e-12)
    assert loose["slo_attainment"] == 1.0


def test_load_control_lowers_thresholds_under_load():
    _, _, light = _serve(0.5, 30, 4.0)
    _, _, heavy = _serve(50.0, 30, 4.0)
    assert heavy["mean_threshold"] < light["mean_threshold"]


def test_eviction_hands_the_slot_to_a_more_urgent_request():
    """Two slots, a step budget for one 1200-token recompute, no caching (every
    step recomputes): the resident request that is deferred is evicted when a
    request with less slack waits, and resumes later from its saved state."""
    eng = FakeEngine(2, "none")
    cfg = serving.ServeConfig(GAMMAS, 32, "none", 1300)
    srv = serving.Server(eng, cfg, PROFILE, TABLE, 2047, clock=eng.clock)
    rng = np.random.default_rng(3)
    mk = lambda rid, t, slo: serving.Arrival(rid, t, rng.integers(0, 2047, 1072), 128, slo)
    trace = [mk(0, 0.0, 1e4), mk(1, 0.0, 1e4), mk(2, 0.05, 3.0)]
    rep = srv.run(trace)
    assert rep["completed"] == 3 and rep["evictions"] >= 1 and rep["deferred"] >= 1
    assert max(a.evictions for a in trace[:2]) >= 1 and trace[2].evictions == 0
    for a in trace:
        assert a.req.unmasked == a.gen_len
