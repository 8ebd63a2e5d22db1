"""Randomised batches of the denoising step on the GPU against the oracle
(tiny fp32 model; "Background and Challenges" for the step and the unmask
rule, "Support for Approximate Caching" for the prefix and dual caches):
seeded mixes of 3-10 requests with prompts of 1-150 tokens, blocks of 8-64
with ragged last blocks, thresholds from 0.5 to 1 and each cache mode, run to
completion in one engine. Every step is teacher-forced: each request's
tokens, mask and block are set to the oracle's before the step, so refresh
and cache steps of different requests mix in one launch as the blocks of the
requests end at different steps, and each request's confidences and
decisions are compared with its own oracle step."""
import json
import os

import numpy as np
import pytest

import oracle
import synth
from helpers import device_model, host_weights
from paper_2606_29094_amd import engine
from test_gpu_edges import _check, _prompt

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "tiny_fp32.json")
CASES = [(mode, seed) for mode in ("none", "prefix", "dual") for seed in (11, 12)]


@pytest.fixture(scope="module")
def tiny(gpu):
    g = json.load(open(GOLDEN))
    cfg = synth.TINY_FP32
    model, t = device_model(cfg, g["inv_tau"])
    W = host_weights(t, cfg)
    yield cfg, model, W, g["inv_tau"]
    model.close()


@pytest.mark.parametrize("mode,seed", CASES, ids=lambda v: str(v))
def test_random_batch_to_completion(tiny, mode, seed):
    cfg, model, W, inv_tau = tiny
    rng = np.random.default_rng(seed)
    R = int(rng.integers(3, 11))
    spec = []
    for i in range(R):
        b = int(rng.choice([8, 16, 32, 64]))
        P = int(rng.integers(1, 151))
        nb = 3 if i < 2 else int(rng.integers(1, 4))      # the first two: several blocks
        G = nb * b - int(rng.integers(0, b // 2 + 1))       # ragged last block
        # high thresholds keep blocks open for several steps, low ones close them fast
        gam = float(rng.choice([0.9, 0.95, 1.0] if i % 2 == 0 else [0.5, 0.8, 0.9]))
        spec.append((P, max(G, 1), b, gam))
    L = max(P + G for P, G, _, _ in spec)
    eng = engine.Engine(model, R, L, mode)
    reqs, oreqs = [], []
    for i, (P, G, b, gam) in enumerate(spec):
        prompt = _prompt(cfg, P, 1000 * seed + i)
        r = engine.Request(prompt, G, b, gam)
        eng.admit(r, cfg.mask_id)
        reqs.append(r)
        oreqs.append(oracle.Request.new(prompt, G, b, gam, cfg.mask_id))
    steps = refresh_mixed = 0
    while not all(o.done for o in oreqs):
        live = [j for j, o in enumerate(oreqs) if not o.done]
        for j in live:
            eng.set_state(reqs[j], oreqs[j].tokens, oreqs[j].mask, oreqs[j].k)
        act = [reqs[j] for j in live]
        starts = [r.block_start for r in act]
        kinds = {r.refreshed_block != r.block_start for r in act}
        refresh_mixed += int(len(kinds) == 2)
        eng.step(act)
        out = eng.read_outputs(len(act))
        for i, j in enumerate(live):
            res = oracle.denoise_step(cfg, W, oreqs[j], mode, inv_tau, keep_logits=True)
            _check(res, {k: v[i] for k, v in out.items()}, starts[i], reqs[j].threshold)
        steps += 1
        assert steps < 400
    eng.close()
    if mode != "none":
        assert refresh_mixed > 0, "no step mixed refresh and cache requests"
