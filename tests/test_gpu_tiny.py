"""GPU parity of the tiny fp32 model (2 layers, d=256, V=2048) against the
oracle, through the C ABI: step logits, confidences, unmask decisions and the
whole generation, teacher-forced step by step, plus the stored trajectory."""
import copy
import json
import os

import numpy as np
import pytest
import torch

import oracle
import synth
from helpers import CONF_TOL, LOGIT_TOL, device_model, host_weights, logit_err, top2_gap
from paper_2606_29094_amd import dlm, engine

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "tiny_fp32.json")


@pytest.fixture(scope="module")
def tiny(gpu):
    g = json.load(open(GOLDEN))
    cfg = synth.TINY_FP32
    model, t = device_model(cfg, g["inv_tau"])
    W = host_weights(t, cfg)
    return cfg, model, W, g


def _engine(model, mode, n_slots=1, seq=128):
    return engine.Engine(model, n_slots, seq, mode)


def test_device_weights_equal_host_generator(tiny):
    cfg, model, W, g = tiny
    host = synth.model_weights(cfg)
    for l in range(cfg.n_layers):
        for k in ("wq", "wk", "wv", "wo", "wg", "wu", "wd"):
            assert np.array_equal(W.layer(l)[k], host["layers"][l][k]), (l, k)
    assert np.array_equal(W.globals["embed"], host["embed"])
    assert np.array_equal(W.globals["lm_head"], host["lm_head"])


def test_step1_logits_match_oracle(tiny):
    cfg, model, W, g = tiny
    prompt, G, thr = synth.request(synth.C1, 0)
    eng = _engine(model, "none")
    r = engine.Request(prompt, G, 32, thr)
    eng.admit(r, cfg.mask_id)
    z = eng.debug_logits([r]).cpu().numpy()
    oreq = oracle.Request.new(prompt, G, 32, thr, cfg.mask_id)
    h, rows, _ = oracle.step_forward(cfg, W, oreq, "none")
    s, e = oreq.block_bounds
    z_ref = oracle.head_logits(cfg, W, h[s:e], g["inv_tau"])
    err = logit_err(z, z_ref)
    print("tiny step-1 logits max rel err", err)
    assert err < LOGIT_TOL["f32"]


def _compare_step(res, out_r, blk_start, gamma, logits_tol_gap=1e-4):
    """Compare one request's GPU step outputs with the oracle StepResult."""
    A = res.masked_positions
    bc = out_r["block_conf"][A - blk_start]
    bt = out_r["block_tok"][A - blk_start]
    assert np.all(np.abs(bc - res.masked_conf) <= CONF_TOL), np.abs(bc - res.masked_conf).max()
    n = int(out_r["n"])
    got = set(out_r["pos"][:n].tolist())
    want = set(res.positions.tolist())
    near = set(A[np.abs(res.masked_conf - gamma) <= CONF_TOL].tolist())
    forced = not np.any(res.masked_conf > gamma)
    if forced:
        # nothing passes: exactly one position is unmasked, the most confident
        # one; when the top confidences are within the tolerance, any of the
        # tied top positions
        assert n == 1, (n, sorted(got))
        c = np.sort(res.masked_conf)[::-1]
        if len(c) > 1 and c[0] - c[1] <= CONF_TOL:
            tied = set(A[res.masked_conf >= c[0] - 2 * CONF_TOL].tolist())
            assert got <= tied, (sorted(got), sorted(tied))
            return 1
        assert got == want
        return 0
    assert (got ^ want) <= near, (got, want)
    # tokens of agreeing positions
    for p, t in zip(out_r["pos"][:n], out_r["tok"][:n]):
        if p in want:
            assert t == res.tokens[list(res.positions).index(p)]
    return len(got ^ want)


def test_trajectory_teacher_forced_and_golden(tiny):
    cfg, model, W, g = tiny
    prompt, G, thr = synth.request(synth.C1, 0)
    eng = _engine(model, "none")
    r = engine.Request(prompt, G, 32, thr)
    eng.admit(r, cfg.mask_id)
    oreq = oracle.Request.new(prompt, G, 32, thr, cfg.mask_id)
    exempt = 0
    steps = 0
    while not oreq.done:
        eng.set_state(r, oreq.tokens, oreq.mask, oreq.k)
        blk_start = r.block_start
        eng.step([r])
        out = eng.read_outputs(1)
        res = oracle.denoise_step(cfg, W, oreq, "none", g["inv_tau"])
        gold = g["steps"][steps]
        assert gold["positions"] == res.positions.tolist()
        exempt += _compare_step(res, {k: v[0] for k, v in out.items()}, blk_start, thr)
        steps += 1
    assert steps == g["n_steps"]
    assert oreq.tokens.tolist() == g["final_tokens"]
    print("tiny trajectory steps", steps, "tied-top forced steps", exempt)


def test_free_running_generation_matches_golden(tiny):
    cfg, model, W, g = tiny
    prompt, G, thr = synth.request(synth.C1, 0)
    eng = _engine(model, "none")
    r = engine.Request(prompt, G, 32, thr)
    eng.admit(r, cfg.mask_id)
    n = 0
    while not r.done:
        eng.step([r])
        n += 1
        assert n <= G
    toks, mask = eng.read_state(r)
    assert not mask.any()
    print("free-running: steps", n, "golden", g["n_steps"])
    # the stored trajectory's decisions are all outside the 1e-3 bands except
    # forced steps among tied top confidences, where the GPU and the oracle
    # pick the same position (checked step by step in the teacher-forced
    # test), so the free-running generation is the stored one
    assert n == g["n_steps"]
    assert toks.tolist() == g["final_tokens"]


def test_step_is_deterministic(tiny):
    cfg, model, W, g = tiny
    prompt, G, thr = synth.request(synth.C1, 0)
    outs = []
    for _ in range(2):
        eng = _engine(model, "none")
        r = engine.Request(prompt, G, 32, thr)
        eng.admit(r, cfg.mask_id)
        eng.step([r])
        o = eng.read_outputs(1)
        outs.append((o["block_conf"].copy(), o["pos"].copy(), eng.read_state(r)[0]))
    assert np.array_equal(outs[0][0], outs[1][0])
    assert np.array_equal(outs[0][1], outs[1][1])
    assert np.array_equal(outs[0][2], outs[1][2])


@pytest.mark.parametrize("mode", ["dual", "prefix"])
def test_cache_modes_teacher_forced(tiny, mode):
    """Cache modes: every step (recompute and cache steps) against the oracle
    run in the same mode from the same state."""
    cfg, model, W, g = tiny
    prompt, G, thr = synth.request(synth.C1, 0)
    eng = _engine(model, mode)
    r = engine.Request(prompt, G, 32, thr)
    eng.admit(r, cfg.mask_id)
    oreq = oracle.Request.new(prompt, G, 32, thr, cfg.mask_id)
    kinds = []
    while not oreq.done:
        # the GPU runs from the oracle's state; refresh follows the block protocol
        eng.set_state(r, oreq.tokens, oreq.mask, oreq.k)
        blk_start = r.block_start
        refresh_gpu = r.refreshed_block != blk_start
        eng.step([r])
        out = eng.read_outputs(1)
        res = oracle.denoise_step(cfg, W, oreq, mode, g["inv_tau"])
        assert res.refresh == refresh_gpu
        kinds.append(res.refresh)
        _compare_step(res, {k: v[0] for k, v in out.items()}, blk_start, thr)
    assert kinds[0] and not all(kinds)


def test_profiler_sampling_counts(tiny):
    """Kernel timing with sampling: every launch of the selected class is
    counted, one in `every` is timed (events carried by the kernel's dispatch),
    and the timed durations are positive."""
    cfg, model, W, g = tiny
    prompt, G, thr = synth.request(synth.C1, 0)
    eng = _engine(model, "none")
    r = engine.Request(prompt, G, 32, thr)
    eng.admit(r, cfg.mask_id)
    dlm.profile_sample(model.handle, 3)
    dlm.profile_enable(model.handle, True, "gemm_qkv")
    n_steps = 0
    while n_steps < 4 and not r.done:
        eng.step([r])
        n_steps += 1
    dlm.profile_enable(model.handle, False)
    prof = dlm.profile_read(model.handle)
    dlm.profile_sample(model.handle, 1)
    launches = n_steps * cfg.n_layers
    calls, ms, seen = prof["gemm_qkv"]
    assert seen == launches and calls == (launches + 2) // 3
    assert ms > 0 and set(prof) == {"gemm_qkv"}
    assert dlm.profile_read(model.handle) == {}
