"""Edge cases of the denoising step on the GPU, through the C ABI, against the
oracle (tiny fp32 model): the threshold extremes (1: exactly the most
confident position per step; 0: the whole masked block at once), an active
block with nothing masked, the largest batch (64 requests of mixed lengths in
one step), blocks of 64 with a ragged last block, and a long sequence."""
import json
import os

import numpy as np
import pytest

import oracle
import synth
from helpers import CONF_TOL, device_model, host_weights, top2_gap
from paper_2606_29094_amd import dlm, engine

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "tiny_fp32.json")


@pytest.fixture(scope="module")
def tiny(gpu):
    g = json.load(open(GOLDEN))
    cfg = synth.TINY_FP32
    model, t = device_model(cfg, g["inv_tau"])
    W = host_weights(t, cfg)
    yield cfg, model, W, g["inv_tau"]
    model.close()


def _prompt(cfg, n, seed):
    return np.random.default_rng(seed).integers(0, cfg.vocab - 1, n)


def _check(res, out_r, blk_start, gamma):
    """Confidences within 1e-3; decisions equal unless a confidence is within
    the tolerance of the threshold or of the top one (then exempt)."""
    A = res.masked_positions
    n = int(out_r["n"])
    if len(A) == 0:
        assert n == 0
        return
    bc = out_r["block_conf"][A - blk_start]
    assert np.all(np.abs(bc - res.masked_conf) <= CONF_TOL)
    got = set(out_r["pos"][:n].tolist())
    want = set(res.positions.tolist())
    if got == want:
        for p, t in zip(out_r["pos"][:n], out_r["tok"][:n]):
            i = list(res.positions).index(p)
            # the prediction may differ only on a near-tie of the top logits
            if t != res.tokens[i]:
                j = list(A).index(p)
                assert top2_gap(res.logits[j:j + 1])[0] <= 1e-4
        return
    near = set(A[np.abs(res.masked_conf - gamma) <= CONF_TOL].tolist())
    c = np.sort(res.masked_conf)[::-1]
    tie_top = len(c) > 1 and c[0] - c[1] <= CONF_TOL
    assert (got ^ want) <= near or (len(got) == len(want) == 1 and tie_top), (got, want)


def _run_teacher_forced(cfg, model, W, inv_tau, prompt, G, block, gamma, mode, max_steps=400):
    L = len(prompt) + G
    eng = engine.Engine(model, 1, L, mode)
    r = engine.Request(prompt, G, block, gamma)
    eng.admit(r, cfg.mask_id)
    oreq = oracle.Request.new(prompt, G, block, gamma, cfg.mask_id)
    steps, counts = 0, []
    while not oreq.done and steps < max_steps:
        eng.set_state(r, oreq.tokens, oreq.mask, oreq.k)
        blk = r.block_start
        eng.step([r])
        out = eng.read_outputs(1)
        res = oracle.denoise_step(cfg, W, oreq, mode, inv_tau, keep_logits=True)
        _check(res, {k: v[0] for k, v in out.items()}, blk, gamma)
        counts.append(int(out["n"][0]))
        steps += 1
    eng.close()
    assert oreq.done
    return steps, counts


@pytest.mark.parametrize("mode", ["none", "dual"])
def test_threshold_one_unmasks_one_per_step(tiny, mode):
    cfg, model, W, inv_tau = tiny
    steps, counts = _run_teacher_forced(cfg, model, W, inv_tau, _prompt(cfg, 40, 1), 48, 16, 1.0,
                                        mode)
    assert counts == [1] * 48 and steps == 48


@pytest.mark.parametrize("mode", ["none", "prefix"])
def test_threshold_zero_unmasks_each_block_at_once(tiny, mode):
    cfg, model, W, inv_tau = tiny
    steps, counts = _run_teacher_forced(cfg, model, W, inv_tau, _prompt(cfg, 40, 2), 80, 32, 0.0,
                                        mode)
    assert counts == [32, 32, 16] and steps == 3


def test_block_with_nothing_masked(tiny):
    """The caller unmasked the whole active block: nothing changes, n = 0."""
    cfg, model, W, inv_tau = tiny
    P, G = 50, 64
    prompt = _prompt(cfg, P, 3)
    eng = engine.Engine(model, 1, P + G, "none")
    r = engine.Request(prompt, G, 32, 0.9)
    eng.admit(r, cfg.mask_id)
    rng = np.random.default_rng(4)
    toks = np.concatenate([prompt, rng.integers(0, cfg.vocab - 1, G)])
    mask = np.zeros(P + G, np.uint8)
    mask[P + 32:] = 1                       # block 0 unmasked, block 1 masked
    eng.set_state(r, toks, mask, 0)
    r.masked_in_block = 1                   # keep the host from advancing first
    eng.enqueue_step([r])
    out = eng.read_outputs(1)
    t2, m2 = eng.read_state(r)
    assert int(out["n"][0]) == 0
    assert np.array_equal(t2, toks) and np.array_equal(m2, mask.astype(bool))
    assert np.all(out["block_conf"][0][:32] == -1.0)
    eng.close()


def test_sixty_four_requests_in_one_step(tiny):
    """DLM_MAX_REQ requests of mixed prompt and output lengths and blocks of
    8 .. 64, one no-cache step, each against its own oracle step."""
    cfg, model, W, inv_tau = tiny
    rng = np.random.default_rng(5)
    R = dlm.DLM_MAX_REQ
    spec = [(int(rng.integers(1, 120)), int(rng.choice([8, 16, 32, 64])), float(rng.choice([0.3, 0.9, 1.0])))
            for _ in range(R)]
    L = max(P + 2 * b for P, b, _ in spec)
    eng = engine.Engine(model, R, L, "none")
    reqs, oreqs = [], []
    for i, (P, b, gam) in enumerate(spec):
        G = 2 * b - int(rng.integers(0, b))          # ragged last block
        prompt = _prompt(cfg, P, 100 + i)
        r = engine.Request(prompt, G, b, gam)
        eng.admit(r, cfg.mask_id)
        reqs.append(r)
        oreqs.append(oracle.Request.new(prompt, G, b, gam, cfg.mask_id))
    starts = [r.block_start for r in reqs]
    eng.step(reqs)
    out = eng.read_outputs(R)
    for j, (r, o) in enumerate(zip(reqs, oreqs)):
        res = oracle.denoise_step(cfg, W, o, "none", inv_tau, keep_logits=True)
        _check(res, {k: v[j] for k, v in out.items()}, starts[j], r.threshold)
    eng.close()


def test_block_64_ragged_tail_dual(tiny):
    cfg, model, W, inv_tau = tiny
    steps, counts = _run_teacher_forced(cfg, model, W, inv_tau, _prompt(cfg, 30, 6), 100, 64, 0.9,
                                        "dual")
    assert sum(counts) == 100


def test_long_sequence_step(tiny):
    """A 2048-position sequence (1984 prompt + 64 masked): one no-cache step."""
    cfg, model, W, inv_tau = tiny
    P, G = 1984, 64
    prompt = _prompt(cfg, P, 7)
    eng = engine.Engine(model, 1, P + G, "none")
    r = engine.Request(prompt, G, 32, 0.9)
    eng.admit(r, cfg.mask_id)
    eng.step([r])
    out = eng.read_outputs(1)
    o = oracle.Request.new(prompt, G, 32, 0.9, cfg.mask_id)
    res = oracle.denoise_step(cfg, W, o, "none", inv_tau, keep_logits=True)
    _check(res, {k: v[0] for k, v in out.items()}, P, 0.9)
    eng.close()
