"""GPU parity of the bf16 models at full width (the real layer shapes of the
MHA-8B and GQA-7B configurations) and reduced depth (2 layers), against the
oracle with bf16 storage rounding: step logits (2e-2), confidences (bounded by
each row's logit error, see helpers), unmask decisions, for no-cache,
dual-cache and prefix-cache steps, ragged request lengths, short last blocks
and batches that mix recompute and cache steps."""
import dataclasses

import numpy as np
import pytest

import oracle
import synth
import synth.device as sdev
from helpers import calibrated_inv_tau, gpu_step_with_logits, host_weights, run_teacher_forced
from paper_2606_29094_amd import engine

pytestmark = pytest.mark.gpu
N_LAYERS = 2


@pytest.fixture(scope="module")
def mha(gpu):
    cfg = synth.MHA_8B
    t = sdev.model_tensors(cfg, N_LAYERS)
    return cfg, t, host_weights(t, cfg)


@pytest.fixture(scope="module")
def gqa(gpu):
    cfg = synth.GQA_7B
    t = sdev.model_tensors(cfg, N_LAYERS)
    return cfg, t, host_weights(t, cfg)


def _model(cfg, t, inv_tau):
    shape = dataclasses.replace(engine.ModelShape.of(cfg), n_layers=N_LAYERS)
    return engine.DeviceModel(shape, t, inv_tau)


def test_mha_nocache_full_width(mha):
    """MHA shapes of the 256+256 no-cache workload (512 recomputed rows)."""
    cfg, t, W = mha
    prompt, G, thr = synth.request(synth.C2, 0)
    oreqs = [oracle.Request.new(prompt, G, 32, thr, cfg.mask_id)]
    inv_tau = calibrated_inv_tau(cfg, W, oreqs, "none")
    eng = engine.Engine(_model(cfg, t, inv_tau), 1, 512, "none")
    reqs = [engine.Request(prompt, G, 32, thr)]
    eng.admit(reqs[0], cfg.mask_id)
    st = run_teacher_forced(cfg, W, eng, reqs, oreqs, "none", inv_tau, 2)
    print("mha none:", st)


@pytest.mark.parametrize("mode", ["dual", "prefix"])
def test_mha_cache_steps_ragged_batch(mha, mode):
    """Three requests with ragged prompts and generation lengths (the last
    block of the third is short): recompute steps then cache steps."""
    cfg, t, W = mha
    specs = [(200, 96), (77, 64), (131, 40)]
    prompts = [synth.tokens(500 + i, p, cfg.vocab) for i, (p, _) in enumerate(specs)]
    gammas = [0.9, 0.7, 0.95]
    oreqs = [oracle.Request.new(p, g, 32, gm, cfg.mask_id)
             for p, (_, g), gm in zip(prompts, specs, gammas)]
    inv_tau = calibrated_inv_tau(cfg, W, oreqs, mode)
    eng = engine.Engine(_model(cfg, t, inv_tau), 3, 320, mode)
    reqs = [engine.Request(p, g, 32, gm) for p, (_, g), gm in zip(prompts, specs, gammas)]
    for r in reqs:
        eng.admit(r, cfg.mask_id)
    st = run_teacher_forced(cfg, W, eng, reqs, oreqs, mode, inv_tau, 4)
    print(mode, st)
    assert any(st["kinds"]) and not all(st["kinds"])


def test_mha_cache_steps_long_keys(mha):
    """Recompute then cache steps of three requests with longer, ragged key
    ranges (600, 200 and 520 positions; 32-row cache steps attend over all of
    them)."""
    cfg, t, W = mha
    specs = [(504, 96), (136, 64), (424, 96)]
    prompts = [synth.tokens(700 + i, p, cfg.vocab) for i, (p, _) in enumerate(specs)]
    gammas = [0.9, 0.8, 0.95]
    oreqs = [oracle.Request.new(p, g, 32, gm, cfg.mask_id)
             for p, (_, g), gm in zip(prompts, specs, gammas)]
    inv_tau = calibrated_inv_tau(cfg, W, oreqs, "dual")
    eng = engine.Engine(_model(cfg, t, inv_tau), 3, 640, "dual")
    reqs = [engine.Request(p, g, 32, gm) for p, (_, g), gm in zip(prompts, specs, gammas)]
    for r in reqs:
        eng.admit(r, cfg.mask_id)
    st = run_teacher_forced(cfg, W, eng, reqs, oreqs, "dual", inv_tau, 3)
    print("long keys:", st)
    assert any(st["kinds"]) and not all(st["kinds"])


def test_gqa_dual_refresh_then_cache(gqa):
    """GQA (28 query / 4 kv heads), blocks of 64, dual cache."""
    cfg, t, W = gqa
    prompts = [synth.tokens(900 + i, 128, cfg.vocab) for i in range(2)]
    oreqs = [oracle.Request.new(p, 128, 64, 0.9, cfg.mask_id) for p in prompts]
    inv_tau = calibrated_inv_tau(cfg, W, oreqs, "dual")
    eng = engine.Engine(_model(cfg, t, inv_tau), 2, 256, "dual")
    reqs = [engine.Request(p, 128, 64, 0.9) for p in prompts]
    for r in reqs:
        eng.admit(r, cfg.mask_id)
    st = run_teacher_forced(cfg, W, eng, reqs, oreqs, "dual", inv_tau, 3)
    print("gqa dual:", st)
    assert st["kinds"][:2] == [True, True] and not all(st["kinds"])


def test_mixed_refresh_and_cache_in_one_batch(mha):
    """A request at a block boundary (recompute step) batched with two
    requests in cache steps."""
    cfg, t, W = mha
    prompts = [synth.tokens(700 + i, p, cfg.vocab) for i, p in enumerate((150, 60, 97))]
    oreqs = [oracle.Request.new(p, 64, 32, 0.8, cfg.mask_id) for p in prompts]
    inv_tau = calibrated_inv_tau(cfg, W, oreqs, "dual")
    eng = engine.Engine(_model(cfg, t, inv_tau), 3, 256, "dual")
    reqs = [engine.Request(p, 64, 32, 0.8) for p in prompts]
    for r in reqs:
        eng.admit(r, cfg.mask_id)
    run_teacher_forced(cfg, W, eng, reqs, oreqs, "dual", inv_tau, 1)
    # request 0 jumps to its second block (block 1 filled in), the others stay
    oq = oreqs[0]
    s, e = oq.block_bounds
    oq.tokens[s:e] = synth.tokens(77, e - s, cfg.vocab)
    oq.mask[s:e] = False
    oq.k += 1
    st = run_teacher_forced(cfg, W, eng, reqs, oreqs, "dual", inv_tau, 1)
    assert st["kinds"] == [True, False, False]
    print("mixed:", st)


def test_mha_nocache_step_is_bitwise_repeatable(mha):
    """The 512-row no-cache step twice from the same state: logits and
    confidences identical bit for bit (no atomics in the arithmetic: split-K
    slices are summed in slice order by their consumer)."""
    cfg, t, W = mha
    prompt, G, thr = synth.request(synth.C2, 0)
    model = _model(cfg, t, 8.0)
    runs = []
    for _ in range(2):
        eng = engine.Engine(model, 1, 512, "none")
        r = engine.Request(prompt, G, 32, thr)
        eng.admit(r, cfg.mask_id)
        z, out, _ = gpu_step_with_logits(eng, [r])
        runs.append((z[0].copy(), out["block_conf"].copy(), out["pos"].copy()))
        eng.close()
    model.close()
    for a, b in zip(runs[0], runs[1]):
        assert np.array_equal(a, b)
