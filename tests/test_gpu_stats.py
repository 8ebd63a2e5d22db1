"""GPU parity of the per-request confidence statistics (the Step Predictor's
confidence features, computed in the unmask kernel) against the oracle, through
the C ABI: the oracle is fed the GPU's post-step token confidences and mask,
so the comparison isolates the statistics (the confidences themselves are
covered by the step parity tests). Also checks that every position the step
unmasks records the confidence it was unmasked with."""
import json
import os

import numpy as np
import pytest

import synth
from helpers import device_model
from oracle import stats as ost
from paper_2606_29094_amd import dlm, engine

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "tiny_fp32.json")
# fp32 kernel vs fp64 oracle on the same fp32 inputs: order statistics are
# exact, an interpolated quartile is one fp32 rounding of the same formula, the
# mean an fp32 sum of n values <= 1 (relative error below n * 2^-24)
ULP = 2.0 ** -23


@pytest.fixture(scope="module")
def tiny(gpu):
    g = json.load(open(GOLDEN))
    model, t = device_model(synth.TINY_FP32, g["inv_tau"])
    yield synth.TINY_FP32, model
    model.close()


def _check(stats_gpu, tok_conf, mask, req):
    want = ost.confidence_stats(tok_conf.astype(np.float64), mask.astype(np.uint8),
                                req.prompt_len, req.block_start_at_step, req.block_len_at_step)
    n = int(want[0])
    assert stats_gpu[0] == n and stats_gpu[7] == want[7], (stats_gpu, want)
    assert stats_gpu[1] == want[1] and stats_gpu[6] == want[6]
    for i in (2, 3, 5):
        assert abs(stats_gpu[i] - want[i]) <= 2 * ULP * max(abs(want[i]), 1e-30), (i, stats_gpu, want)
    assert abs(stats_gpu[4] - want[4]) <= max(n, 1) * ULP * max(abs(want[4]), 1e-30) + 1e-30
    return n


@pytest.mark.parametrize("gen_len,frac", [(64, 0.0), (64, 0.5), (1024, 0.3), (4096, 0.9),
                                          (8128, 0.97)])
def test_stats_on_synthetic_state(tiny, gen_len, frac):
    """Random unmasked output positions with random recorded confidences
    (duplicates included), active block in the middle, one no-cache step."""
    cfg, model = tiny
    rng = np.random.default_rng(gen_len + int(frac * 100))
    P, block = 64, 32
    prompt = rng.integers(0, cfg.vocab - 1, P)
    seq = P + gen_len
    eng = engine.Engine(model, 1, seq, "none", stats=True)
    r = engine.Request(prompt, gen_len, block, 0.9)
    eng.admit(r, cfg.mask_id)
    k = (gen_len // block) // 2
    tokens = np.concatenate([prompt, rng.integers(0, cfg.vocab - 1, gen_len)])
    mask = np.zeros(seq, np.uint8)
    mask[P:] = rng.random(gen_len) >= frac
    s = P + k * block
    mask[s:s + block] = 1                        # the active block starts fully masked
    tok_conf = rng.random(seq).astype(np.float32)
    tok_conf[P:P + gen_len // 4] = np.float32(0.5)   # ties
    tok_conf[:P] = np.float32(7.0)               # the prompt must not enter
    eng.set_state(r, tokens, mask, k, tok_conf)
    r.block_start_at_step, r.block_len_at_step = r.block_start, r.block_len
    eng.step([r])
    out = eng.read_outputs(1)
    tc = eng.read_tok_conf(r)
    _, m_after = eng.read_state(r)
    n_new = int(out["n"][0])
    pos = out["pos"][0, :n_new]
    assert np.array_equal(tc[pos], out["conf"][0, :n_new])
    n = _check(out["stats"][0], tc, m_after, r)
    print(f"G={gen_len} frac={frac}: n={n}, new={n_new}, stats={out['stats'][0]}")


def test_stats_along_generation(tiny):
    """Stats after every step of a free-running generation of 3 requests."""
    cfg, model = tiny
    reqs = []
    eng = engine.Engine(model, 3, 64 + 160, "dual", stats=True)
    for i, (G, thr) in enumerate([(64, 0.9), (160, 0.5), (96, 0.99)]):
        prompt, _, _ = synth.request(synth.C1, i)
        r = engine.Request(prompt, G, 32, thr)
        eng.admit(r, cfg.mask_id)
        reqs.append(r)
    steps = 0
    while not all(r.done for r in reqs) and steps < 400:
        active = [r for r in reqs if not r.done]
        for r in active:
            r.block_start_at_step, r.block_len_at_step = r.block_start, r.block_len
        eng.step(active)
        out = eng.read_outputs(len(active))
        for j, r in enumerate(active):
            _, m_after = eng.read_state(r)
            _check(out["stats"][j], eng.read_tok_conf(r), m_after, r)
        steps += 1
    assert all(r.done for r in reqs)
    for r in reqs:
        _, m = eng.read_state(r)
        assert not m.any()
        tc = eng.read_tok_conf(r)[r.prompt_len:]
        assert np.all((tc > 0) & (tc <= 1))


def test_stats_need_token_confidences(tiny):
    """Asking for statistics without a tok_conf buffer is rejected up front."""
    cfg, model = tiny
    eng = engine.Engine(model, 1, 128, "none", stats=True)
    prompt, G, thr = synth.request(synth.C1, 0)
    r = engine.Request(prompt, G, 32, thr)
    eng.admit(r, cfg.mask_id)
    batch = dlm.make_batch(eng.dlm_reqs([r]), eng.tokens, eng.mask, eng.mode_id, None)
    with pytest.raises(dlm.DlmError) as e:
        dlm.denoise_step(model.handle, eng.cache, batch, [thr], eng.step_out, eng.workspace)
    assert e.value.status == dlm.DLM_EINVAL
