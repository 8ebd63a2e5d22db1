"""dlm_denoise_step_noalloc (the step with the library's fixed per-GPU scratch
instead of a workspace argument) against dlm_denoise_step on the same
inputs: the same outputs bit for bit (same kernels, same plans), for two
calls in a row, the second with fewer rows than the first, through the C
ABI; a step whose workspace exceeds the fixed scratch is rejected with
DLM_ESIZE and changes nothing."""
import dataclasses
import json
import os

import numpy as np
import pytest
import torch

import synth
import synth.device as sdev
from paper_2606_29094_amd import dlm, engine

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "tiny_fp32.json")


def _engines(model, cfg, mode, specs, block, seed):
    """Two engines holding the same requests (one per entry point)."""
    out = []
    for _ in range(2):
        reqs = [engine.Request(synth.tokens(seed + i, P, cfg.vocab), G, block, g)
                for i, (P, G, g) in enumerate(specs)]
        L = max(r.seq_len for r in reqs)
        eng = engine.Engine(model, len(reqs), L, mode, max_rows=sum(r.seq_len for r in reqs))
        for r in reqs:
            eng.admit(r, cfg.mask_id)
        out.append((eng, reqs))
    return out


def _step_noalloc(eng, reqs):
    dreqs = eng.dlm_reqs(reqs)
    batch = dlm.make_batch(dreqs, eng.tokens, eng.mask, eng.mode_id, eng.tok_conf)
    dlm.denoise_step_noalloc(eng.model.handle, eng.cache, batch, [r.threshold for r in reqs],
                             eng.step_out)
    for r, d in zip(reqs, dreqs):
        if d.flags & dlm.DLM_REQ_REFRESH:
            r.refreshed_block = r.block_start
    return eng.finish_step(reqs)


def _same(a, b):
    (ea, ra), (eb, rb) = a, b
    oa, ob = ea.read_outputs(len(ra)), eb.read_outputs(len(rb))
    for j, (x, y) in enumerate(zip(ra, rb)):
        n = int(oa["n"][j])
        assert int(ob["n"][j]) == n
        bl = x.block
        for k in ("pos", "tok", "conf"):
            assert np.array_equal(oa[k][j][:n], ob[k][j][:n]), k
        for k in ("block_conf", "block_tok"):
            assert np.array_equal(oa[k][j][:bl], ob[k][j][:bl]), k
        for s, t in zip(ea.read_state(x), eb.read_state(y)):
            assert np.array_equal(s, t)
        assert (x.k, x.steps) == (y.k, y.steps)


def _rows(eng, reqs):
    return sum(b - a for a, b in eng.step_rows(reqs))


@pytest.mark.parametrize("mode", ["dual", "prefix"])
def test_noalloc_matches_step_tiny(gpu, mode):
    inv_tau = json.load(open(GOLDEN))["inv_tau"]
    cfg = synth.TINY_FP32
    t = sdev.model_tensors(cfg)
    model = engine.DeviceModel(engine.ModelShape.of(cfg), t, inv_tau)
    a, b = _engines(model, cfg, mode, [(64, 64, 0.9), (37, 50, 0.7), (100, 28, 0.95)], 32, 70)
    rows = []
    for _ in range(2):                       # a recompute step, then a smaller cache step
        rows.append(_rows(*a))
        a[0].step(a[1])
        _step_noalloc(*b)
        torch.cuda.synchronize()
        _same(a, b)
    assert rows[1] < rows[0]
    for e, _ in (a, b):
        e.close()
    model.close()


def test_noalloc_matches_step_mha_and_rejects_oversized(gpu):
    cfg = dataclasses.replace(synth.MHA_8B, n_layers=2)
    t = sdev.model_tensors(synth.MHA_8B, 2)
    shape = dataclasses.replace(engine.ModelShape.of(synth.MHA_8B), n_layers=2)
    model = engine.DeviceModel(shape, t, 8.0)
    for specs in ([(256, 256, 0.9)], [(150, 100, 0.8)]):    # 512 rows, then 250
        a, b = _engines(model, cfg, "none", specs, 32, 5)
        a[0].step(a[1])
        _step_noalloc(*b)
        torch.cuda.synchronize()
        _same(a, b)
        for e, _ in (a, b):
            e.close()
    # 1024 rows need more than the fixed scratch: rejected, nothing enqueued
    (e, reqs), (e2, _) = _engines(model, cfg, "none", [(768, 256, 0.9)], 32, 6)
    assert dlm.workspace_bytes(model.handle, 1024, 1) > dlm.DLM_SCRATCH_BYTES
    before = e.read_state(reqs[0])
    with pytest.raises(dlm.DlmError) as err:
        _step_noalloc(e, reqs)
    assert err.value.status == dlm.DLM_ESIZE
    torch.cuda.synchronize()
    after = e.read_state(reqs[0])
    assert all(np.array_equal(x, y) for x, y in zip(before, after))
    e.close()
    e2.close()
    model.close()
    del t
    torch.cuda.empty_cache()
