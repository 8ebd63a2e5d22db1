"""The benchmarked workloads at their real shapes and full depth, checked
kernel by kernel on identical inputs (dlm_debug_trace at the first, a middle
and the last layer: every kernel against the oracle's operation on the exact
values it was given) and at the head and the unmask rule for every request
(oracle confidence() / select_unmask() on the GPU's own logits; confidences
within 1e-3, decisions exact outside the 1e-3 bands):

* MHA-8B, 8 requests x (1024 + 256), blocks of 32: the recompute step
  (10240 rows), then the dual-cache step (256 rows) and, separately, the
  prefix-cache step (2048 rows);
* MHA-8B, 32 heterogeneous requests (prompts 128..2048, outputs 128/256,
  thresholds 0.7..0.95): a step mixing recompute and cache steps;
* GQA-7B, 64 requests x (512 + 512), blocks of 64: the recompute step
  (65536 rows) and the 4096-row dual-cache step."""
import json
import os

import numpy as np
import pytest
import torch

import synth
import synth.device as sdev
from kernel_checks import summarize, trace_step_and_check
from paper_2606_29094_amd import engine

pytestmark = pytest.mark.gpu
GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _inv_tau(name):
    return json.load(open(os.path.join(GOLD, name)))["inv_tau"]


@pytest.fixture(scope="module")
def mha(gpu):
    cfg = synth.MHA_8B
    t = sdev.model_tensors(cfg)
    inv_tau = _inv_tau("mha_8b_step1.json")
    model = engine.DeviceModel(engine.ModelShape.of(cfg), t, inv_tau)
    yield cfg, t, model, inv_tau
    model.close()
    del t
    torch.cuda.empty_cache()


def _engine(model, cfg, w, ids, mode):
    reqs = []
    for i in ids:
        prompt, G, thr = synth.request(w, i)
        reqs.append(engine.Request(prompt, G, w.block, thr))
    L = max(r.seq_len for r in reqs)
    eng = engine.Engine(model, len(reqs), L, mode, max_rows=sum(r.seq_len for r in reqs))
    for r in reqs:
        eng.admit(r, cfg.mask_id)
    return eng, reqs


def _check(name, cfg, t, eng, reqs, inv_tau, layers):
    logs, counts, out = trace_step_and_check(cfg, t, eng, reqs, layers, inv_tau, n_sample=32)
    print(name, summarize(logs), counts, flush=True)
    return out


@pytest.mark.parametrize("mode", ["dual", "prefix"])
def test_mha_batch8_recompute_then_cache_step(mha, mode):
    cfg, t, model, inv_tau = mha
    w = synth.C3_DUAL if mode == "dual" else synth.C3_PREFIX
    eng, reqs = _engine(model, cfg, w, range(8), mode)
    assert sum(b - a for a, b in eng.step_rows(reqs)) == 8 * 1280
    _check(f"mha b8 {mode} recompute", cfg, t, eng, reqs, inv_tau, [0, 31])
    rows = sum(b - a for a, b in eng.step_rows(reqs))
    assert rows == (256 if mode == "dual" else 2048), rows
    _check(f"mha b8 {mode} cache step ({rows} rows)", cfg, t, eng, reqs, inv_tau, [0, 16, 31])
    eng.close()


def test_mha_heterogeneous_mixed_step(mha):
    """32 requests: after the first (recompute) step, every other request has
    its active block completed by the caller and moves to its next block
    (a recompute step), the others take a cache step."""
    cfg, t, model, inv_tau = mha
    w = synth.C4
    eng, reqs = _engine(model, cfg, w, range(32), "dual")
    eng.step(reqs)
    rng = np.random.default_rng(3)
    for i, r in enumerate(reqs):
        if i % 2 == 0 and not r.done:
            toks, mask = eng.read_state(r)
            s, e = r.block_start, r.block_start + r.block_len
            toks[s:e] = np.where(mask[s:e], rng.integers(0, cfg.vocab - 1, e - s), toks[s:e])
            mask[s:e] = False
            eng.set_state(r, toks, mask, r.k + 1)
    flags = [r.refreshed_block != r.block_start for r in reqs]
    assert any(flags) and not all(flags)
    rows = sum(b - a for a, b in eng.step_rows(reqs))
    _check(f"mha hetero mixed ({rows} rows, {sum(flags)} recompute)", cfg, t, eng, reqs,
           inv_tau, [0, 31])
    eng.close()


def test_gqa_batch64_recompute_then_cache_step(gpu):
    cfg = synth.GQA_7B
    t = sdev.model_tensors(cfg)
    inv_tau = _inv_tau("gqa_7b_step1.json")
    model = engine.DeviceModel(engine.ModelShape.of(cfg), t, inv_tau)
    eng, reqs = _engine(model, cfg, synth.C5, range(64), "dual")
    assert sum(b - a for a, b in eng.step_rows(reqs)) == 65536
    _check("gqa b64 recompute", cfg, t, eng, reqs, inv_tau, [0, 27])
    rows = sum(b - a for a, b in eng.step_rows(reqs))
    assert rows == 4096, rows
    _check("gqa b64 cache step (4096 rows)", cfg, t, eng, reqs, inv_tau, [0, 13, 27])
    eng.close()
    model.close()
    del t
    torch.cuda.empty_cache()
