"""Kernel-level parity on identical inputs, through the C ABI
(dlm_debug_trace): every kernel of a traced layer against the oracle's
operation on the exact values the kernel was given (embedding gather,
attention norm, each QKV K-split slice, rotary embedding of queries and keys,
the value write, attention over the slot, output projection + residual, FFN
norm, SwiGLU, down projection + residual; final norm and logits at the last
layer), then the fused LM head and the unmask decision of every request
against the oracle's confidence() and select_unmask() on the GPU's own logits
(confidences within 1e-3, decisions exact outside the 1e-3 bands).

Models: the tiny fp32 model, and the MHA-8B / GQA-7B layer shapes at full
width with 2 layers; steps: no-cache, recompute, dual-cache and prefix-cache
steps over ragged batches."""
import dataclasses
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
GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "tiny_fp32.json")


def _model(cfg, n_layers, inv_tau):
    t = sdev.model_tensors(cfg, n_layers)
    shape = dataclasses.replace(engine.ModelShape.of(cfg), n_layers=n_layers)
    return engine.DeviceModel(shape, t, inv_tau), t, dataclasses.replace(cfg, n_layers=n_layers)


@pytest.fixture(scope="module")
def tiny(gpu):
    inv_tau = json.load(open(GOLDEN))["inv_tau"]
    m, t, cfg = _model(synth.TINY_FP32, 2, inv_tau)
    yield m, t, cfg, inv_tau
    m.close()


@pytest.fixture(scope="module")
def mha2(gpu):
    m, t, cfg = _model(synth.MHA_8B, 2, 8.0)
    yield m, t, cfg, 8.0
    m.close()
    del t
    torch.cuda.empty_cache()


@pytest.fixture(scope="module")
def gqa2(gpu):
    m, t, cfg = _model(synth.GQA_7B, 2, 8.0)
    yield m, t, cfg, 8.0
    m.close()
    del t
    torch.cuda.empty_cache()


def _batch(model, cfg, mode, specs, block, seed):
    """specs: [(prompt_len, gen_len, threshold)]."""
    reqs = [engine.Request(synth.tokens(seed + i, P, cfg.vocab), G, block, g)
            for i, (P, G, g) in enumerate(specs)]
    L = max(r.seq_len for r in reqs)
    eng = engine.Engine(model, len(reqs), L, mode, max_rows=sum(r.seq_len for r in reqs))
    for r in reqs:
        eng.admit(r, cfg.mask_id)
    return eng, reqs


def _run(name, cfg, t, eng, reqs, inv_tau, warm_steps=0):
    for _ in range(warm_steps):
        eng.step(reqs)
    logs, counts, _ = trace_step_and_check(cfg, t, eng, reqs, list(range(cfg.n_layers)), inv_tau)
    print(name, summarize(logs), counts)
    return counts


@pytest.mark.parametrize("mode,warm", [("none", 0), ("none", 2), ("dual", 1), ("prefix", 1)])
def test_tiny_fp32_kernels(tiny, mode, warm):
    model, t, cfg, inv_tau = tiny
    eng, reqs = _batch(model, cfg, mode, [(64, 64, 0.9), (37, 50, 0.7), (100, 28, 0.95)], 32, 40)
    _run(f"tiny {mode} after {warm}", cfg, t, eng, reqs, inv_tau, warm)
    eng.close()


def test_mha_nocache_512_rows_kernels(mha2):
    """The single-request 256 + 256 no-cache step (512 rows)."""
    model, t, cfg, inv_tau = mha2
    eng, reqs = _batch(model, cfg, "none", [(256, 256, 0.9)], 32, 0)
    _run("mha none 512", cfg, t, eng, reqs, inv_tau)
    eng.close()


@pytest.mark.parametrize("mode", ["dual", "prefix"])
def test_mha_cache_step_ragged_kernels(mha2, mode):
    """Recompute step of three ragged requests, then their cache step."""
    model, t, cfg, inv_tau = mha2
    eng, reqs = _batch(model, cfg, mode, [(200, 96, 0.9), (77, 64, 0.7), (131, 40, 0.95)], 32, 10)
    _run(f"mha {mode} recompute", cfg, t, eng, reqs, inv_tau)
    _run(f"mha {mode} cache", cfg, t, eng, reqs, inv_tau)
    eng.close()


def test_gqa_cache_step_block64_kernels(gqa2):
    """GQA (28 query / 4 kv heads), blocks of 64: recompute then cache step
    of four requests with ragged prompts."""
    model, t, cfg, inv_tau = gqa2
    eng, reqs = _batch(model, cfg, "dual", [(128, 128, 0.9), (190, 128, 0.5), (64, 100, 0.99),
                                            (255, 64, 0.7)], 64, 20)
    _run("gqa dual recompute", cfg, t, eng, reqs, inv_tau)
    _run("gqa dual cache", cfg, t, eng, reqs, inv_tau)
    eng.close()
