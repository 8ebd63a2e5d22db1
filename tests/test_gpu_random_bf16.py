"""Randomised bf16 batches against the oracle (small 2-layer models with the
grouped-query layout of the GQA model, ratio 7, and a multi-head one):
seeded mixes of 4-10 requests with prompts of 1-200 tokens, blocks of 16-64
with ragged last blocks and thresholds from 0.7 to 0.95, in each cache mode
("Support for Approximate Caching"), teacher-forced for several batched
steps. The varying row counts take the bf16 GEMMs through different tile,
split and sub-tile plans and the attention through partial query and key
tiles; each request's logits, confidences and decisions are checked as in the
other bf16 tests (the head and unmask rule on the GPU's own logits exactly,
the rest within the bf16 bounds)."""
import numpy as np
import pytest

import oracle
import synth
import synth.device as sdev
from helpers import calibrated_inv_tau, host_weights, run_teacher_forced
from paper_2606_29094_amd import engine

pytestmark = pytest.mark.gpu

MODELS = {  # name: (n_q_heads, n_kv_heads, head_dim, d_model, d_ffn)
    "gqa7": (14, 2, 64, 448, 1024),
    "mha": (4, 4, 128, 512, 1536),
}
CASES = [("gqa7", "dual", 21), ("gqa7", "prefix", 22), ("gqa7", "none", 23), ("mha", "dual", 24)]


@pytest.mark.parametrize("model,mode,seed", CASES, ids=lambda v: str(v))
def test_random_bf16_batch(gpu, model, mode, seed):
    hq, hkv, dh, d, ffn = MODELS[model]
    cfg = synth.ModelConfig(f"rand-{model}", 2, d, hq, hkv, dh, ffn, 4096, "bf16")
    t = sdev.model_tensors(cfg)
    W = host_weights(t, cfg)
    rng = np.random.default_rng(seed)
    R = int(rng.integers(4, 11))
    specs = []
    for i in range(R):
        b = int(rng.choice([16, 32, 64]))
        P = int(rng.integers(1, 201))
        G = int(rng.integers(1, 4)) * b - int(rng.integers(0, b // 2 + 1))
        specs.append((P, max(G, 1), b, float(rng.choice([0.7, 0.8, 0.9, 0.95]))))
    prompts = [synth.tokens(5000 + 100 * seed + i, P, cfg.vocab) for i, (P, _, _, _) in enumerate(specs)]
    oreqs = [oracle.Request.new(p, G, b, g, cfg.mask_id) for p, (_, G, b, g) in zip(prompts, specs)]
    inv_tau = calibrated_inv_tau(cfg, W, oreqs, mode)
    dm = engine.DeviceModel(engine.ModelShape.of(cfg), t, inv_tau)
    L = max(P + G for P, G, _, _ in specs)
    eng = engine.Engine(dm, R, L, mode)
    reqs = [engine.Request(p, G, b, g) for p, (_, G, b, g) in zip(prompts, specs)]
    for r in reqs:
        eng.admit(r, cfg.mask_id)
    st = run_teacher_forced(cfg, W, eng, reqs, oreqs, mode, inv_tau, 6)
    print(cfg.name, mode, R, st)
    if mode != "none":
        assert any(st["kinds"]), "no recompute step"
    eng.close()
    dm.close()
