"""GPU parity of the attention paths for every query/key-value head ratio
and head size the library dispatches on, with small bf16 models (2 layers)
against the oracle: ratios 2, 4, 7 and 8 use the shared-tile grouped-query
kernel (blocks of 8, 8, 7 and 8 waves), ratio 3 the per-head kernel; head
sizes 64 and 128. Requests of ragged lengths (key tiles of 64 with a partial
last tile), recompute steps then dual-cache steps, teacher-forced."""
import dataclasses

import pytest

import oracle
import synth
import synth.device as sdev
from helpers import calibrated_inv_tau, host_weights, run_teacher_forced
from paper_2606_29094_amd import engine

pytestmark = pytest.mark.gpu

SHAPES = [  # (n_q_heads, n_kv_heads, head_dim, d_model)
    (8, 4, 64, 512),
    (8, 2, 128, 512),
    (14, 2, 64, 448),
    (16, 2, 128, 512),
    (6, 2, 64, 384),
]


@pytest.mark.parametrize("hq,hkv,dh,d", SHAPES,
                         ids=[f"g{hq // hkv}-dh{dh}" for hq, hkv, dh, _ in SHAPES])
def test_head_ratio_dual(gpu, hq, hkv, dh, d):
    cfg = synth.ModelConfig(f"gqa-g{hq // hkv}-dh{dh}", 2, d, hq, hkv, dh, 1024, 4096, "bf16")
    t = sdev.model_tensors(cfg)
    W = host_weights(t, cfg)
    specs = [(70, 60), (130, 40), (13, 100)]          # (prompt, generated): L = 130, 170, 113
    prompts = [synth.tokens(300 + i, p, cfg.vocab) for i, (p, _) in enumerate(specs)]
    gammas = [0.9, 0.7, 0.95]
    oreqs = [oracle.Request.new(p, g, 32, gm, cfg.mask_id)
             for p, (_, g), gm in zip(prompts, specs, gammas)]
    inv_tau = calibrated_inv_tau(cfg, W, oreqs, "dual")
    model = engine.DeviceModel(engine.ModelShape.of(cfg), t, inv_tau)
    eng = engine.Engine(model, 3, 192, "dual")
    reqs = [engine.Request(p, g, 32, gm) for p, (_, g), gm in zip(prompts, specs, gammas)]
    for r in reqs:
        eng.admit(r, cfg.mask_id)
    st = run_teacher_forced(cfg, W, eng, reqs, oreqs, "dual", inv_tau, 4)
    print(cfg.name, st)
    assert any(st["kinds"]) and not all(st["kinds"])
    eng.close()
    model.close()
