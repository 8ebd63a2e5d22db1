"""GPU parity of the fused LM head (dlm_head_confidence) at full vocabulary
size against the oracle's confidence of the same rows, plus its closed forms:
a zero hidden row gives confidence 1/V and token 0; a row aligned with one
vocabulary row gives that token."""
import numpy as np
import pytest
import torch

import oracle
import synth
import synth.device as sdev
from helpers import CONF_TOL
from paper_2606_29094_amd import dlm, engine

pytestmark = pytest.mark.gpu


def _model_with_head(cfg, inv_tau):
    """A 1-layer model of the given shape (only the head is exercised)."""
    import dataclasses
    t = sdev.model_tensors(cfg, n_layers=1)
    shape = dataclasses.replace(engine.ModelShape.of(cfg), n_layers=1)
    return engine.DeviceModel(shape, t, inv_tau), t


def _oracle_conf(u, W_lm, inv_tau, chunk=16384):
    """confidence() of z = u W^T * inv_tau, z computed in fp64 by vocab chunks
    (same values as one matmul; chunking only bounds host memory)."""
    u = np.asarray(u, np.float64)
    z = np.empty((u.shape[0], W_lm.shape[0]))
    for s in range(0, W_lm.shape[0], chunk):
        z[:, s:s + chunk] = u @ W_lm[s:s + chunk].astype(np.float64).T
    return oracle.confidence(z * inv_tau), z * inv_tau


@pytest.mark.parametrize("cfg,inv_tau", [(synth.MHA_8B, 10.0), (synth.GQA_7B, 8.0),
                                         (synth.TINY_FP32, 13.0)],
                         ids=["mha-v126464", "gqa-v152064", "tiny-f32"])
def test_head_confidence_matches_oracle(gpu, cfg, inv_tau):
    model, t = _model_with_head(cfg, inv_tau)
    W = t["lm_head"].float().cpu().numpy()
    rng = np.random.default_rng(7)
    dt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    # 300 and 400 rows: several row tiles (the launch whose blocks walk the
    # active tiles), with 128x192 two-ring tiles at 300 rows and 256x256
    # split-phase tiles at 400 (a ragged second row tile)
    for M in (1, 37, 256) + ((300, 400) if cfg.dtype == "bf16" else ()):
        u = torch.from_numpy(rng.standard_normal((M, cfg.d_model)).astype(np.float32)).to(dt)
        u[0] = 0                                   # closed form: 1/V, token 0
        if M > 1:
            u[1] = t["lm_head"][1234].float().cpu().to(dt) * 50   # aligned with token 1234
        u_d = u.to(gpu).contiguous()
        conf = torch.empty(M, dtype=torch.float32, device=gpu)
        tok = torch.empty(M, dtype=torch.int32, device=gpu)
        ws = torch.empty(dlm.workspace_bytes(model.handle, M, 1) + (1 << 20), dtype=torch.uint8,
                         device=gpu)
        dlm.head_confidence(model.handle, u_d, M, conf, tok, ws)
        torch.cuda.synchronize()
        (c_ref, t_ref), z = _oracle_conf(u.float().numpy(), W, inv_tau)
        c = conf.cpu().numpy()
        tk = tok.cpu().numpy()
        assert np.all(np.abs(c - c_ref) <= CONF_TOL), np.abs(c - c_ref).max()
        assert c[0] == pytest.approx(1.0 / cfg.vocab, rel=1e-4) and tk[0] == 0
        if M > 1:
            assert tk[1] == 1234
        srt = np.sort(z, axis=1)
        tie = (srt[:, -1] - srt[:, -2]) < 1e-3 * np.abs(z).max(axis=1)
        assert np.all((tk == t_ref) | tie)
        print(cfg.name, M, "max conf err", np.abs(c - c_ref).max(), "token ties exempt", tie.sum())
