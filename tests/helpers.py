"""Shared helpers of the GPU tests: device models, host copies for the oracle,
and the comparison rules (tolerances and exemptions)."""
from __future__ import annotations

import numpy as np
import torch

import oracle
import synth
import synth.device as sdev
from paper_2606_29094_amd import engine

# Tolerances: bf16 logits 2e-2, fp32 logits 1e-4 (max abs error over a row
# divided by the row's max |z|); confidences 1e-3 absolute; unmask decisions
# exact except at positions whose oracle confidence is within 1e-3 of the
# threshold, rows whose top-2 scaled logits are closer than the logit
# tolerance (the token may differ), and force-one steps whose top-2
# confidences are within 1e-3 (the position may differ).
LOGIT_TOL = {"bf16": 2e-2, "f32": 1e-4}
CONF_TOL = 1e-3


def host_weights(tensors, cfg) -> oracle.Weights:
    """Copy device weights to the host in the oracle's dict layout (inputs
    only: these are the generator's values, not results of the library)."""
    d, dh = cfg.d_model, cfg.head_dim
    qd, kd = cfg.n_q_heads * dh, cfg.n_kv_heads * dh
    f = lambda t: t.float().cpu().numpy()
    layers = []
    for l in tensors["layers"]:
        qkv = f(l["w_qkv"])
        gu = f(l["w_gate_up"])
        layers.append({"wq": qkv[:qd], "wk": qkv[qd:qd + kd], "wv": qkv[qd + kd:],
                       "wo": f(l["w_o"]), "wg": gu[:cfg.d_ffn], "wu": gu[cfg.d_ffn:],
                       "wd": f(l["w_down"]), "attn_norm": f(l["attn_norm"]),
                       "ffn_norm": f(l["ffn_norm"])})
    g = {"embed": f(tensors["embed"]), "lm_head": f(tensors["lm_head"]),
         "final_norm": f(tensors["final_norm"])}
    return oracle.Weights(g, layers=layers)


def device_model(cfg, inv_tau, n_layers=None):
    import dataclasses
    t = sdev.model_tensors(cfg, n_layers)
    shape = engine.ModelShape.of(cfg)
    if n_layers is not None:
        shape = dataclasses.replace(shape, n_layers=n_layers)
    return engine.DeviceModel(shape, t, inv_tau), t


def logit_err(z_gpu, z_ref):
    z_gpu = np.asarray(z_gpu, np.float64)
    z_ref = np.asarray(z_ref, np.float64)
    return float(np.max(np.abs(z_gpu - z_ref).max(axis=1) / np.abs(z_ref).max(axis=1)))


def top2_gap(z):
    s = np.sort(np.asarray(z, np.float64), axis=1)
    return s[:, -1] - s[:, -2]
