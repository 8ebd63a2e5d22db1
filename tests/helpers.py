"""Shared helpers of the GPU tests: device models, host copies for the oracle,
and the comparison rules (tolerances and exemptions)."""
from __future__ import annotations

import copy

import numpy as np
import torch

import oracle
import synth
import synth.device as sdev
from kernel_checks import check_head_unmask
from paper_2606_29094_amd import engine

# Tolerances: bf16 logits 2e-2, fp32 logits 1e-4 (max abs error over a row
# divided by the row's max |z|); confidences 1e-3 absolute; unmask decisions
# exact except at positions whose oracle confidence is within 1e-3 of the
# threshold, rows whose top-2 scaled logits are closer than the logit
# tolerance (the token may differ), and force-one steps whose top-2
# confidences are within 1e-3 (the position may differ).
LOGIT_TOL = {"bf16": 2e-2, "f32": 1e-4}
CONF_TOL = 1e-3
# bf16 end to end (forward + head): the fp64 oracle rounds to bf16 at the same
# storage points but cannot reproduce the roundings the GPU takes from fp32
# sums; every divergent rounding is a 2^-8 step and the calibrated 1/tau
# (about 10) scales the resulting logit differences. The confidence is then
# checked against what the row's own logit error allows: if every scaled logit
# of a row is within eta of the oracle's, S = sum exp(z - max z) moves by at
# most a factor exp(2 eta), so |conf_gpu - conf_ref| <= conf_ref (exp(2 eta) - 1)
# (plus the 1e-3 of the confidence computation itself). This band is an extra
# end-to-end check only: it is wide at full depth and does not bind the
# 1e-3 confidence contract, which bf16 storage cannot meet end to end against
# an fp64 oracle. What binds, on every step these helpers run: the logits
# within LOGIT_TOL of the oracle's, and the fused head's confidences (1e-3)
# and the unmask decisions (exact outside the 1e-3 bands) against the
# oracle's confidence() and select_unmask() applied to the GPU's own logits of
# the step (kernel_checks.check_head_unmask); each kernel on identical inputs
# is checked in test_gpu_trace / test_gpu_configs.


def conf_bound(conf_ref, eta):
    return np.asarray(conf_ref) * np.expm1(2.0 * np.asarray(eta)) + CONF_TOL


def gpu_step_with_logits(eng, reqs):
    """Scaled logits of every active-block row for the step about to run,
    then the step itself with the same recompute/cache flags."""
    saved = [r.refreshed_block for r in reqs]
    z = eng.debug_logits(reqs).cpu().numpy()
    for r, s in zip(reqs, saved):
        r.refreshed_block = s
    starts = [r.block_start for r in reqs]
    lens = [r.block_len for r in reqs]
    eng.step(reqs)
    out = eng.read_outputs(len(reqs))
    rows, off = [], 0
    for L in lens:
        rows.append(z[off:off + L])
        off += L
    return rows, out, starts


def check_step_e2e(res, out_r, blk_start, gamma, z_gpu_blk, dtype="bf16"):
    """Compare one request's GPU step with the oracle StepResult ``res``
    (computed with keep_logits). Returns (max logit err, max conf err, exempt)."""
    A = res.masked_positions
    if len(A) == 0:
        assert int(out_r["n"]) == 0
        return 0.0, 0.0, 0
    zg = z_gpu_blk[A - blk_start]
    zr = res.logits
    lerr = logit_err(zg, zr)
    assert lerr < LOGIT_TOL[dtype], lerr
    eta = np.abs(zg - zr).max(axis=1)
    bound = conf_bound(res.masked_conf, eta)
    bc = out_r["block_conf"][A - blk_start]
    cerr = np.abs(bc - res.masked_conf)
    assert np.all(cerr <= bound), (cerr.max(), bound[np.argmax(cerr - bound)])
    # tokens: equal unless the oracle's top-2 scaled logits are within 2 eta
    bt = out_r["block_tok"][A - blk_start]
    assert np.all((bt == res.masked_tok) | (top2_gap(zr) <= 2 * eta))
    return lerr, float(cerr.max()), check_decisions(A, res.masked_conf, bound, gamma, out_r,
                                                     set(res.positions.tolist()))


def check_decisions(A, conf_ref, bound, gamma, out_r, want):
    """Unmask decisions given confidence intervals [conf_ref - bound, conf_ref + bound].

    Positions certainly above the threshold must be unmasked, positions
    certainly not above it must not be (unless forced); a forced single unmask
    must pick a position whose interval reaches the top interval. Returns the
    number of positions where the GPU and the oracle differ (all exempt)."""
    n = int(out_r["n"])
    got = set(out_r["pos"][:n].tolist())
    assert len(got) == n and n >= (1 if len(A) else 0)
    sure_pass = set(A[conf_ref - bound > gamma].tolist())
    sure_fail = set(A[conf_ref + bound <= gamma].tolist())
    top = int(np.argmax(conf_ref))
    plausible_top = set(A[conf_ref + bound >= conf_ref[top] - bound[top]].tolist())
    if sure_pass:
        assert sure_pass <= got and not (got & sure_fail), (sorted(got), sorted(sure_pass))
    elif len(got) == 1 and got <= plausible_top:
        pass                                   # forced single unmask (or one undecided pass)
    else:
        assert not (got & sure_fail), (sorted(got), sorted(sure_fail))
    return len(got ^ want)


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


def calibrated_inv_tau(cfg, W, oreqs, mode):
    """Calibrate on the oracle's first step of these requests (share 0.3 > 0.9)."""
    zs = []
    for oq in oreqs:
        q = copy.deepcopy(oq)
        h, rows, _ = oracle.step_forward(cfg, W, q, mode)
        s, e = q.block_bounds
        A = np.nonzero(q.mask[s:e])[0] + s
        zs.append(oracle.head_logits(cfg, W, h[A - rows[0]], 1.0))
    return float(oracle.calibrate(np.concatenate(zs), 0.9, 0.3)[1])


def run_teacher_forced(cfg, W, eng, reqs, oreqs, mode, inv_tau, n_steps):
    """n_steps batched steps; before each, every request is set to the
    oracle's state; each request's step is compared with the oracle's."""
    stats = {"lerr": 0.0, "cerr": 0.0, "exempt": 0, "kinds": [], "head": {}}
    for _ in range(n_steps):
        active = [i for i, oq in enumerate(oreqs) if not oq.done]
        if not active:
            break
        for i in active:
            eng.set_state(reqs[i], oreqs[i].tokens, oreqs[i].mask, oreqs[i].k)
        flags = [reqs[i].refreshed_block != reqs[i].block_start for i in active]
        z_rows, out, starts = gpu_step_with_logits(eng, [reqs[i] for i in active])
        for j, i in enumerate(active):
            res = oracle.denoise_step(cfg, W, oreqs[i], mode, inv_tau, keep_logits=True)
            assert res.refresh == (flags[j] or mode == "none")
            stats["kinds"].append(res.refresh)
            out_j = {k: v[j] for k, v in out.items()}
            l, c, e = check_step_e2e(res, out_j, starts[j], reqs[i].threshold, z_rows[j])
            check_head_unmask(z_rows[j], out_j, starts[j], res.masked_positions,
                              reqs[i].threshold, stats["head"])
            stats["lerr"] = max(stats["lerr"], l)
            stats["cerr"] = max(stats["cerr"], c)
            stats["exempt"] += e
    assert stats["head"].get("checked", 0) > 0, stats["head"]
    return stats
