"""Full-depth parity of the bf16 models against stored oracle values
(tests/golden/*_step1.json, written by make_golden.py from the oracle alone):
the first denoising step (block 0's recompute step) at the real sizes of the
workloads, compared on the outputs the oracle stored - the confidence and
prediction of every masked position of the active block, the unmask decision,
and a sample of the scaled logits (every 97th vocabulary column of the first
rows)."""
import json
import os

import numpy as np
import pytest
import torch

import synth
import synth.device as sdev
from helpers import LOGIT_TOL, conf_bound, check_decisions
from kernel_checks import check_head_unmask
from paper_2606_29094_amd import engine

pytestmark = pytest.mark.gpu
GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    path = os.path.join(GOLD, name)
    if not os.path.exists(path):
        pytest.skip(f"{name} not generated")
    return json.load(open(path))


@pytest.fixture(scope="module")
def mha_full(gpu):
    g = _golden("mha_8b_step1.json")
    cfg = synth.MHA_8B
    t = sdev.model_tensors(cfg)
    model = engine.DeviceModel(engine.ModelShape.of(cfg), t, g["inv_tau"])
    yield cfg, model, g
    model.close()
    del t
    torch.cuda.empty_cache()


def _compare(gr, z_blk, out_r, blk_start):
    """gr: stored oracle values of one request; z_blk: GPU scaled logits of
    the block rows; out_r: GPU step outputs of that request."""
    A = np.array(gr["positions"])
    conf_ref = np.array(gr["conf"])
    stride = gr["logit_stride"]
    zs_ref = np.array(gr["logits_sample"])               # first rows, sampled columns
    zs_gpu = z_blk[A[:len(zs_ref)] - blk_start][:, ::stride]
    rel = np.abs(zs_gpu - zs_ref).max(axis=1) / np.array(gr["max_abs_logit"][:len(zs_ref)])
    assert rel.max() < LOGIT_TOL["bf16"], rel.max()
    # eta: the sampled rows' error, doubled for the unsampled columns and rows
    eta = 2.0 * np.abs(zs_gpu - zs_ref).max()
    bound = conf_bound(conf_ref, eta)
    bc = out_r["block_conf"][A - blk_start]
    cerr = np.abs(bc - conf_ref)
    assert np.all(cerr <= bound), (cerr.max(), bound.min())
    bt = out_r["block_tok"][A - blk_start]
    tok_ok = (bt == np.array(gr["tok"])) | (np.array(gr["top2_gap"]) <= 2 * eta)
    assert tok_ok.all()
    exempt = check_decisions(A, conf_ref, bound, gr["threshold"], out_r, set(gr["unmasked"]))
    return rel.max(), cerr.max(), exempt


def _head_all(z, out, starts, reqs):
    """The fused head and the unmask decision of every request against the
    oracle's confidence() / select_unmask() on the GPU's own logits of the
    step (the whole block is masked at the first step)."""
    counts, off = {}, 0
    for j, r in enumerate(reqs):
        L = r.block_len_at_start
        check_head_unmask(z[off:off + L], {k: v[j] for k, v in out.items()}, starts[j],
                          np.arange(starts[j], starts[j] + L), r.threshold, counts)
        off += L
    assert counts.get("checked", 0) > 0, counts
    return counts


def _run(model, cfg, workload, reqs_idx, mode):
    """Admit the requests, take the logits of the first step, then the step."""
    reqs = []
    for r in reqs_idx:
        prompt, G, thr = synth.request(workload, r)
        reqs.append(engine.Request(prompt, G, workload.block, thr))
    L = max(r.seq_len for r in reqs)
    eng = engine.Engine(model, len(reqs), L, mode, max_rows=sum(r.seq_len for r in reqs))
    for r in reqs:
        eng.admit(r, cfg.mask_id)
    saved = [r.refreshed_block for r in reqs]
    z = eng.debug_logits(reqs).cpu().numpy()
    for r, s in zip(reqs, saved):
        r.refreshed_block = s
    starts = [r.block_start for r in reqs]
    for r in reqs:
        r.block_len_at_start = r.block_len
    eng.step(reqs)
    out = eng.read_outputs(len(reqs))
    eng.close()
    print("head + unmask on the GPU's own logits, every request:", _head_all(z, out, starts, reqs))
    return z, out, starts


def test_mha_nocache_step1_full_depth(mha_full):
    cfg, model, g = mha_full
    gr = [x for x in g["requests"] if x["workload"] == synth.C2.name][0]
    z, out, starts = _run(model, cfg, synth.C2, [0], "none")
    res = _compare(gr, z[:32], {k: v[0] for k, v in out.items()}, starts[0])
    print("mha no-cache full depth: logit rel err %.2e, conf err %.3f, exempt %d" % res)


def test_mha_dual_batch8_step1_full_depth(mha_full):
    """The whole 8-request batch (10240 recomputed rows): every request's head
    and decisions on the GPU's logits; request 0 also against the stored
    oracle values."""
    cfg, model, g = mha_full
    gr = [x for x in g["requests"] if x["workload"] == synth.C3_DUAL.name][0]
    z, out, starts = _run(model, cfg, synth.C3_DUAL, list(range(8)), "dual")
    res = _compare(gr, z[:32], {k: v[0] for k, v in out.items()}, starts[0])
    print("mha dual B=8 full depth (request 0): logit rel err %.2e, conf err %.3f, exempt %d" % res)


def test_mha_hetero_request0_full_depth(mha_full):
    cfg, model, g = mha_full
    gr = [x for x in g["requests"] if x["workload"] == synth.C4.name][0]
    z, out, starts = _run(model, cfg, synth.C4, [0], "dual")
    res = _compare(gr, z[:32], {k: v[0] for k, v in out.items()}, starts[0])
    print("mha heterogeneous request 0 (P=%d) full depth: logit rel err %.2e, conf err %.3f, "
          "exempt %d" % ((gr["prompt_len"],) + res))


def test_gqa_dual_step1_full_depth(gpu):
    g = _golden("gqa_7b_step1.json")
    cfg = synth.GQA_7B
    t = sdev.model_tensors(cfg)
    model = engine.DeviceModel(engine.ModelShape.of(cfg), t, g["inv_tau"])
    z, out, starts = _run(model, cfg, synth.C5, list(range(64)), "dual")
    off = 0
    for j, gr in enumerate(g["requests"]):
        blk = z[off:off + synth.C5.block]
        off += synth.C5.block
        res = _compare(gr, blk, {k: v[j] for k, v in out.items()}, starts[j])
        print("gqa dual full depth request %d: logit rel err %.2e, conf err %.3f, exempt %d"
              % ((j,) + res))
    model.close()
