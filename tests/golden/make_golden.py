"""Write the stored expected values under tests/golden/ (calls only oracle/ and synth/).

For each model it runs the oracle's first denoising step (block 0's recompute
step) on a few requests of the workloads that use the model, calibrates the
logit temperature on the pooled masked positions of that step (share 0.3 of
positions above threshold 0.9) and stores, per request, the confidence and
prediction of every masked position of the active block plus a sample of the
scaled logits.

Usage: python tests/golden/make_golden.py [tiny|mha|gqa ...]
The full-scale models take several minutes of CPU (weights are drawn with a
process pool, layer by layer).
"""
from __future__ import annotations

import json
import os
import sys
import time
from multiprocessing import Pool

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
import synth   # noqa: E402

CHUNK = 1 << 23
LOGIT_STRIDE = 97     # stored logits sample: every 97th vocab column


def _chunk(args):
    seed, tid, start, count, std, dtype = args
    v = synth.normal_f64(seed, tid, start, count, std).astype(np.float32)
    if dtype == "bf16":
        v = synth.bf16_bits_to_f32(synth.f32_to_bf16_bits(v))
    return v


def gen_tensor(pool, cfg, tid, shape):
    n = int(np.prod(shape))
    jobs = [(cfg.weight_seed, tid, s, min(CHUNK, n - s), cfg.weight_std, cfg.dtype)
            for s in range(0, n, CHUNK)]
    return np.concatenate(pool.map(_chunk, jobs)).reshape(shape)


def gen_layer(pool, cfg, l):
    names = {synth.KIND_Q: "wq", synth.KIND_K: "wk", synth.KIND_V: "wv",
             synth.KIND_O: "wo", synth.KIND_GATE: "wg", synth.KIND_UP: "wu",
             synth.KIND_DOWN: "wd"}
    out = {names[k]: gen_tensor(pool, cfg, synth.layer_tid(l, k), s)
           for k, s in synth.layer_shapes(cfg).items()}
    out["attn_norm"] = np.ones(cfg.d_model, np.float32)
    out["ffn_norm"] = np.ones(cfg.d_model, np.float32)
    return out


def run_model(cfg, entries, pool, log):
    """entries: list of (workload, request index). Step 1 of each, layer-synchronous."""
    t0 = time.time()
    g = {"embed": gen_tensor(pool, cfg, synth.TID_EMBED, (cfg.vocab, cfg.d_model)),
         "lm_head": gen_tensor(pool, cfg, synth.TID_LM_HEAD, (cfg.vocab, cfg.d_model)),
         "final_norm": np.ones(cfg.d_model, np.float32)}
    log(f"{cfg.name}: globals drawn in {time.time() - t0:.0f}s")
    states = []
    for w, r in entries:
        prompt, G, thr = synth.request(w, r)
        req = oracle.Request.new(prompt, G, w.block, thr, cfg.mask_id)
        L = req.seq_len
        req.cache_k = [np.zeros((L, cfg.n_kv_heads, cfg.head_dim))]
        req.cache_v = [np.zeros((L, cfg.n_kv_heads, cfg.head_dim))]
        h = oracle.embed_rows(cfg, oracle.Weights(g, layers=[]), req, 0, L)
        states.append([w, r, req, h])
    for l in range(cfg.n_layers):
        t1 = time.time()
        lw = gen_layer(pool, cfg, l)
        t2 = time.time()
        for st in states:
            req = st[2]
            st[3] = oracle.layer_forward(cfg, lw, st[3], 0, req.seq_len,
                                         req.cache_k[0], req.cache_v[0])
        log(f"{cfg.name}: layer {l} drawn {t2 - t1:.0f}s, forward {time.time() - t2:.0f}s")
    W = oracle.Weights(g, layers=[])
    raws = []
    for w, r, req, h in states:
        s, e = req.block_bounds
        A = np.nonzero(req.mask[s:e])[0] + s
        raws.append((A, oracle.head_logits(cfg, W, h[A], 1.0)))
    pooled = np.concatenate([z for _, z in raws])
    tau, inv_tau, achieved, k, n = oracle.calibrate(pooled, 0.9, 0.3)
    log(f"{cfg.name}: tau {tau:.6g} inv_tau {float(inv_tau):.8g} share {achieved:.3f} ({k}/{n})")
    reqs_out = []
    for (w, r, req, h), (A, z) in zip(states, raws):
        zs = z * float(inv_tau)
        conf, tok = oracle.confidence(zs)
        top2 = np.sort(zs, axis=1)[:, -2:]
        sel = oracle.select_unmask(conf, req.gamma)
        reqs_out.append({
            "workload": w.name, "request": r, "prompt_len": req.prompt_len,
            "gen_len": req.gen_len, "threshold": req.gamma,
            "positions": A.tolist(), "conf": conf.tolist(), "tok": tok.tolist(),
            "top2_gap": (top2[:, 1] - top2[:, 0]).tolist(),
            "max_abs_logit": np.abs(zs).max(axis=1).tolist(),
            "unmasked": A[sel].tolist(),
            "logit_stride": LOGIT_STRIDE,
            "logits_sample": np.round(zs[:, ::LOGIT_STRIDE], 6).tolist() if len(A) <= 4 else
                             np.round(zs[:4, ::LOGIT_STRIDE], 6).tolist(),
        })
    return {"model": cfg.to_dict(), "tau": tau, "inv_tau": float(inv_tau),
            "share_above": achieved, "k": k, "n": n, "calibration_threshold": 0.9,
            "requests": reqs_out}


def tiny():
    """Tiny fp32 model: calibration plus the whole generation of its workload."""
    cfg = synth.TINY_FP32
    W = oracle.Weights.from_dict(synth.model_weights(cfg))
    prompt, G, thr = synth.request(synth.C1, 0)
    req = oracle.Request.new(prompt, G, synth.C1.block, thr, cfg.mask_id)
    h, rows, _ = oracle.step_forward(cfg, W, req, "none")
    s, e = req.block_bounds
    A = np.nonzero(req.mask[s:e])[0] + s
    tau, inv_tau, achieved, k, n = oracle.calibrate(oracle.head_logits(cfg, W, h[A], 1.0))
    reqs, trace = oracle.generate(cfg, W, [prompt], [G], [thr], synth.C1.block, "none",
                                  float(inv_tau))
    steps = []
    for st in trace:
        res = st[0][1]
        steps.append({"positions": res.positions.tolist(), "tokens": res.tokens.tolist(),
                      "conf": res.conf.tolist(),
                      "masked_positions": res.masked_positions.tolist(),
                      "masked_conf": res.masked_conf.tolist()})
    return {"model": cfg.to_dict(), "workload": synth.C1.name, "tau": tau,
            "inv_tau": float(inv_tau), "share_above": achieved, "k": k, "n": n,
            "n_steps": len(trace), "final_tokens": reqs[0].tokens.tolist(), "steps": steps}


def main(which):
    def log(m):
        print(m, flush=True)
    if "tiny" in which:
        out = tiny()
        with open(os.path.join(HERE, "tiny_fp32.json"), "w") as f:
            json.dump(out, f)
        log(f"tiny: tau {out['tau']:.6g} steps {out['n_steps']}")
    nproc = int(os.environ.get("GOLDEN_PROCS", "8"))
    if "mha" in which:
        with Pool(nproc) as pool:
            out = run_model(synth.MHA_8B, [(synth.C2, 0), (synth.C3_DUAL, 0), (synth.C4, 0)],
                            pool, log)
        with open(os.path.join(HERE, "mha_8b_step1.json"), "w") as f:
            json.dump(out, f)
    if "gqa" in which:
        with Pool(nproc) as pool:
            out = run_model(synth.GQA_7B, [(synth.C5, r) for r in range(4)], pool, log)
        with open(os.path.join(HERE, "gqa_7b_step1.json"), "w") as f:
            json.dump(out, f)


if __name__ == "__main__":
    main(sys.argv[1:] or ["tiny"])
