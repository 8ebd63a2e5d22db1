"""Measurements the threshold controller consumes (paper, "Design Overview":
a one-time profile of per-step latency over batch sizes; "Step Prediction":
remaining-step estimates per candidate threshold).

* latency_profile(): per-step latency of recompute steps and of dual-cache
  steps as a function of the step's batch size in tokens (recomputed rows),
  on synthetic requests of the workload's shapes; the wall time of one
  dlm_denoise_step call including the read-back of the unmask counts, which
  is what a serving loop waits for.
* steps_per_block(): for each candidate threshold, how many denoising steps a
  block takes on synthetic requests (mean, and the mean over blocks of the
  first and the remaining steps), from full generations.
* StepTable.pred_steps_left(): the remaining-step estimate built from those
  measurements: the current block's remaining masked fraction plus the
  blocks still to come, each at the measured mean for the threshold; and the
  recompute steps left (one per block whose recompute has not run yet).

Usage: python -m paper_2606_29094_amd.profiling --model mha-8b --out FILE
"""
from __future__ import annotations

import argparse
import json
import math
import time
from dataclasses import dataclass
from typing import Dict, List, Sequence

import numpy as np


def _model(cfg, inv_tau):
    import synth.device as sdev
    from . import engine
    t = sdev.model_tensors(cfg)
    return engine.DeviceModel(engine.ModelShape.of(cfg), t, inv_tau), t


def _time_steps(eng, reqs, n_warm, n_timed):
    import torch
    for _ in range(n_warm):
        eng.step(reqs)
    torch.cuda.synchronize()
    ts = []
    for _ in range(n_timed):
        t0 = time.perf_counter()
        eng.step(reqs)
        ts.append(time.perf_counter() - t0)
    return float(np.median(ts))


def latency_profile(cfg, inv_tau: float, recompute_tokens: Sequence[int] = (256, 512, 1024, 2048,
                                                                               4096, 8192, 16384),
                    cache_batches: Sequence[int] = (1, 2, 4, 8, 16, 32, 64),
                    seq_len: int = 1280, block: int = 32, n_timed: int = 5) -> dict:
    """Recompute curve: B requests of min(tokens, 2048) positions each
    (no-cache mode, every step recomputes all); cache curve: B requests of
    seq_len positions in dual-cache mode, block `block`, after their
    recompute step (tokens = block * B). Threshold 1 keeps every step to one
    unmasked token per request, so repeated steps stay the same kind."""
    from . import engine
    model, _ = _model(cfg, inv_tau)
    rng = np.random.default_rng(0)
    out = {"recompute": {"tokens": [], "latency_s": []}, "cache": {"tokens": [], "latency_s": []}}
    for N in recompute_tokens:
        L = min(N, 2048)
        B = max(1, N // L)
        P = L - 2 * block if L > 2 * block else L // 2
        eng = engine.Engine(model, B, L, "none")
        reqs = []
        for _ in range(B):
            r = engine.Request(rng.integers(0, cfg.vocab - 1, P), L - P, block, 1.0)
            eng.admit(r, cfg.mask_id)
            reqs.append(r)
        out["recompute"]["tokens"].append(B * L)
        out["recompute"]["latency_s"].append(_time_steps(eng, reqs, 2, n_timed))
        eng.close()
    for B in cache_batches:
        P = seq_len - 8 * block
        eng = engine.Engine(model, B, seq_len, "dual")
        reqs = []
        for _ in range(B):
            r = engine.Request(rng.integers(0, cfg.vocab - 1, P), seq_len - P, block, 1.0)
            eng.admit(r, cfg.mask_id)
            reqs.append(r)
        eng.step(reqs)                      # the recompute step of block 0
        out["cache"]["tokens"].append(block * B)
        out["cache"]["latency_s"].append(_time_steps(eng, reqs, 1, n_timed))
        eng.close()
    model.close()
    out.update({"model": cfg.name, "tp": 1, "cache_seq_len": seq_len, "block": block,
                "timing": "median wall time of one step incl. the unmask-count read-back"})
    return out


def steps_per_block(cfg, inv_tau: float, workload, gammas: Sequence[float]) -> dict:
    """Full generations of the workload's first batch at each threshold."""
    import synth
    from . import engine
    model, _ = _model(cfg, inv_tau)
    res = {}
    for g in gammas:
        reqs = []
        L = max(len(synth.request(workload, r)[0]) + synth.request(workload, r)[1]
                for r in range(workload.batch))
        eng = engine.Engine(model, workload.batch, L, workload.cache_mode)
        for r in range(workload.batch):
            prompt, G, _ = synth.request(workload, r)
            q = engine.Request(prompt, G, workload.block, g)
            eng.admit(q, cfg.mask_id)
            reqs.append(q)
        per_block: List[int] = []
        counts = {id(q): 0 for q in reqs}
        while any(not q.done for q in reqs):
            act = [q for q in reqs if not q.done]
            ks = {id(q): q.k for q in act}
            eng.step(act)
            for q in act:
                counts[id(q)] += 1
                if q.k != ks[id(q)]:                 # the block finished this step
                    per_block.append(counts[id(q)])
                    counts[id(q)] = 0
        eng.close()
        res[f"{g:g}"] = {"mean_steps_per_block": float(np.mean(per_block)),
                         "blocks": len(per_block), "max": int(max(per_block)),
                         "min": int(min(per_block))}
    model.close()
    return {"model": cfg.name, "workload": workload.name, "block": workload.block,
            "steps_per_block": res}


@dataclass
class StepTable:
    """Remaining-step estimates from measured steps per block."""
    gammas: List[float]
    steps_per_block: List[float]
    block: int

    @classmethod
    def from_json(cls, d: dict) -> "StepTable":
        items = sorted((float(k), v["mean_steps_per_block"]) for k, v in d["steps_per_block"].items())
        return cls([g for g, _ in items], [s for _, s in items], int(d["block"]))

    def pred_steps_left(self, req) -> List[float]:
        """req: an engine Request (block index k, masked count of the block)."""
        n_blocks = math.ceil(req.gen_len / req.block)
        left_blocks = n_blocks - req.k - 1
        frac = req.masked_in_block / max(req.block_len, 1) if not req.done else 0.0
        return [s * (frac + max(left_blocks, 0)) if not req.done else 0.0
                for s in self.steps_per_block]

    def recomp_steps_left(self, req, mode: str) -> float:
        if req.done:
            return 0.0
        n_blocks = math.ceil(req.gen_len / req.block)
        if mode == "none":
            return float(max(self.pred_steps_left(req)))
        pending_current = 1 if req.refreshed_block != req.block_start else 0
        return float(n_blocks - req.k - 1 + pending_current)


def main():
    import synth
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--model", default="mha-8b", choices=["mha-8b", "gqa-7b"])
    ap.add_argument("--gammas", default="0.5,0.6,0.7,0.8,0.9")
    ap.add_argument("--out", required=True)
    args = ap.parse_args()
    cfg = synth.MHA_8B if args.model == "mha-8b" else synth.GQA_7B
    gold = {"mha-8b": "mha_8b_step1.json", "gqa-7b": "gqa_7b_step1.json"}[args.model]
    import os
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    inv_tau = float(json.load(open(os.path.join(root, "tests", "golden", gold)))["inv_tau"])
    wl = synth.C3_DUAL if args.model == "mha-8b" else synth.C5
    t0 = time.time()
    lp = latency_profile(cfg, inv_tau)
    print(f"latency profile: {time.time() - t0:.1f} s", flush=True)
    sp = steps_per_block(cfg, inv_tau, wl, [float(g) for g in args.gammas.split(",")])
    print(f"steps per block: {time.time() - t0:.1f} s", flush=True)
    with open(args.out, "w") as f:
        json.dump({"latency_profile": lp, "step_table": sp, "inv_tau": inv_tau}, f, indent=1)
    print(json.dumps({"latency_profile": lp, "step_table": sp}))


if __name__ == "__main__":
    main()
