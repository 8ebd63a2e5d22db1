#!/usr/bin/env python3
"""Denoising-step throughput on one MI355X.

Default workload: the largest single-GPU configuration, the bf16 GQA model
shaped like Dream-7B (28 layers, d 3584, 28 query / 4 key-value heads of 128,
SwiGLU 18944, vocab 152064; synthetic N(0, 0.02) weights), batch 64, each
request 512 random prompt tokens + 512 [MASK] tokens decoded in blocks of 64
with a dual KV cache (the first step of every block recomputes the whole
sequence and rewrites the request's cache, the other steps recompute the
block only), threshold 0.9, logits scaled by the calibrated 1/tau. One step =
one dlm_denoise_step call over the whole batch (embedding, every layer, fused
LM head and confidence, unmask) plus the per-step read-back of the unmask
counts. A finished request is replaced at once (the same prompt again, or the
slot's next request for the heterogeneous workload), so the batch stays full
and requests at different blocks mix recompute and cache steps in one step.

--workload selects the other configurations (the single-request no-cache
step of the MHA model, batch 8 with prefix or dual cache, the heterogeneous
batch of 32).

Prints one JSON line: steps/s (value), unmasked tokens/s, the roofline of the
dominant kernel (in-library HIP events on the launch stream over the timed
region), the whole-step roofline, the latency and roofline of a refresh step
of the whole batch (timed after the timed region, with a cache), and the CPU
oracle timed on a bounded sample.
"""
from __future__ import annotations

import argparse
import dataclasses
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0
PEAK_F32_TFLOPS = 157.3
PEAK_HBM_GBS = 8000.0
GOLDEN = {"mha-8b": "mha_8b_step1.json", "gqa-7b": "gqa_7b_step1.json",
          "tiny-fp32": "tiny_fp32.json"}


def load_inv_tau(model_name: str):
    path = os.path.join(ROOT, "tests", "golden", GOLDEN[model_name])
    with open(path) as f:
        return float(json.load(f)["inv_tau"]), os.path.relpath(path, ROOT)


def measured_traffic(kernel_class: str, workload: str):
    """HBM bytes per launch of a kernel class on a workload from the committed
    rocprofv3 counter summary (profiles/traffic_<class>_<workload>.json), or
    None when there is none or the kernel's sources changed since the counters
    were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel_class}_{workload}.json")
    if not os.path.exists(path):
        return None, None
    with open(path) as f:
        t = json.load(f)
    src = b"".join(open(os.path.join(ROOT, p), "rb").read() for p in t["source_files"])
    if hashlib.sha256(src).hexdigest() != t["source_sha256"]:
        return None, os.path.relpath(path, ROOT) + " (stale: kernel changed)"
    return float(t["hbm_bytes_per_launch"]), os.path.relpath(path, ROOT)


def launched_rows(dreqs, mode, refresh_flag):
    """(recomputed rows, keys) of each request of a step already enqueued,
    from its request descriptors (refresh_flag: the descriptor's recompute bit)."""
    out = []
    for d in dreqs:
        if d.flags & refresh_flag:
            out.append((d.seq_len, d.seq_len))
        elif mode == "dual":
            out.append((d.block_len, d.seq_len))
        else:
            out.append((d.seq_len - d.block_start, d.seq_len))
    return out


def class_work(shape, rows, m_rows):
    """Algorithmic FLOPs and HBM bytes of each kernel class in one step
    (all layers), given per-request (recomputed rows, keys) and LM-head rows."""
    d, dh, hq, hkv, ffn, V, nl = (shape.d_model, shape.head_dim, shape.n_q_heads,
                                  shape.n_kv_heads, shape.d_ffn, shape.vocab, shape.n_layers)
    es = 2 if shape.dtype == "bf16" else 4
    qkv = (hq + 2 * hkv) * dh
    qd = hq * dh
    N = sum(n for n, _ in rows)
    qk = sum(n * L for n, L in rows)
    keys = sum(L for _, L in rows)
    return {
        "gemm_qkv": (nl * 2.0 * N * d * qkv, nl * (es * (qkv * d + N * d) + 4.0 * N * qkv)),
        "gemm_o": (nl * 2.0 * N * qd * d, nl * (es * (d * qd + N * qd) + 8.0 * N * d)),
        "gemm_gate_up_swiglu": (nl * 2.0 * N * d * 2 * ffn,
                                nl * es * (2.0 * ffn * d + N * d + N * ffn)),
        "gemm_down": (nl * 2.0 * N * ffn * d, nl * (es * (d * ffn + N * ffn) + 8.0 * N * d)),
        "attention": (nl * 4.0 * qk * hq * dh, nl * es * (2.0 * N * qd + 2.0 * keys * hkv * dh)),
        "lm_head": (2.0 * m_rows * d * V, es * (V * d + m_rows * d)),
    }


def step_work(shape, rows, m_rows):
    """Whole-step algorithmic FLOPs and bytes: weights read once, every key and
    value read once and every recomputed row's written once, logits never stored."""
    d, dh, hq, hkv, ffn, V, nl = (shape.d_model, shape.head_dim, shape.n_q_heads,
                                  shape.n_kv_heads, shape.d_ffn, shape.vocab, shape.n_layers)
    es = 2 if shape.dtype == "bf16" else 4
    p_lay = d * (hq + 2 * hkv) * dh + hq * dh * d + 3 * d * ffn
    N = sum(n for n, _ in rows)
    F = 2.0 * N * nl * p_lay + 4.0 * nl * hq * dh * sum(n * L for n, L in rows) \
        + 2.0 * m_rows * d * V
    kv_row = 2 * nl * hkv * dh * es
    B = es * (nl * p_lay + V * d) + kv_row * (sum(L for _, L in rows) + N)
    return F, B


def cpu_baseline(cfg, tensors, w, inv_tau, n_sample_layers, n_sample_reqs, rows_per_step,
                 masked_per_step):
    """Time the oracle (fp64 NumPy) on a bounded sample of the workload's step and
    scale it to one step of the timed region.

    The sample: the rows the workload's steady step recomputes for
    n_sample_reqs requests (the whole sequence without a cache; the active
    block with a dual cache; block and suffix with a prefix cache; keys over
    the whole slot) through the first n_sample_layers layers, plus the LM head
    and confidence of their block rows. The oracle's cost is linear in the
    recomputed rows (every row attends over its whole slot), so the step time
    is (layer time per sampled row) x (recomputed rows per timed step) x
    n_layers / n_sample_layers + (head time per row) x (masked rows per timed
    step)."""
    import oracle
    import synth
    try:
        from threadpoolctl import threadpool_info
        threads = max([t.get("num_threads", 1) for t in threadpool_info()] or [1])
    except Exception:
        threads = None
    f = lambda t: t.float().cpu().numpy()
    dh = cfg.head_dim
    qd, kd = cfg.n_q_heads * dh, cfg.n_kv_heads * dh

    def host_layer(l):
        # copied to the host one layer at a time (not timed), so the sample's
        # memory stays at about one layer of fp32 weights
        t = tensors["layers"][l]
        qkv, gu = f(t["w_qkv"]), f(t["w_gate_up"])
        return {"wq": qkv[:qd], "wk": qkv[qd:qd + kd], "wv": qkv[qd + kd:],
                "wo": f(t["w_o"]), "wg": gu[:cfg.d_ffn], "wu": gu[cfg.d_ffn:],
                "wd": f(t["w_down"]), "attn_norm": f(t["attn_norm"]),
                "ffn_norm": f(t["ffn_norm"])}

    W = oracle.Weights({"embed": f(tensors["embed"]), "lm_head": f(tensors["lm_head"]),
                        "final_norm": f(tensors["final_norm"])}, layer_fn=host_layer,
                       n_layers=n_sample_layers)
    mode = w.cache_mode
    reqs, rows, hs = [], [], []
    t_layers = 0.0
    for i in range(n_sample_reqs):
        prompt, G, _ = synth.request(w, i)
        prompt = prompt % cfg.vocab
        req = oracle.Request.new(prompt, G, w.block, 0.9, cfg.mask_id)
        oracle.ensure_cache(cfg, req, n_sample_layers)
        # the mode's steady step: a cache step of block 0 (its cached rows are
        # what the last recompute step wrote; their values do not change the
        # cost), or the whole sequence without a cache
        r0, r1 = oracle.recompute_rows(req, mode, mode == "none")
        t0 = time.perf_counter()
        hs.append(oracle.embed_rows(cfg, W, req, r0, r1))
        t_layers += time.perf_counter() - t0
        reqs.append(req)
        rows.append((r0, r1))
    for l in range(n_sample_layers):
        Wl = W.layer(l)
        ta = time.perf_counter()
        for i, req in enumerate(reqs):
            hs[i] = oracle.layer_forward(cfg, Wl, hs[i], rows[i][0], rows[i][1],
                                         req.cache_k[l], req.cache_v[l])
        t_layers += time.perf_counter() - ta
        del Wl
    t1 = time.perf_counter()
    n_head = 0
    for req, h, (r0, _) in zip(reqs, hs, rows):
        s, e = req.block_bounds
        z = oracle.head_logits(cfg, W, h[s - r0:e - r0], inv_tau)
        conf, tok = oracle.confidence(z)
        oracle.select_unmask(conf, 0.9)
        n_head += e - s
    t_head = time.perf_counter() - t1
    n_rows = sum(b - a for a, b in rows)
    t_step = (t_layers / n_rows * rows_per_step * cfg.n_layers / n_sample_layers
              + t_head / n_head * masked_per_step)
    return {"value": 1.0 / t_step, "unit": "steps/s",
            "cores": len(os.sched_getaffinity(0)), "blas_threads": threads, "kind": "oracle",
            "sample": (f"{n_sample_reqs} request(s) x {n_rows // n_sample_reqs} recomputed rows "
                       f"({mode}-cache steady step, fp64 NumPy) through {n_sample_layers} of "
                       f"{cfg.n_layers} layers + LM head/confidence of {n_head} rows; "
                       f"extrapolated linearly to the timed steps' mean of {rows_per_step:.0f} "
                       f"recomputed and {masked_per_step:.0f} masked rows per step over all "
                       f"layers"),
            "measured_s": t_layers + t_head}


WORKLOADS = {"c2": "C2", "c3-dual": "C3_DUAL", "c3-prefix": "C3_PREFIX", "c4": "C4",
             "c5": "C5"}


def measure_ceilings(torch, dlm):
    """Measured chip ceilings: a loop of independent bf16 MFMAs on every CU and
    a 1 GiB device copy (read + write), best of 3 each, HIP events on the
    launch stream."""
    st = torch.cuda.current_stream()
    out = torch.empty(2048 * 4, dtype=torch.float32, device="cuda:0")
    src = torch.ones(1 << 28, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    best_f, best_c = 0.0, 0.0
    for _ in range(4):                     # first pass is a warm-up
        e0, e1, e2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
        e0.record(st)
        flop = dlm.ceiling_mfma(2048, 512, out.data_ptr(), st.cuda_stream)
        e1.record(st)
        dlm.ceiling_copy(src.data_ptr(), dst.data_ptr(), src.numel() * 4, st.cuda_stream)
        e2.record(st)
        e2.synchronize()
        best_f = max(best_f, flop / (e0.elapsed_time(e1) * 1e-3) / 1e12)
        best_c = max(best_c, 2 * src.numel() * 4 / (e1.elapsed_time(e2) * 1e-3) / 1e9)
    assert dst[-1].item() == 1.0
    del src, dst, out
    torch.cuda.empty_cache()
    return {"mfma_bf16_tflops": best_f, "copy_gbs": best_c,
            "method": "2048 blocks x 4 waves x 16384 v_mfma_f32_16x16x32_bf16 (8 independent "
                      "accumulators per wave); "
                      "1 GiB device copy, 16-byte lanes (read + write bytes)"}


def serve_main(args, w, cfg, inv_tau):
    """Continuous batching of a Poisson trace on one GPU with the threshold
    controller (latency profile and steps-per-block table measured earlier on
    the same kind of GPU and committed under profiles/)."""
    import synth
    import synth.device as sdev
    from paper_2606_29094_amd import engine, serving
    from paper_2606_29094_amd.profiling import StepTable
    ctl_file = os.path.join(ROOT, "profiles", "controller_mha8b.json")
    meas = json.load(open(ctl_file))
    table = StepTable.from_json(meas["step_table"])
    gammas = table.gammas
    if args.fixed_threshold is not None:
        g = args.fixed_threshold
        i = min(range(len(gammas)), key=lambda j: abs(gammas[j] - g))
        table = StepTable([gammas[i]], [table.steps_per_block[i]], table.block)
        gammas = [gammas[i]]
    mcfg = synth.MHA_8B
    t = sdev.model_tensors(mcfg)
    model = engine.DeviceModel(engine.ModelShape.of(mcfg), t, inv_tau)
    slots, prange, gens = 32, (128, 2048), (128, 256)
    max_len = prange[1] + max(gens)
    eng = engine.Engine(model, slots, max_len, "dual", max_rows=16384)
    scfg = serving.ServeConfig(gammas, 32, "dual", max_step_tokens=16384)
    srv = serving.Server(eng, scfg, meas["latency_profile"], table, mcfg.mask_id)
    trace = serving.poisson_trace(args.serve, args.serve_requests, 7, prange, gens, args.slo,
                                  mcfg.vocab)
    # warm-up: a few requests outside the measured trace
    warm = serving.poisson_trace(100.0, 4, 99, prange, gens, 1e9, mcfg.vocab)
    serving.Server(eng, scfg, meas["latency_profile"], table, mcfg.mask_id).run(warm)
    rep = srv.run(trace)
    print(json.dumps({"metric": "serving: SLO attainment / tokens/s", "value": rep["slo_attainment"],
                      "unit": "fraction of requests within SLO", "report": rep,
                      "config": {"workload": "poisson-serve-mha8b-dual", "rate_per_s": args.serve,
                                 "requests": args.serve_requests, "slo_s": args.slo,
                                 "thresholds": gammas, "slots": slots,
                                 "max_step_tokens": 16384, "prompt_range": list(prange),
                                 "gen_choices": list(gens), "inv_tau": inv_tau,
                                 "controller_measurements": os.path.relpath(ctl_file, ROOT)},
                      "data": "synthetic"}), flush=True)


def step_breakdown(per_step):
    """Per-step-type latency and the distributions of recomputed rows and
    refreshing requests over the timed steps."""
    import numpy as np
    kinds = {}
    for kind, dt, n, rf in per_step:
        kinds.setdefault(kind, []).append((dt, n, rf))
    lat = {}
    for kind, v in kinds.items():
        t = np.array([x[0] for x in v]) * 1e3
        lat[kind] = {"steps": len(v), "mean_ms": float(t.mean()), "median_ms": float(np.median(t)),
                     "min_ms": float(t.min()), "max_ms": float(t.max()),
                     "mean_rows": float(np.mean([x[1] for x in v]))}
    n = np.array([x[2] for x in per_step])
    rf = np.array([x[3] for x in per_step])
    q = [0, 25, 50, 75, 100]
    dist = {"rows_quantiles": {str(k): float(v) for k, v in zip(q, np.percentile(n, q))},
            "refresh_requests_quantiles": {str(k): float(v) for k, v in
                                           zip(q, np.percentile(rf, q))},
            "refresh_requests_hist": {str(int(k)): int(c) for k, c in
                                      zip(*np.unique(rf, return_counts=True))}}
    return lat, dist


def main():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None,
                    help="timed steps (default 40; 256 for c4)")
    ap.add_argument("--warmup", type=int, default=None,
                    help="untimed warm-up steps (default 5; 64 for c4)")
    ap.add_argument("--workload", default="c5", choices=sorted(WORKLOADS))
    ap.add_argument("--threshold", type=float, default=None,
                    help="override every request's threshold (the GQA sweep)")
    ap.add_argument("--cpu-layers", type=int, default=None,
                    help="layers of the CPU oracle sample (0 disables the CPU baseline; default: "
                         "24 for the single-request no-cache workload, every layer otherwise)")
    ap.add_argument("--cpu-requests", type=int, default=None,
                    help="requests of the CPU oracle sample (default: 1 without a cache, 4 "
                         "with one)")
    ap.add_argument("--inv-tau", type=float, default=None,
                    help="override the stored calibrated 1/tau")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="only run 10 device-to-device copies of MIB MiB (calibrates the "
                         "HBM byte counters) and exit")
    ap.add_argument("--sample-every", type=int, default=0,
                    help="time one launch in this many of the dominant kernel in the timed "
                         "steps (default 3: a third of the layers, rotating)")
    ap.add_argument("--profile-steps", type=int, default=10,
                    help="untimed steps after the warm-up with every kernel class timed "
                         "(per-class breakdown, choice of the dominant kernel)")
    ap.add_argument("--no-profile", action="store_true",
                    help="time without the per-kernel event records")
    ap.add_argument("--stats", action="store_true",
                    help="also compute the per-request confidence statistics in every step")
    ap.add_argument("--latency-profile", action="store_true",
                    help="only measure per-step latency over batch sizes in tokens (recompute "
                         "and dual-cache steps) for the workload's model and print it")
    ap.add_argument("--serve", type=float, default=None, metavar="RATE",
                    help="run the single-GPU serving loop on a Poisson trace of RATE requests/s "
                         "(heterogeneous MHA-8B requests, dual cache, controller thresholds) "
                         "and print its report")
    ap.add_argument("--serve-requests", type=int, default=200)
    ap.add_argument("--slo", type=float, default=10.0, help="latency SLO of --serve (s)")
    ap.add_argument("--fixed-threshold", type=float, default=None,
                    help="--serve with this single threshold instead of the controller's choice")
    ap.add_argument("--tp-share", type=int, default=1, metavar="N",
                    help="run one tensor-parallel rank's share of the model on this GPU: "
                         "1/N of the query/key-value heads, FFN columns and vocabulary at the "
                         "same rows (the rank's compute only; no collectives)")
    ap.add_argument("--refresh-steps", type=int, default=None,
                    help="after the timed steps, time this many steps in which every request "
                         "refreshes (recomputes its whole sequence); default 2 with a cache, "
                         "0 without")
    ap.add_argument("--no-ceilings", action="store_true",
                    help="skip the measured MFMA-loop and copy ceilings")
    args = ap.parse_args()
    # the heterogeneous stream discards 64 warm-up steps and times 256
    d_steps, d_warm = (256, 64) if args.workload == "c4" else (40, 5)
    args.steps = d_steps if args.steps is None else args.steps
    args.warmup = d_warm if args.warmup is None else args.warmup
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}): the path is "
              "data-parallel over requests with no exchange, so N GPUs run N independent "
              "copies of this benchmark.", file=sys.stderr)
        sys.exit(2)

    import torch
    if args.copy_probe:
        n = args.copy_probe << 20
        x = torch.ones(n, dtype=torch.uint8, device="cuda:0")
        y = torch.empty_like(x)
        for _ in range(10):
            y.copy_(x)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes": n, "copies": 10}))
        return
    import synth
    import synth.device as sdev
    from paper_2606_29094_amd import dlm, engine

    ceilings = None if args.no_ceilings else measure_ceilings(torch, dlm)

    w = getattr(synth, WORKLOADS[args.workload])
    cfg = w.model
    if args.inv_tau is not None:
        inv_tau, tau_src = args.inv_tau, "command line"
    else:
        inv_tau, tau_src = load_inv_tau(cfg.name)
    tp = args.tp_share
    if tp > 1:
        # one rank of tensor parallelism: heads, FFN columns and vocabulary
        # split N ways (QKV / gate-up column-parallel, O / down row-parallel,
        # vocabulary-parallel head); prompt tokens are folded into the shard's
        # vocabulary (the rank's work does not depend on their values)
        if cfg.n_q_heads % tp or cfg.n_kv_heads % tp or cfg.d_ffn % (16 * tp) or cfg.vocab % tp:
            raise SystemExit(f"--tp-share {tp} does not divide the {cfg.name} shapes")
        cfg = dataclasses.replace(cfg, name=f"{cfg.name}-tp{tp}-rank", n_q_heads=cfg.n_q_heads // tp,
                                  n_kv_heads=cfg.n_kv_heads // tp, d_ffn=cfg.d_ffn // tp,
                                  vocab=cfg.vocab // tp)
        w = dataclasses.replace(w, name=f"{w.name}-tp{tp}-rank", model=cfg)
    if args.serve is not None:
        serve_main(args, w, cfg, inv_tau)
        return
    if args.latency_profile:
        from paper_2606_29094_amd import profiling
        lp = profiling.latency_profile(cfg, inv_tau)
        print(json.dumps({"metric": "per-step latency over batch size (tokens)",
                          "unit": "s", "latency_profile": lp, "data": "synthetic",
                          "config": {"workload": w.name, "inv_tau": inv_tau}}), flush=True)
        return
    tensors = sdev.model_tensors(cfg)
    shape = engine.ModelShape.of(cfg)
    model = engine.DeviceModel(shape, tensors, inv_tau)

    # request stream per slot: the fixed workloads repeat their requests, the
    # heterogeneous one walks through request ids slot, slot + B, ...
    B = w.batch
    hetero = w.prompt_range is not None
    next_id = [b for b in range(B)]

    def make(slot):
        rid = next_id[slot]
        prompt, G, thr = synth.request(w, rid)
        if tp > 1:
            prompt = prompt % cfg.vocab
        if hetero:
            next_id[slot] += B
        if args.threshold is not None:
            thr = args.threshold
        return engine.Request(prompt, G, w.block, thr)

    if hetero:
        max_len = w.prompt_range[1] + max(w.gen_choices)
    else:
        max_len = w.prompt_len + w.gen_len
    eng = engine.Engine(model, B, max_len, w.cache_mode, max_rows=B * max_len, stats=args.stats)
    slots = []
    for b in range(B):
        r = make(b)
        eng.admit(r, cfg.mask_id)
        slots.append(r)

    stats = {"masked": 0, "unmasked": 0, "F": 0.0, "B": 0.0, "refresh_reqs": 0, "rows": 0,
             "cls": {}, "per_step": [], "req_steps": []}

    def account_step(rows, m, refresh):
        stats["masked"] += m
        stats["refresh_reqs"] += refresh
        stats["rows"] += sum(n for n, _ in rows)
        F, Bb = step_work(shape, rows, m)
        stats["F"] += F
        stats["B"] += Bb
        for k, (f, bb) in class_work(shape, rows, m).items():
            a = stats["cls"].setdefault(k, [0.0, 0.0])
            a[0] += f
            a[1] += bb

    prof_work = {}                        # class -> [flops, bytes] over the profile steps

    def one_step(account, prof_acc=None):
        for b in range(B):
            if slots[b].done:
                if account:
                    stats["req_steps"].append((slots[b].steps, slots[b].gen_len))
                eng.release(slots[b])
                slots[b] = make(b)
                eng.admit(slots[b], cfg.mask_id)
        ts = time.perf_counter()
        dreqs = eng.enqueue_step(slots)
        # host bookkeeping while the GPU runs the step (from the descriptors
        # the step was launched with; a step changes no block or mask count
        # on the host before its read-back)
        rows = launched_rows(dreqs, w.cache_mode, dlm.DLM_REQ_REFRESH)
        m = sum(r.masked_in_block for r in slots)
        refresh = sum(1 for d in dreqs if d.flags & dlm.DLM_REQ_REFRESH)
        if account:
            account_step(rows, m, refresh)
        if prof_acc is not None:
            for k, (f, bb) in class_work(shape, rows, m).items():
                a = prof_acc.setdefault(k, [0.0, 0.0])
                a[0] += f
                a[1] += bb
        counts = eng.finish_step(slots)   # read-back of the counts (synchronises)
        dt = time.perf_counter() - ts
        if account:
            if w.cache_mode == "none":
                kind = "no-cache"
            elif refresh == 0:
                kind = "cache"
            elif refresh == len(slots):
                kind = "refresh"
            else:
                kind = "mixed"
            stats["per_step"].append((kind, dt, sum(n for n, _ in rows), refresh))
            stats["unmasked"] += sum(counts)

    # warm-up (untimed), then untimed profile steps with every kernel class
    # timed (the per-class breakdown of the steady state and the dominant
    # class); the timed steps then time every third launch of the dominant
    # class (rotating through the layers). A timed launch carries its two
    # events in its own dispatch (no extra stream commands); timing every
    # launch still cost ~1 % of the step
    for _ in range(args.warmup):
        one_step(False)
    torch.cuda.synchronize()
    warm_prof = {}
    dom = None
    if not args.no_profile:
        dlm.profile_enable(model.handle, True)
        for _ in range(args.profile_steps):
            one_step(False, prof_work)
        torch.cuda.synchronize()
        dlm.profile_enable(model.handle, False)
        warm_prof = dlm.profile_read(model.handle)
        timed_cls = [k for k in warm_prof if k in ("gemm_qkv", "gemm_o", "gemm_gate_up_swiglu",
                                                   "gemm_down", "attention", "lm_head")]
        if timed_cls:
            dom = max(timed_cls, key=lambda k: warm_prof[k][1])
            every = args.sample_every if args.sample_every > 0 else 3
            dlm.profile_sample(model.handle, every)
            dlm.profile_enable(model.handle, True, dom)
    t0 = time.perf_counter()
    for _ in range(args.steps):
        one_step(True)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    prof = {}
    if not args.no_profile:
        dlm.profile_enable(model.handle, False)
        prof = dlm.profile_read(model.handle)

    # refresh steps (every request recomputes its whole sequence), after the
    # timed region: one untimed, then args.refresh_steps timed one by one
    n_refresh = args.refresh_steps
    if n_refresh is None:
        n_refresh = 0 if w.cache_mode == "none" else 2
    refresh_step = None
    if n_refresh > 0:
        ref_t, ref_F, ref_B, ref_rows = [], 0.0, 0.0, 0
        for i in range(n_refresh + 1):
            for b in range(B):
                if slots[b].done:
                    eng.release(slots[b])
                    slots[b] = make(b)
                    eng.admit(slots[b], cfg.mask_id)
            rows = [(r.seq_len, r.seq_len) for r in slots]
            m = sum(r.masked_in_block for r in slots)
            torch.cuda.synchronize()
            ts = time.perf_counter()
            eng.enqueue_step(slots, force_refresh=True)
            eng.finish_step(slots)
            dt = time.perf_counter() - ts
            if i > 0:
                F, Bb = step_work(shape, rows, m)
                ref_t.append(dt)
                ref_F += F
                ref_B += Bb
                ref_rows += sum(n for n, _ in rows)
        t_ref = sum(ref_t) / len(ref_t)
        pk = PEAK_BF16_TFLOPS if shape.dtype == "bf16" else PEAK_F32_TFLOPS
        F1, B1 = ref_F / len(ref_t), ref_B / len(ref_t)
        refresh_step = {"steps": len(ref_t), "mean_ms": 1e3 * t_ref, "rows": ref_rows / len(ref_t),
                        "flop": F1, "bytes": B1, "tflops": F1 / t_ref / 1e12,
                        "frac_mfma": F1 / t_ref / (pk * 1e12),
                        "frac_hbm": B1 / t_ref / (PEAK_HBM_GBS * 1e9)}
    elapsed = t1 - t0
    t_step = elapsed / args.steps
    peak = PEAK_BF16_TFLOPS if shape.dtype == "bf16" else PEAK_F32_TFLOPS
    ridge = peak * 1e12 / (PEAK_HBM_GBS * 1e9)

    # per-class breakdown from the profile steps (all classes timed there)
    kernels = {}
    warm_total = sum(v[1] for v in warm_prof.values()) or 1.0
    for name, (calls, tot, _) in warm_prof.items():
        kernels[name] = {"calls": calls, "avg_us": 1e3 * tot / max(calls, 1),
                         "share_of_kernel_time": tot / warm_total}
        if name in prof_work and calls > 0 and tot > 0:
            # achieved rates of the profile steps: the class's algorithmic work
            # over those steps / its summed event time
            f, bb = prof_work[name]
            kernels[name].update({"tflops": f / (tot * 1e-3) / 1e12,
                                  "gbs": bb / (tot * 1e-3) / 1e9,
                                  "frac_mfma": f / (tot * 1e-3) / (peak * 1e12),
                                  "frac_hbm": bb / (tot * 1e-3) / (PEAK_HBM_GBS * 1e9)})
    roof = None
    if dom is not None and dom in prof and dom in stats["cls"]:
        calls, tot, launches = prof[dom]              # timed launches, their ms, all launches
        F, Bb = stats["cls"][dom]
        F1, B1 = F / launches, Bb / launches           # per launch
        avg_s = tot / calls * 1e-3
        traffic, traffic_src = (measured_traffic(dom, w.name) if tp == 1 else (None, None))
        if F1 / B1 >= ridge:
            achieved = F1 / avg_s / 1e12
            roof = {"kernel": dom, "bound": "mfma", "achieved": achieved, "peak": peak,
                    "unit": "TFLOP/s", "frac": achieved / peak, "traffic": traffic,
                    "traffic_source": traffic_src, "algorithmic_bytes": B1,
                    "flop_per_launch": F1, "avg_launch_us": avg_s * 1e6,
                    "timed_launches": calls, "launches": launches}
        else:
            achieved = B1 / avg_s / 1e9
            roof = {"kernel": dom, "bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS,
                    "unit": "GB/s", "frac": achieved / PEAK_HBM_GBS, "traffic": traffic,
                    "traffic_source": traffic_src, "bytes_per_launch": B1,
                    "avg_launch_us": avg_s * 1e6, "timed_launches": calls, "launches": launches}
    Fs, Bs = stats["F"] / args.steps, stats["B"] / args.steps
    step_roof = {"tflops": Fs / t_step / 1e12, "gbs": Bs / t_step / 1e9,
                 "frac_mfma": Fs / t_step / (peak * 1e12),
                 "frac_hbm": Bs / t_step / (PEAK_HBM_GBS * 1e9),
                 "bound": "mfma" if Fs / Bs >= ridge else "hbm",
                 "flop_per_step": Fs, "bytes_per_step": Bs}

    cpu = None
    cpu_layers = args.cpu_layers
    if cpu_layers is None:
        cpu_layers = min(24, cfg.n_layers) if w.cache_mode == "none" else cfg.n_layers
    if cpu_layers > 0:
        n_req = args.cpu_requests or (1 if w.cache_mode == "none" else 4)
        cpu = cpu_baseline(cfg, tensors, w, inv_tau, min(cpu_layers, cfg.n_layers), n_req,
                           stats["rows"] / args.steps, stats["masked"] / args.steps)

    lat, dist = step_breakdown(stats["per_step"])
    rs = stats["req_steps"]
    req = ({"completed": len(rs), "mean_steps": sum(x[0] for x in rs) / len(rs),
            "mean_tokens_per_step": sum(x[1] for x in rs) / sum(x[0] for x in rs)}
           if rs else {"completed": 0})
    if ceilings is not None:
        ceilings["step_frac_of_measured_mfma"] = Fs / t_step / 1e12 / ceilings["mfma_bf16_tflops"]
        if roof is not None:
            ceilings["dominant_frac_of_measured"] = roof["achieved"] / (
                ceilings["mfma_bf16_tflops"] if roof["unit"] == "TFLOP/s" else ceilings["copy_gbs"])

    out = {
        "metric": "denoise steps/s + unmasked tokens/s per MI355X; % MFMA / HBM roofline",
        "value": args.steps / elapsed,
        "unit": "steps/s",
        "unmasked_tokens_per_s": stats["unmasked"] / elapsed,
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "profile_steps": 0 if args.no_profile else args.profile_steps,
        "ms_per_step": 1e3 * t_step, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16" if shape.dtype == "bf16" else "f32",
        "data": "synthetic",
        "config": {"workload": w.name, "batch": B, "tp_share": tp,
                   "prompt_len": w.prompt_len or list(w.prompt_range),
                   "gen_len": w.gen_len or list(w.gen_choices),
                   "block": w.block, "cache": w.cache_mode,
                   "threshold": args.threshold if args.threshold is not None else
                   (list(w.threshold_choices) if hetero else w.threshold),
                   "inv_tau": inv_tau, "inv_tau_source": tau_src,
                   "weights": "synthetic N(0,0.02) seed 0",
                   "avg_recomputed_rows": stats["rows"] / args.steps,
                   "avg_masked_rows": stats["masked"] / args.steps,
                   "avg_refresh_requests": stats["refresh_reqs"] / args.steps,
                   "confidence_stats": bool(args.stats)},
        "roofline": roof,
        "class_work": {k: {"flop": f, "bytes": bb} for k, (f, bb) in stats["cls"].items()},
        "step_roofline": step_roof,
        "step_latency": lat,
        "refresh_step": refresh_step,
        "step_distribution": dist,
        "requests": req,
        "ceilings": ceilings,
        "kernels_profiled": kernels,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
