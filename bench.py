#!/usr/bin/env python3
"""Denoising-step throughput on one MI355X.

Workload (default): the bf16 MHA model shaped like LLaDA-8B (32 layers, d 4096,
32 heads of 128, SwiGLU 12288, vocab 126464; synthetic N(0, 0.02) weights),
batch 1, 256 random prompt tokens + 256 [MASK] tokens decoded in blocks of 32,
no cache (every step recomputes all 512 positions), threshold 0.9, logits
scaled by the calibrated 1/tau. One step = one dlm_denoise_step call (the whole
hot path: embedding, 32 layers, fused LM head and confidence, unmask) plus the
per-step readback of the unmask count. When the generation finishes the
request is re-admitted with its prompt and the timing continues.

Prints one JSON line: steps/s (value), unmasked tokens/s, the roofline of the
dominant kernel (HIP events on the launch stream over the timed region), the
whole-step roofline, and the CPU oracle timed on a bounded sample.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0
PEAK_F32_TFLOPS = 157.3
PEAK_HBM_GBS = 8000.0


def load_inv_tau(model_name: str):
    path = os.path.join(ROOT, "tests", "golden",
                        {"mha-8b": "mha_8b_step1.json", "gqa-7b": "gqa_7b_step1.json",
                         "tiny-fp32": "tiny_fp32.json"}[model_name])
    with open(path) as f:
        return float(json.load(f)["inv_tau"]), os.path.relpath(path, ROOT)


def measured_traffic(kernel_class: str):
    """HBM bytes per launch of a kernel class from the committed rocprofv3 counter
    summary (profiles/traffic_<class>.json), or None when there is none or the
    kernel's sources changed since the counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel_class}.json")
    if not os.path.exists(path):
        return None, None
    with open(path) as f:
        t = json.load(f)
    src = b"".join(open(os.path.join(ROOT, p), "rb").read() for p in t["source_files"])
    if hashlib.sha256(src).hexdigest() != t["source_sha256"]:
        return None, os.path.relpath(path, ROOT) + " (stale: kernel changed)"
    return float(t["hbm_bytes_per_launch"]), os.path.relpath(path, ROOT)


def kernel_work(shape, n_rows, seq_len, m_rows):
    """Algorithmic FLOPs and HBM bytes of one launch of each kernel class for a
    single-request no-cache step (n_rows recomputed rows, keys = seq_len,
    m_rows LM-head rows)."""
    d, dh, hq, hkv, ffn, V = (shape.d_model, shape.head_dim, shape.n_q_heads,
                              shape.n_kv_heads, shape.d_ffn, shape.vocab)
    es = 2 if shape.dtype == "bf16" else 4
    qkv = (hq + 2 * hkv) * dh
    qd = hq * dh
    N = n_rows
    w = {
        "gemm_qkv": (2.0 * N * d * qkv, es * (qkv * d + N * d) + 4 * N * qkv),
        "gemm_o": (2.0 * N * qd * d, es * (d * qd + N * qd) + 8 * N * d),
        "gemm_gate_up_swiglu": (2.0 * N * d * 2 * ffn, es * (2 * ffn * d + N * d + N * ffn)),
        "gemm_down": (2.0 * N * ffn * d, es * (d * ffn + N * ffn) + 8 * N * d),
        "attention": (4.0 * N * seq_len * hq * dh, es * (2 * N * qd + 2 * seq_len * hkv * dh)),
        "lm_head": (2.0 * m_rows * d * V, es * (V * d + m_rows * d)),
    }
    return w


def step_work(shape, n_rows, seq_len, m_rows):
    """Whole-step algorithmic FLOPs and bytes (weights read once, KV read and
    written once, logits never stored)."""
    d, dh, hq, hkv, ffn, V, nl = (shape.d_model, shape.head_dim, shape.n_q_heads,
                                  shape.n_kv_heads, shape.d_ffn, shape.vocab, shape.n_layers)
    es = 2 if shape.dtype == "bf16" else 4
    p_lay = d * (hq + 2 * hkv) * dh + hq * dh * d + 3 * d * ffn
    F = 2.0 * n_rows * nl * p_lay + 4.0 * nl * hq * dh * n_rows * seq_len + 2.0 * m_rows * d * V
    kv_row = 2 * nl * hkv * dh * es
    B = es * (nl * p_lay + V * d) + kv_row * (seq_len + n_rows)
    return F, B


def cpu_baseline(cfg, tensors, prompt, G, inv_tau, n_sample_layers):
    """Time the oracle (fp64 NumPy) on a bounded sample of one step: the first
    n_sample_layers layers over all rows plus the LM head and confidence of the
    block's 32 masked rows; scaled to a whole step (layers x n_layers / n)."""
    import numpy as np
    import oracle
    try:
        from threadpoolctl import threadpool_info
        threads = max([t.get("num_threads", 1) for t in threadpool_info()] or [1])
    except Exception:
        threads = None
    f = lambda t: t.float().cpu().numpy()
    d, dh = cfg.d_model, cfg.head_dim
    qd, kd = cfg.n_q_heads * dh, cfg.n_kv_heads * dh
    layers = []
    for l in range(n_sample_layers):
        t = tensors["layers"][l]
        qkv, gu = f(t["w_qkv"]), f(t["w_gate_up"])
        layers.append({"wq": qkv[:qd], "wk": qkv[qd:qd + kd], "wv": qkv[qd + kd:],
                       "wo": f(t["w_o"]), "wg": gu[:cfg.d_ffn], "wu": gu[cfg.d_ffn:],
                       "wd": f(t["w_down"]), "attn_norm": f(t["attn_norm"]),
                       "ffn_norm": f(t["ffn_norm"])})
    W = oracle.Weights({"embed": f(tensors["embed"]), "lm_head": f(tensors["lm_head"]),
                        "final_norm": f(tensors["final_norm"])}, layers=layers)
    req = oracle.Request.new(prompt, G, 32, 0.9, cfg.mask_id)
    L = req.seq_len
    oracle.ensure_cache(cfg, req, n_sample_layers)
    t0 = time.perf_counter()
    h = oracle.embed_rows(cfg, W, req, 0, L)
    for l in range(n_sample_layers):
        h = oracle.layer_forward(cfg, W.layer(l), h, 0, L, req.cache_k[l], req.cache_v[l])
    t1 = time.perf_counter()
    s, e = req.block_bounds
    z = oracle.head_logits(cfg, W, h[s:e], inv_tau)
    conf, tok = oracle.confidence(z)
    oracle.select_unmask(conf, 0.9)
    t2 = time.perf_counter()
    t_step = (t1 - t0) * cfg.n_layers / n_sample_layers + (t2 - t1)
    return {"value": 1.0 / t_step, "unit": "steps/s",
            "cores": len(os.sched_getaffinity(0)), "blas_threads": threads, "kind": "oracle",
            "sample": (f"{n_sample_layers} of {cfg.n_layers} layers of one no-cache step "
                       f"({L} rows, fp64 NumPy) + LM head/confidence of {e - s} rows; layer "
                       f"time scaled x{cfg.n_layers}/{n_sample_layers}"),
            "measured_s": t2 - t0}


def main():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=40)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--cpu-layers", type=int, default=4,
                    help="layers of the CPU oracle sample (0 disables the CPU baseline)")
    ap.add_argument("--inv-tau", type=float, default=None,
                    help="override the stored calibrated 1/tau")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="only run 10 device-to-device copies of MIB MiB (calibrates the "
                         "HBM byte counters) and exit")
    ap.add_argument("--no-profile", action="store_true",
                    help="time without the per-kernel event records")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}): the path is "
              "data-parallel over requests with no exchange, so N GPUs run N independent "
              "copies of this benchmark.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
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

    w = synth.C2
    cfg = w.model
    if args.inv_tau is not None:
        inv_tau, tau_src = args.inv_tau, "command line"
    else:
        inv_tau, tau_src = load_inv_tau(cfg.name)
    dev = torch.device("cuda:0")
    tensors = sdev.model_tensors(cfg)
    shape = engine.ModelShape.of(cfg)
    model = engine.DeviceModel(shape, tensors, inv_tau)
    prompt, G, thr = synth.request(w, 0)
    L = len(prompt) + G
    eng = engine.Engine(model, 1, L, w.cache_mode)
    req = engine.Request(prompt, G, w.block, thr)
    eng.admit(req, cfg.mask_id)

    def one_step():
        nonlocal req
        if req.done:
            eng.release(req)
            req = engine.Request(prompt, G, w.block, thr)
            eng.admit(req, cfg.mask_id)
        m = req.masked_in_block
        n = eng.step([req])[0]
        return m, n

    for _ in range(args.warmup):
        one_step()
    torch.cuda.synchronize()
    if not args.no_profile:
        dlm.profile_read(model.handle)          # drop anything pending
        dlm.profile_enable(model.handle, True)
    masked_rows = 0
    unmasked = 0
    t0 = time.perf_counter()
    for _ in range(args.steps):
        m, n = one_step()
        masked_rows += m
        unmasked += n
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    prof = {}
    if not args.no_profile:
        dlm.profile_enable(model.handle, False)
        prof = dlm.profile_read(model.handle)
    elapsed = t1 - t0
    ms_per_step = 1e3 * elapsed / args.steps

    # roofline of the dominant kernel (largest total event time)
    m_avg = masked_rows / args.steps
    work = kernel_work(shape, L, L, m_avg)
    kernels = {}
    for name, (calls, tot) in prof.items():
        avg_ms = tot / max(calls, 1)
        entry = {"calls": calls, "avg_us": 1e3 * avg_ms, "share": tot / (1e3 * elapsed)}
        if name in work:
            F, B = work[name]
            entry["tflops"] = F / (avg_ms * 1e-3) / 1e12
            entry["gbs"] = B / (avg_ms * 1e-3) / 1e9
        kernels[name] = entry
    roof = None
    if prof:
        dom = max((k for k in prof if k in work), key=lambda k: prof[k][1])
        F, B = work[dom]
        avg_s = prof[dom][1] / prof[dom][0] * 1e-3
        peak = PEAK_BF16_TFLOPS if shape.dtype == "bf16" else PEAK_F32_TFLOPS
        traffic, traffic_src = measured_traffic(dom)
        ai = F / B
        if ai >= peak * 1e12 / (PEAK_HBM_GBS * 1e9):
            achieved = F / avg_s / 1e12
            roof = {"kernel": dom, "bound": "mfma", "achieved": achieved, "peak": peak,
                    "unit": "TFLOP/s", "frac": achieved / peak, "traffic": traffic,
                    "traffic_source": traffic_src, "algorithmic_bytes": B,
                    "flop_per_launch": F, "avg_launch_us": avg_s * 1e6}
        else:
            achieved = B / avg_s / 1e9
            roof = {"kernel": dom, "bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS,
                    "unit": "GB/s", "frac": achieved / PEAK_HBM_GBS, "traffic": traffic,
                    "traffic_source": traffic_src, "bytes_per_launch": B,
                    "avg_launch_us": avg_s * 1e6}
    Fs, Bs = step_work(shape, L, L, m_avg)
    t_step = elapsed / args.steps
    step_roof = {"tflops": Fs / t_step / 1e12, "gbs": Bs / t_step / 1e9,
                 "frac_mfma": Fs / t_step / (PEAK_BF16_TFLOPS * 1e12),
                 "frac_hbm": Bs / t_step / (PEAK_HBM_GBS * 1e9),
                 "flop_per_step": Fs, "bytes_per_step": Bs}

    cpu = None
    if args.cpu_layers > 0:
        cpu = cpu_baseline(cfg, tensors, prompt, G, inv_tau, args.cpu_layers)

    out = {
        "metric": "denoise steps/s + unmasked tokens/s per MI355X; % MFMA / HBM roofline",
        "value": args.steps / elapsed,
        "unit": "steps/s",
        "unmasked_tokens_per_s": unmasked / elapsed,
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms_per_step, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": w.name, "batch": w.batch, "prompt_len": w.prompt_len,
                   "gen_len": w.gen_len, "block": w.block, "cache": w.cache_mode,
                   "threshold": w.threshold, "inv_tau": inv_tau, "inv_tau_source": tau_src,
                   "weights": "synthetic N(0,0.02) seed 0", "recomputed_rows": L,
                   "avg_masked_rows": m_avg},
        "roofline": roof,
        "step_roofline": step_roof,
        "kernels": kernels,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
