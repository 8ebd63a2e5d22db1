"""Seeded synthetic inputs for the denoising-step workloads.

This module is shared by the CPU oracle, the tests and the benchmark, and holds
none of the method's arithmetic: it only draws weights and tokens.

Generator definition (one specification, implemented here in NumPy and again in
``synth/csrc/synth.hip`` for the device):

* SplitMix64 (Steele, Lea and Flood, "Fast splittable pseudorandom number
  generators", OOPSLA 2014): ``mix(z)`` is its output finaliser and a stream
  seeded with state ``s`` yields ``mix(s + (i + 1) * GOLDEN)`` for i = 0, 1, ...
* The stream key of tensor ``tid`` under ``seed`` is ``mix(mix(seed) ^ tid)``.
* Element i of a tensor draws the 64-bit word ``w = mix(key + (i + 1) * GOLDEN)``,
  splits it into two 32-bit halves ``u1 = (hi + 0.5) / 2**32`` and
  ``u2 = (lo + 0.5) / 2**32`` and applies the Box-Muller transform in fp64:
  ``n = sqrt(-2 ln u1) * cos(2 pi u2)``; the weight is ``std * n``.
* Storage: fp64 -> fp32 with round-to-nearest-even, then (bf16 models)
  fp32 -> bf16 with round-to-nearest-even.
* Tokens: element i of stream (seed, TOKENS) maps ``hi`` to ``(hi * V) >> 32``.
"""
from __future__ import annotations

import numpy as np

from .configs import (ModelConfig, Workload, MODELS, WORKLOADS, TINY_FP32,
                      MHA_8B, GQA_7B, C1, C2, C3_DUAL, C3_PREFIX, C4, C5)

GOLDEN = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)

# tensor ids: per-layer tensors are 1 + 16 * layer + kind
KIND_Q, KIND_K, KIND_V, KIND_O, KIND_GATE, KIND_UP, KIND_DOWN = range(7)
TID_EMBED = 1 << 40
TID_LM_HEAD = (1 << 40) + 1
TID_TOKENS = (1 << 40) + 2
TID_WORKLOAD = (1 << 40) + 3


def layer_tid(layer: int, kind: int) -> int:
    return 1 + 16 * layer + kind


def _mix(z: np.ndarray) -> np.ndarray:
    z = (z ^ (z >> np.uint64(30))) * _M1
    z = (z ^ (z >> np.uint64(27))) * _M2
    return z ^ (z >> np.uint64(31))


def _mix_int(z: int) -> int:
    m = (1 << 64) - 1
    z &= m
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & m
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & m
    return z ^ (z >> 31)


def stream_key(seed: int, tid: int) -> int:
    return _mix_int(_mix_int(seed) ^ (tid & ((1 << 64) - 1)))


def words(seed: int, tid: int, start: int, count: int) -> np.ndarray:
    """64-bit words start .. start+count-1 of the (seed, tid) stream."""
    key = np.uint64(stream_key(seed, tid))
    idx = np.arange(start + 1, start + count + 1, dtype=np.uint64)
    with np.errstate(over="ignore"):
        return _mix(key + idx * GOLDEN)


def normal_f64(seed: int, tid: int, start: int, count: int, std: float) -> np.ndarray:
    w = words(seed, tid, start, count)
    hi = (w >> np.uint64(32)).astype(np.float64)
    lo = (w & np.uint64(0xFFFFFFFF)).astype(np.float64)
    u1 = (hi + 0.5) * (1.0 / 4294967296.0)
    u2 = (lo + 0.5) * (1.0 / 4294967296.0)
    return std * (np.sqrt(-2.0 * np.log(u1)) * np.cos(2.0 * np.pi * u2))


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit pattern, round to nearest even (inputs are finite)."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))
    return ((b + bias) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def weight_values(seed: int, tid: int, shape, std: float, dtype: str,
                  start: int = 0) -> np.ndarray:
    """Stored values of a synthetic weight tensor as float32 (bf16-exact for bf16).

    ``start`` is the flat element offset of the first value (for row samples).
    """
    n = int(np.prod(shape))
    f32 = normal_f64(seed, tid, start, n, std).astype(np.float32)
    if dtype == "bf16":
        f32 = bf16_bits_to_f32(f32_to_bf16_bits(f32))
    return f32.reshape(shape)


def weight_rows(cfg: ModelConfig, tid: int, n_cols: int, rows) -> np.ndarray:
    """Selected rows of a [*, n_cols] synthetic weight tensor (float32 values)."""
    rows = np.asarray(rows, dtype=np.int64)
    out = np.empty((len(rows), n_cols), dtype=np.float32)
    for i, r in enumerate(rows):
        out[i] = weight_values(cfg.weight_seed, tid, (n_cols,), cfg.weight_std,
                               cfg.dtype, start=int(r) * n_cols)
    return out


def layer_shapes(cfg: ModelConfig):
    d, dh = cfg.d_model, cfg.head_dim
    return {
        KIND_Q: (cfg.n_q_heads * dh, d),
        KIND_K: (cfg.n_kv_heads * dh, d),
        KIND_V: (cfg.n_kv_heads * dh, d),
        KIND_O: (d, cfg.n_q_heads * dh),
        KIND_GATE: (cfg.d_ffn, d),
        KIND_UP: (cfg.d_ffn, d),
        KIND_DOWN: (d, cfg.d_ffn),
    }


def layer_weights(cfg: ModelConfig, layer: int) -> dict:
    """All weights of one layer as float32 arrays, [out, in] row-major.

    Norm gains are 1.0 (not drawn)."""
    sh = layer_shapes(cfg)
    names = {KIND_Q: "wq", KIND_K: "wk", KIND_V: "wv", KIND_O: "wo",
             KIND_GATE: "wg", KIND_UP: "wu", KIND_DOWN: "wd"}
    out = {names[k]: weight_values(cfg.weight_seed, layer_tid(layer, k), s,
                                   cfg.weight_std, cfg.dtype)
           for k, s in sh.items()}
    out["attn_norm"] = np.ones(cfg.d_model, np.float32)
    out["ffn_norm"] = np.ones(cfg.d_model, np.float32)
    return out


def global_weights(cfg: ModelConfig) -> dict:
    sh = (cfg.vocab, cfg.d_model)
    return {
        "embed": weight_values(cfg.weight_seed, TID_EMBED, sh, cfg.weight_std, cfg.dtype),
        "lm_head": weight_values(cfg.weight_seed, TID_LM_HEAD, sh, cfg.weight_std, cfg.dtype),
        "final_norm": np.ones(cfg.d_model, np.float32),
    }


def model_weights(cfg: ModelConfig, n_layers: int | None = None) -> dict:
    """Whole synthetic model on the host (small models and reduced depth only)."""
    n = cfg.n_layers if n_layers is None else n_layers
    w = global_weights(cfg)
    w["layers"] = [layer_weights(cfg, l) for l in range(n)]
    return w


def tokens(seed: int, count: int, vocab: int) -> np.ndarray:
    """``count`` token ids uniform in [0, vocab - 1]."""
    hi = words(seed, TID_TOKENS, 0, count) >> np.uint64(32)
    return ((hi * np.uint64(vocab)) >> np.uint64(32)).astype(np.int32)


def uniform_ints(seed: int, tid: int, count: int, lo: int, hi_incl: int) -> np.ndarray:
    span = np.uint64(hi_incl - lo + 1)
    hi = words(seed, tid, 0, count) >> np.uint64(32)
    return (lo + ((hi * span) >> np.uint64(32))).astype(np.int64)


def request(w: Workload, r: int):
    """Request r of a workload: (prompt tokens, gen_len, threshold).

    Fixed-shape workloads use their prompt/gen lengths; the heterogeneous one
    draws P ~ U[lo, hi], G from ``gen_choices`` and the threshold from
    ``threshold_choices`` with the request's own seed."""
    seed = w.request_seed_base + r
    if w.prompt_range is not None:
        p, g, t = uniform_ints(seed, TID_WORKLOAD, 3, 0, 1 << 20)
        P = int(w.prompt_range[0] + p % (w.prompt_range[1] - w.prompt_range[0] + 1))
        G = int(w.gen_choices[int(g) % len(w.gen_choices)])
        thr = float(w.threshold_choices[int(t) % len(w.threshold_choices)])
    else:
        P, G, thr = w.prompt_len, w.gen_len, w.threshold
    return tokens(seed, P, w.model.vocab), G, thr


__all__ = [
    "ModelConfig", "Workload", "MODELS", "WORKLOADS", "TINY_FP32", "MHA_8B", "GQA_7B",
    "C1", "C2", "C3_DUAL", "C3_PREFIX", "C4", "C5",
    "words", "normal_f64", "weight_values", "weight_rows", "layer_weights",
    "global_weights", "model_weights", "tokens", "request", "layer_tid",
    "f32_to_bf16_bits", "bf16_bits_to_f32", "stream_key",
    "TID_EMBED", "TID_LM_HEAD", "TID_TOKENS",
    "KIND_Q", "KIND_K", "KIND_V", "KIND_O", "KIND_GATE", "KIND_UP", "KIND_DOWN",
]
