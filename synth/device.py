"""Device-side weight generation (same definition as ``synth``) via libsynth.so.

Used to materialise full-scale synthetic models directly in GPU memory; the
host implementation in ``synth`` regenerates any sample of it for checking.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libsynth.so")
_lib = None


def build() -> str:
    import subprocess
    src = os.path.join(HERE, "csrc", "synth.hip")
    tmp = LIB_PATH + ".tmp"
    cmd = ["/opt/rocm/bin/hipcc", "--offload-arch=gfx950", "-O3", "-fPIC", "-shared",
           "-std=c++17", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-o", tmp, src]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("libsynth build failed:\n" + r.stderr)
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libsynth.so is not built (run __graft_entry__.build())")
        L = ctypes.CDLL(LIB_PATH)
        L.synth_fill_normal.argtypes = [ctypes.c_void_p, ctypes.c_long, ctypes.c_int,
                                        ctypes.c_uint64, ctypes.c_uint64, ctypes.c_long,
                                        ctypes.c_double, ctypes.c_void_p]
        L.synth_fill_normal.restype = ctypes.c_int
        L.synth_fill_const.argtypes = [ctypes.c_void_p, ctypes.c_long, ctypes.c_float,
                                       ctypes.c_void_p]
        L.synth_fill_const.restype = ctypes.c_int
        _lib = L
    return _lib


def fill_normal(tensor, seed: int, tid: int, std: float, start: int = 0, stream=None):
    """Fill a contiguous torch CUDA tensor (float32 or bfloat16) in place."""
    import torch
    assert tensor.is_cuda and tensor.is_contiguous()
    dtype = {torch.float32: 0, torch.bfloat16: 1}[tensor.dtype]
    st = stream if stream is not None else torch.cuda.current_stream().cuda_stream
    rc = lib().synth_fill_normal(ctypes.c_void_p(tensor.data_ptr()), tensor.numel(), dtype,
                                 seed & ((1 << 64) - 1), tid & ((1 << 64) - 1), start,
                                 float(std), ctypes.c_void_p(st))
    if rc != 0:
        raise RuntimeError(f"synth_fill_normal failed with hipError {rc}")
    return tensor


def fill_const(tensor, value: float, stream=None):
    import torch
    assert tensor.is_cuda and tensor.dtype == torch.float32 and tensor.is_contiguous()
    st = stream if stream is not None else torch.cuda.current_stream().cuda_stream
    rc = lib().synth_fill_const(ctypes.c_void_p(tensor.data_ptr()), tensor.numel(),
                                float(value), ctypes.c_void_p(st))
    if rc != 0:
        raise RuntimeError(f"synth_fill_const failed with hipError {rc}")
    return tensor


def model_tensors(cfg, n_layers=None, device="cuda:0", stream=None):
    """Synthetic model drawn directly in device memory, in the layouts the
    library takes: w_qkv = [Wq; Wk; Wv] rows, w_gate_up = [Wgate; Wup] rows,
    norm gains 1.0 in fp32."""
    import torch
    from . import (TID_EMBED, TID_LM_HEAD, KIND_Q, KIND_K, KIND_V, KIND_O, KIND_GATE,
                   KIND_UP, KIND_DOWN, layer_tid)
    n = cfg.n_layers if n_layers is None else n_layers
    dt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    d, dh = cfg.d_model, cfg.head_dim
    seed, std = cfg.weight_seed, cfg.weight_std

    def mat(rows, cols):
        return torch.empty(rows, cols, dtype=dt, device=device)

    t = {"embed": fill_normal(mat(cfg.vocab, d), seed, TID_EMBED, std, stream=stream),
         "lm_head": fill_normal(mat(cfg.vocab, d), seed, TID_LM_HEAD, std, stream=stream),
         "final_norm": torch.ones(d, dtype=torch.float32, device=device),
         "layers": []}
    qd, kd = cfg.n_q_heads * dh, cfg.n_kv_heads * dh
    for l in range(n):
        qkv = mat(qd + 2 * kd, d)
        fill_normal(qkv[:qd], seed, layer_tid(l, KIND_Q), std, stream=stream)
        fill_normal(qkv[qd:qd + kd], seed, layer_tid(l, KIND_K), std, stream=stream)
        fill_normal(qkv[qd + kd:], seed, layer_tid(l, KIND_V), std, stream=stream)
        gu = mat(2 * cfg.d_ffn, d)
        fill_normal(gu[:cfg.d_ffn], seed, layer_tid(l, KIND_GATE), std, stream=stream)
        fill_normal(gu[cfg.d_ffn:], seed, layer_tid(l, KIND_UP), std, stream=stream)
        t["layers"].append({
            "attn_norm": torch.ones(d, dtype=torch.float32, device=device),
            "w_qkv": qkv,
            "w_o": fill_normal(mat(d, qd), seed, layer_tid(l, KIND_O), std, stream=stream),
            "ffn_norm": torch.ones(d, dtype=torch.float32, device=device),
            "w_gate_up": gu,
            "w_down": fill_normal(mat(d, cfg.d_ffn), seed, layer_tid(l, KIND_DOWN), std,
                                  stream=stream),
        })
    return t
