"""ctypes binding of libdlm.so: the same entry points as include/dlm.h.

Argument marshalling only: torch tensors supply device memory and streams,
every step of the computation runs in the library's HIP kernels. If the
library is not built the import of any entry point raises; there is no
fallback path.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, c_float, c_int32, c_size_t, c_uint8, c_void_p

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libdlm.so")

DLM_OK, DLM_EINVAL, DLM_ESIZE, DLM_EHIP, DLM_ESTATE, DLM_EUNSUPPORTED = 0, -1, -2, -3, -4, -5
DLM_F32, DLM_BF16 = 0, 1
DLM_CACHE_NONE, DLM_CACHE_PREFIX, DLM_CACHE_DUAL = 0, 1, 2
DLM_MAX_BLOCK, DLM_MAX_REQ, DLM_MAX_SEQ = 64, 64, 8192
DLM_NSTATS = 8
DLM_SCRATCH_BYTES = 128 << 20
DLM_REQ_REFRESH = 1
MODES = {"none": DLM_CACHE_NONE, "prefix": DLM_CACHE_PREFIX, "dual": DLM_CACHE_DUAL}

EXPORTS = ["dlm_load_weights", "dlm_model_destroy", "dlm_workspace_bytes",
           "dlm_kv_cache_alloc", "dlm_cache_destroy", "dlm_cache_invalidate",
           "dlm_denoise_step", "dlm_denoise_step_noalloc", "dlm_cache_refresh",
           "dlm_debug_logits", "dlm_debug_trace", "dlm_debug_gemm_info", "dlm_debug_gemm",
           "dlm_head_confidence", "dlm_profile_enable", "dlm_profile_read",
           "dlm_profile_sample", "dlm_ceiling_mfma", "dlm_ceiling_copy", "dlm_last_error"]


class DlmConfig(ctypes.Structure):
    _fields_ = [("n_layers", c_int32), ("d_model", c_int32), ("n_q_heads", c_int32),
                ("n_kv_heads", c_int32), ("head_dim", c_int32), ("d_ffn", c_int32),
                ("vocab", c_int32), ("mask_id", c_int32), ("rms_eps", c_float),
                ("rope_theta", c_float), ("inv_tau", c_float), ("dtype", c_int32)]


class DlmLayerWeights(ctypes.Structure):
    _fields_ = [("attn_norm", c_void_p), ("w_qkv", c_void_p), ("w_o", c_void_p),
                ("ffn_norm", c_void_p), ("w_gate_up", c_void_p), ("w_down", c_void_p)]


class DlmWeights(ctypes.Structure):
    _fields_ = [("embed", c_void_p), ("lm_head", c_void_p), ("final_norm", c_void_p),
                ("layers", POINTER(DlmLayerWeights))]


class DlmReq(ctypes.Structure):
    _fields_ = [("slot", c_int32), ("seq_len", c_int32), ("prompt_len", c_int32),
                ("block_start", c_int32), ("block_len", c_int32), ("tok_offset", c_int32),
                ("flags", c_int32)]


class DlmBatch(ctypes.Structure):
    _fields_ = [("n_req", c_int32), ("reqs", POINTER(DlmReq)), ("tokens", c_void_p),
                ("mask", c_void_p), ("mode", c_int32), ("tok_conf", c_void_p)]


class DlmStepOut(ctypes.Structure):
    _fields_ = [("n_unmasked", c_void_p), ("pos", c_void_p), ("tok", c_void_p),
                ("conf", c_void_p), ("block_conf", c_void_p), ("block_tok", c_void_p),
                ("stats", c_void_p)]


class DlmTrace(ctypes.Structure):
    _fields_ = [("layer", c_int32), ("qkv_cap", c_int32), ("h_in", c_void_p),
                ("a_attn", c_void_p), ("qkv", c_void_p), ("q", c_void_p),
                ("attn_out", c_void_p), ("h_mid", c_void_p), ("a_ffn", c_void_p),
                ("act", c_void_p), ("h_out", c_void_p), ("u", c_void_p), ("logits", c_void_p),
                ("qkv_splits", c_int32)]


TRACE_BUFFERS = ("h_in", "a_attn", "qkv", "q", "attn_out", "h_mid", "a_ffn", "act", "h_out",
                 "u", "logits")


class DlmProfileEntry(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 32), ("calls", c_int32), ("total_ms", ctypes.c_double),
                ("launches", c_int32)]


class DlmError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"dlm status {status}: {msg}")
        self.status = status


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built: run __graft_entry__.build() "
                               "(there is no fallback implementation)")
        L = ctypes.CDLL(LIB_PATH)
        L.dlm_load_weights.argtypes = [POINTER(DlmConfig), POINTER(DlmWeights), POINTER(c_void_p)]
        L.dlm_model_destroy.argtypes = [c_void_p]
        L.dlm_model_destroy.restype = None
        L.dlm_workspace_bytes.argtypes = [c_void_p, c_int32, c_int32, POINTER(c_size_t)]
        L.dlm_kv_cache_alloc.argtypes = [c_void_p, c_int32, c_int32, c_void_p, c_size_t,
                                         POINTER(c_size_t), POINTER(c_void_p)]
        L.dlm_cache_destroy.argtypes = [c_void_p]
        L.dlm_cache_destroy.restype = None
        L.dlm_cache_invalidate.argtypes = [c_void_p, c_int32]
        L.dlm_denoise_step.argtypes = [c_void_p, c_void_p, POINTER(DlmBatch), POINTER(c_float),
                                       POINTER(DlmStepOut), c_void_p, c_size_t, c_void_p]
        L.dlm_denoise_step_noalloc.argtypes = [c_void_p, c_void_p, POINTER(DlmBatch),
                                               POINTER(c_float), POINTER(DlmStepOut), c_void_p]
        L.dlm_cache_refresh.argtypes = [c_void_p, c_void_p, POINTER(DlmBatch), c_void_p,
                                        c_size_t, c_void_p]
        L.dlm_debug_logits.argtypes = [c_void_p, c_void_p, POINTER(DlmBatch), c_void_p,
                                       c_void_p, c_size_t, c_void_p]
        L.dlm_debug_trace.argtypes = [c_void_p, c_void_p, POINTER(DlmBatch), POINTER(DlmTrace),
                                      c_void_p, c_size_t, c_void_p]
        L.dlm_head_confidence.argtypes = [c_void_p, c_void_p, c_int32, c_void_p, c_void_p,
                                          c_void_p, c_size_t, c_void_p]
        L.dlm_debug_gemm_info.argtypes = [c_int32, POINTER(c_int32), POINTER(c_int32),
                                          POINTER(c_int32)]
        L.dlm_debug_gemm.argtypes = [c_int32, c_int32, c_int32, c_int32, c_int32, c_int32,
                                     c_void_p, c_void_p, c_void_p, c_int32, c_int32, c_int32,
                                     c_void_p]
        L.dlm_profile_enable.argtypes = [c_void_p, c_int32, ctypes.c_char_p]
        L.dlm_profile_read.argtypes = [c_void_p, POINTER(DlmProfileEntry), c_int32,
                                       POINTER(c_int32)]
        L.dlm_profile_sample.argtypes = [c_void_p, c_int32]
        L.dlm_ceiling_mfma.argtypes = [c_int32, c_int32, c_void_p, POINTER(ctypes.c_double),
                                       c_void_p]
        L.dlm_ceiling_copy.argtypes = [c_void_p, c_void_p, c_size_t, c_void_p]
        L.dlm_last_error.argtypes = []
        L.dlm_last_error.restype = ctypes.c_char_p
        for name in ["dlm_load_weights", "dlm_workspace_bytes", "dlm_kv_cache_alloc",
                     "dlm_cache_invalidate", "dlm_denoise_step", "dlm_denoise_step_noalloc",
                     "dlm_cache_refresh",
                     "dlm_debug_logits", "dlm_debug_trace", "dlm_head_confidence",
                     "dlm_debug_gemm_info", "dlm_debug_gemm",
                     "dlm_profile_enable",
                     "dlm_profile_read", "dlm_profile_sample"]:
            getattr(L, name).restype = c_int32
        _lib = L
    return _lib


def last_error() -> str:
    return lib().dlm_last_error().decode()


def check(status: int):
    if status != DLM_OK:
        raise DlmError(status, last_error())


def _ptr(t):
    return None if t is None else c_void_p(t.data_ptr())


def _stream(stream):
    if stream is not None:
        return c_void_p(stream)
    import torch
    return c_void_p(torch.cuda.current_stream().cuda_stream)


# ------------------------------------------------------------- entry points
def load_weights(cfg: DlmConfig, weights: DlmWeights) -> c_void_p:
    h = c_void_p()
    check(lib().dlm_load_weights(ctypes.byref(cfg), ctypes.byref(weights), ctypes.byref(h)))
    return h


def model_destroy(h):
    lib().dlm_model_destroy(h)


def workspace_bytes(model, max_rows: int, max_reqs: int) -> int:
    out = c_size_t()
    check(lib().dlm_workspace_bytes(model, max_rows, max_reqs, ctypes.byref(out)))
    return out.value


def kv_cache_alloc(model, n_slots: int, max_seq_len: int, dev_buf=None, buf_bytes: int = 0):
    """Returns (cache handle or None, required bytes)."""
    req = c_size_t()
    h = c_void_p()
    check(lib().dlm_kv_cache_alloc(model, n_slots, max_seq_len, _ptr(dev_buf), buf_bytes,
                                   ctypes.byref(req), ctypes.byref(h)))
    return (h if dev_buf is not None else None), req.value


def cache_destroy(h):
    lib().dlm_cache_destroy(h)


def cache_invalidate(cache, slot: int):
    check(lib().dlm_cache_invalidate(cache, slot))


def make_batch(reqs, tokens, mask, mode: int, tok_conf=None):
    arr = (DlmReq * len(reqs))(*reqs)
    b = DlmBatch(len(reqs), ctypes.cast(arr, POINTER(DlmReq)), tokens.data_ptr(),
                 mask.data_ptr(), mode, None if tok_conf is None else tok_conf.data_ptr())
    b._keep = arr
    return b


def make_step_out(n_unmasked, pos, tok, conf, block_conf=None, block_tok=None, stats=None):
    return DlmStepOut(n_unmasked.data_ptr(), pos.data_ptr(), tok.data_ptr(), conf.data_ptr(),
                      None if block_conf is None else block_conf.data_ptr(),
                      None if block_tok is None else block_tok.data_ptr(),
                      None if stats is None else stats.data_ptr())


def denoise_step(model, cache, batch: DlmBatch, thresholds, out: DlmStepOut, workspace,
                 stream=None):
    thr = (c_float * batch.n_req)(*[float(t) for t in thresholds])
    check(lib().dlm_denoise_step(model, cache, ctypes.byref(batch), thr, ctypes.byref(out),
                                 _ptr(workspace), workspace.numel() * workspace.element_size(),
                                 _stream(stream)))


def denoise_step_noalloc(model, cache, batch: DlmBatch, thresholds, out: DlmStepOut,
                         stream=None):
    """dlm_denoise_step with the library's fixed scratch instead of a workspace."""
    thr = (c_float * batch.n_req)(*[float(t) for t in thresholds])
    check(lib().dlm_denoise_step_noalloc(model, cache, ctypes.byref(batch), thr,
                                         ctypes.byref(out), _stream(stream)))


def cache_refresh(model, cache, batch: DlmBatch, workspace, stream=None):
    check(lib().dlm_cache_refresh(model, cache, ctypes.byref(batch), _ptr(workspace),
                                  workspace.numel() * workspace.element_size(), _stream(stream)))


def debug_logits(model, cache, batch: DlmBatch, logits_out, workspace, stream=None):
    check(lib().dlm_debug_logits(model, cache, ctypes.byref(batch), _ptr(logits_out),
                                 _ptr(workspace), workspace.numel() * workspace.element_size(),
                                 _stream(stream)))


def debug_trace(model, cache, batch: DlmBatch, layer: int, buffers: dict, qkv_cap: int,
                workspace, stream=None) -> int:
    """Record layer `layer` of the step's forward into the given device tensors
    (keys of TRACE_BUFFERS; missing keys record nothing). Returns the number of
    QKV K-split slices written."""
    unknown = set(buffers) - set(TRACE_BUFFERS)
    if unknown:
        raise ValueError(f"unknown trace buffers {sorted(unknown)}")
    ptrs = [None if buffers.get(k) is None else buffers[k].data_ptr() for k in TRACE_BUFFERS]
    tr = DlmTrace(layer, qkv_cap, *ptrs, 0)
    check(lib().dlm_debug_trace(model, cache, ctypes.byref(batch), ctypes.byref(tr),
                                _ptr(workspace), workspace.numel() * workspace.element_size(),
                                _stream(stream)))
    return tr.qkv_splits


def head_confidence(model, u_rows, m_rows: int, conf, tok, workspace, stream=None):
    check(lib().dlm_head_confidence(model, _ptr(u_rows), m_rows, _ptr(conf), _ptr(tok),
                                    _ptr(workspace),
                                    workspace.numel() * workspace.element_size(),
                                    _stream(stream)))


def debug_gemm_info(cfg: int):
    """(bm, bn, flags) of a GEMM tile configuration, or None when the
    configuration does not exist; flags: bit 1 / bit 2 allowed half / quarter
    sub-tiles, bit 8 no SwiGLU epilogue."""
    bm, bn, subs = c_int32(), c_int32(), c_int32()
    rc = lib().dlm_debug_gemm_info(cfg, ctypes.byref(bm), ctypes.byref(bn), ctypes.byref(subs))
    if rc != DLM_OK:
        return None
    return bm.value, bn.value, subs.value


def debug_gemm(cfg: int, epilogue: int, a, b, c, sub: int = 0, n_tail: int = 0,
               group_m: int = 0, splits: int = 1, stream=None):
    """One launch of GEMM configuration cfg: epilogue 0 stores a @ b.T (fp32;
    with splits > 1 one slice per K range, c of shape (splits, M, N)), 1 stores
    silu(gate) * up (bf16, N/2 columns), 2 adds a @ b.T into c."""
    M, K = a.shape
    N = b.shape[0]
    for t in (a, b, c):
        if not t.is_contiguous():
            raise ValueError("GEMM operands must be contiguous")
    if b.shape[1] != K:
        raise ValueError("a and b disagree on K")
    want = (M, N // 2) if epilogue == 1 else ((splits, M, N) if splits > 1 else (M, N))
    if tuple(c.shape) != want:
        raise ValueError(f"c has shape {tuple(c.shape)}, expected {want}")
    check(lib().dlm_debug_gemm(cfg, epilogue, sub, n_tail, group_m, splits, _ptr(a), _ptr(b),
                               _ptr(c), M, N, K, _stream(stream)))


def profile_enable(model, on: bool, only_class: str | None = None):
    check(lib().dlm_profile_enable(model, 1 if on else 0,
                                   None if only_class is None else only_class.encode()))


def profile_sample(model, every: int):
    """Time one launch in `every` of each selected class (1: all)."""
    check(lib().dlm_profile_sample(model, every))


def profile_read(model, cap: int = 64) -> dict:
    """{kernel class: (timed launches, their total ms, all launches)} since the
    last read."""
    arr = (DlmProfileEntry * cap)()
    n = c_int32()
    check(lib().dlm_profile_read(model, arr, cap, ctypes.byref(n)))
    return {arr[i].name.decode(): (arr[i].calls, arr[i].total_ms, arr[i].launches)
            for i in range(n.value)}


def ceiling_mfma(n_blocks: int, iters: int, out_ptr: int, stream: int) -> float:
    """Enqueue the bf16 MFMA loop; returns the FLOPs it executes."""
    f = ctypes.c_double()
    check(lib().dlm_ceiling_mfma(n_blocks, iters, out_ptr, ctypes.byref(f), stream))
    return f.value


def ceiling_copy(src_ptr: int, dst_ptr: int, nbytes: int, stream: int) -> None:
    """Enqueue a device copy of nbytes (16-byte aligned, multiple of 16)."""
    check(lib().dlm_ceiling_copy(src_ptr, dst_ptr, nbytes, stream))
