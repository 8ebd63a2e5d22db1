"""ctypes binding of libdlmctl.so, the confidence-threshold controller (host
code). Argument marshalling only: every decision is taken in the library.

Thresholds are candidate indices 0..n-1 in ascending order; a request's
allowed set is a bit mask over them.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, c_double, c_int32, c_uint32
from typing import List, Optional, Sequence

from . import dlm

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libdlmctl.so")
EXPORTS = ["dlm_ctl_latency", "dlm_ctl_predicted_time_left", "dlm_ctl_update_threshold",
           "dlm_ctl_req_load", "dlm_ctl_capacity", "dlm_ctl_update_allowed",
           "dlm_ctl_last_error"]
MAX_GAMMA = 32


class Curve(ctypes.Structure):
    _fields_ = [("n", c_int32), ("tokens", POINTER(c_double)), ("latency_s", POINTER(c_double))]


class Profile(ctypes.Structure):
    _fields_ = [("recompute", Curve), ("cache", Curve)]


class Params(ctypes.Structure):
    _fields_ = [("n_gamma", c_int32), ("gamma", POINTER(c_double)), ("cache_block", c_int32),
                ("max_seqs_per_batch", c_int32), ("slo_s", c_double)]


class Req(ctypes.Structure):
    _fields_ = [("num_tokens", c_double), ("recomp_steps_left", c_double),
                ("pred_steps_left", POINTER(c_double)), ("slo_left_s", c_double),
                ("allowed", c_uint32), ("gamma_idx", c_int32)]


class Instance(ctypes.Structure):
    _fields_ = [("profile", POINTER(Profile)), ("num_tokens", c_double), ("num_reqs", c_int32)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built (run paper_2606_29094_amd.build)")
        L = ctypes.CDLL(LIB_PATH)
        L.dlm_ctl_latency.argtypes = [POINTER(Curve), c_double, POINTER(c_double)]
        L.dlm_ctl_predicted_time_left.argtypes = [POINTER(Params), POINTER(Instance), POINTER(Req),
                                                  c_int32, POINTER(c_double)]
        L.dlm_ctl_update_threshold.argtypes = [POINTER(Params), POINTER(Instance), POINTER(Req)]
        L.dlm_ctl_req_load.argtypes = [POINTER(Params), POINTER(Req), c_int32, POINTER(c_double)]
        L.dlm_ctl_capacity.argtypes = [POINTER(Params), POINTER(Profile), c_int32, c_double,
                                       POINTER(c_double)]
        L.dlm_ctl_update_allowed.argtypes = [POINTER(Params), POINTER(Req), c_int32, c_double]
        L.dlm_ctl_last_error.argtypes = []
        L.dlm_ctl_last_error.restype = ctypes.c_char_p
        for name in EXPORTS[:-1]:
            getattr(L, name).restype = c_int32
        _lib = L
    return _lib


def _check(status):
    if status != dlm.DLM_OK:
        raise dlm.DlmError(status, lib().dlm_ctl_last_error().decode())


def _arr(xs):
    xs = [float(x) for x in xs]
    return (c_double * max(len(xs), 1))(*xs)


def make_curve(tokens: Sequence[float], latency_s: Sequence[float]) -> Curve:
    t, l = _arr(tokens), _arr(latency_s)
    c = Curve(len(tokens), t, l)
    c._keep = (t, l)
    return c


def make_profile(recompute, cache=None) -> Profile:
    """recompute / cache: (tokens, latency_s) pairs of sequences."""
    rc = make_curve(*recompute)
    cc = make_curve(*cache) if cache is not None else Curve(0, None, None)
    p = Profile(rc, cc)
    p._keep = (rc, cc)
    return p


def make_params(gammas: Sequence[float], cache_block: int = 0, max_seqs_per_batch: int = 1,
                slo_s: float = 1.0) -> Params:
    g = _arr(gammas)
    p = Params(len(gammas), g, cache_block, max_seqs_per_batch, slo_s)
    p._keep = g
    return p


def make_req(num_tokens, pred_steps_left, slo_left_s=0.0, recomp_steps_left=0.0,
             allowed: Optional[int] = None) -> Req:
    s = _arr(pred_steps_left)
    full = (1 << len(pred_steps_left)) - 1
    r = Req(num_tokens, recomp_steps_left, s, slo_left_s, full if allowed is None else allowed, -1)
    r._keep = s
    return r


def make_instance(profile: Profile, num_tokens: float, num_reqs: int) -> Instance:
    i = Instance(ctypes.pointer(profile), num_tokens, num_reqs)
    i._keep = profile
    return i


def latency(curve: Curve, tokens: float) -> float:
    out = c_double()
    _check(lib().dlm_ctl_latency(ctypes.byref(curve), tokens, ctypes.byref(out)))
    return out.value


def predicted_time_left(p: Params, inst: Instance, req: Req, gi: int) -> float:
    out = c_double()
    _check(lib().dlm_ctl_predicted_time_left(ctypes.byref(p), ctypes.byref(inst),
                                             ctypes.byref(req), gi, ctypes.byref(out)))
    return out.value


def update_threshold(p: Params, inst: Instance, req: Req) -> int:
    _check(lib().dlm_ctl_update_threshold(ctypes.byref(p), ctypes.byref(inst), ctypes.byref(req)))
    return req.gamma_idx


def req_load(p: Params, req: Req, gi: int) -> float:
    out = c_double()
    _check(lib().dlm_ctl_req_load(ctypes.byref(p), ctypes.byref(req), gi, ctypes.byref(out)))
    return out.value


def capacity(p: Params, profiles: List[Profile], tokens_per_req: float = 0.0) -> float:
    arr = (Profile * max(len(profiles), 1))(*profiles)
    out = c_double()
    _check(lib().dlm_ctl_capacity(ctypes.byref(p), arr, len(profiles), tokens_per_req,
                                  ctypes.byref(out)))
    return out.value


def update_allowed(p: Params, reqs: List[Req], cap: float) -> List[int]:
    """Runs Alg. 2 over reqs (arrival order); writes and returns the masks."""
    arr = (Req * max(len(reqs), 1))(*reqs)
    _check(lib().dlm_ctl_update_allowed(ctypes.byref(p), arr, len(reqs), cap))
    for i, r in enumerate(reqs):
        r.allowed = arr[i].allowed
    return [r.allowed for r in reqs]


def mask_to_list(mask: int, n: int) -> List[int]:
    return [i for i in range(n) if (mask >> i) & 1]
