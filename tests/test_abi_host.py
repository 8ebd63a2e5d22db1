"""Host-side checks of the C ABI (no GPU needed): the library loads and
exports every entry point the header declares, validation rejects malformed
calls before anything is enqueued, the cache size query, slot state errors,
and the host-side block bookkeeping of the engine."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2606_29094_amd import dlm

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dlm.h")


def _lib_or_skip():
    if not os.path.exists(dlm.LIB_PATH):
        pytest.skip("libdlm.so not built")
    return dlm.lib()


def test_header_declarations_are_exported():
    L = _lib_or_skip()
    src = open(HEADER).read()
    declared = set(re.findall(r"\b(dlm_[a-z_]+)\s*\(", src))
    assert declared, "no declarations parsed"
    assert declared == set(dlm.EXPORTS), declared ^ set(dlm.EXPORTS)
    for name in declared:
        assert hasattr(L, name), name


def _cfg(**kw):
    c = dict(n_layers=2, d_model=256, n_q_heads=4, n_kv_heads=4, head_dim=64, d_ffn=688,
             vocab=2048, mask_id=2047, rms_eps=1e-5, rope_theta=1e4, inv_tau=10.0,
             dtype=dlm.DLM_F32)
    c.update(kw)
    return dlm.DlmConfig(**c)


FAKE = 0x1000   # never dereferenced: no kernel is launched by these tests


def _weights(n_layers=2):
    arr = (dlm.DlmLayerWeights * n_layers)(*[dlm.DlmLayerWeights(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE)
                                              for _ in range(n_layers)])
    w = dlm.DlmWeights(FAKE, FAKE, FAKE, arr)
    w._keep = arr
    return w


def _load(cfg=None):
    return dlm.load_weights(cfg or _cfg(), _weights())


@pytest.mark.parametrize("bad,status", [
    (dict(head_dim=96), dlm.DLM_EUNSUPPORTED),
    (dict(n_q_heads=6, n_kv_heads=4), dlm.DLM_EINVAL),
    (dict(d_model=200), dlm.DLM_EUNSUPPORTED),
    (dict(d_ffn=690), dlm.DLM_EUNSUPPORTED),
    (dict(mask_id=2048), dlm.DLM_EINVAL),
    (dict(inv_tau=float("nan")), dlm.DLM_EINVAL),
    (dict(dtype=7), dlm.DLM_EINVAL),
])
def test_load_weights_rejects_bad_config(bad, status):
    _lib_or_skip()
    with pytest.raises(dlm.DlmError) as e:
        dlm.load_weights(_cfg(**bad), _weights())
    assert e.value.status == status
    assert dlm.last_error()


def test_load_weights_rejects_null_layer_pointer():
    _lib_or_skip()
    w = _weights()
    w.layers[1].w_o = None
    with pytest.raises(dlm.DlmError) as e:
        dlm.load_weights(_cfg(), w)
    assert e.value.status == dlm.DLM_EINVAL and "layer 1" in dlm.last_error()


def test_cache_size_query_and_workspace():
    _lib_or_skip()
    m = _load()
    h, need = dlm.kv_cache_alloc(m, 3, 100)
    assert h is None
    # K and V, 2 layers, 3 slots, 4 kv heads, positions rounded up to 128, fp32
    assert need == 2 * 2 * 3 * 4 * 128 * 64 * 4
    ws1 = dlm.workspace_bytes(m, 128, 1)
    ws2 = dlm.workspace_bytes(m, 1024, 8)
    assert 0 < ws1 < ws2
    with pytest.raises(dlm.DlmError):
        dlm.workspace_bytes(m, 0, 1)
    with pytest.raises(dlm.DlmError):
        dlm.workspace_bytes(m, 16, dlm.DLM_MAX_REQ + 1)
    dlm.model_destroy(m)


class _Buf:
    """Stand-in for a device tensor (only data_ptr / numel / element_size are
    read by the binding; validation fails before any use of the address)."""

    def __init__(self, addr, n=1 << 30):
        self.addr, self.n = addr, n

    def data_ptr(self):
        return self.addr

    def numel(self):
        return self.n

    def element_size(self):
        return 1


def _cache(m, slots=2, seq=128):
    _, need = dlm.kv_cache_alloc(m, slots, seq)
    h, _ = dlm.kv_cache_alloc(m, slots, seq, _Buf(0x100000), need)
    return h


def _step(m, c, reqs, thr=None, mode=dlm.DLM_CACHE_DUAL, ws=None):
    b = dlm.make_batch(reqs, _Buf(0x200000), _Buf(0x300000), mode)
    out = dlm.make_step_out(_Buf(0x400000), _Buf(0x500000), _Buf(0x600000), _Buf(0x700000))
    dlm.denoise_step(m, c, b, thr or [0.9] * len(reqs), out, ws or _Buf(0x800000, 1 << 20),
                     stream=0)


def _req(slot=0, seq=96, P=32, s=32, blen=32, off=0, flags=0):
    return dlm.DlmReq(slot, seq, P, s, blen, off, flags)


@pytest.mark.parametrize("req,thr,status,msg", [
    (_req(slot=5), None, dlm.DLM_EINVAL, "slot"),
    (_req(seq=200), None, dlm.DLM_ESIZE, "seq_len"),
    (_req(P=40, s=32), None, dlm.DLM_EINVAL, "prompt_len"),
    (_req(blen=65), None, dlm.DLM_EINVAL, "block"),
    (_req(s=80, blen=32), None, dlm.DLM_EINVAL, "block"),
    (_req(flags=4), None, dlm.DLM_EINVAL, "flags"),
    (_req(flags=1), [1.5], dlm.DLM_EINVAL, "threshold"),
    (_req(flags=1), [float("nan")], dlm.DLM_EINVAL, "threshold"),
])
def test_denoise_step_validation(req, thr, status, msg):
    _lib_or_skip()
    m = _load()
    c = _cache(m)
    with pytest.raises(dlm.DlmError) as e:
        _step(m, c, [req], thr)
    assert e.value.status == status, dlm.last_error()
    assert msg in dlm.last_error()


def test_cache_step_on_stale_slot_is_a_state_error():
    _lib_or_skip()
    m = _load()
    c = _cache(m)
    with pytest.raises(dlm.DlmError) as e:
        _step(m, c, [_req(flags=0)])
    assert e.value.status == dlm.DLM_ESTATE
    # invalidate is accepted for valid slots only
    dlm.cache_invalidate(c, 1)
    with pytest.raises(dlm.DlmError):
        dlm.cache_invalidate(c, 2)


def test_duplicate_slot_and_workspace_checks():
    _lib_or_skip()
    m = _load()
    c = _cache(m)
    with pytest.raises(dlm.DlmError) as e:
        _step(m, c, [_req(flags=1), _req(flags=1, off=96)])
    assert "used twice" in dlm.last_error()
    with pytest.raises(dlm.DlmError) as e:
        _step(m, c, [_req(flags=1)], ws=_Buf(0x800000, 1024))
    assert e.value.status == dlm.DLM_ESIZE
    with pytest.raises(dlm.DlmError) as e:
        _step(m, c, [_req(flags=1)], ws=_Buf(0x800010))
    assert "aligned" in dlm.last_error()


def test_token_ranges_must_not_overlap():
    _lib_or_skip()
    m = _load()
    c = _cache(m)
    with pytest.raises(dlm.DlmError) as e:
        _step(m, c, [_req(slot=0, flags=1), _req(slot=1, flags=1, off=50)])
    assert e.value.status == dlm.DLM_EINVAL and "overlap" in dlm.last_error()
    # disjoint ranges pass the plan checks (and stop at the too-small workspace)
    with pytest.raises(dlm.DlmError) as e:
        _step(m, c, [_req(slot=0, flags=1), _req(slot=1, flags=1, off=96)], ws=_Buf(0x800000, 1024))
    assert e.value.status == dlm.DLM_ESIZE, dlm.last_error()
    dlm.model_destroy(m)


@pytest.mark.parametrize("dims", [
    dict(),
    dict(d_model=4096, n_q_heads=32, n_kv_heads=32, head_dim=128, d_ffn=12288, vocab=126464,
         mask_id=126336, dtype=dlm.DLM_BF16),
    dict(d_model=3584, n_q_heads=28, n_kv_heads=4, head_dim=128, d_ffn=18944, vocab=152064,
         mask_id=151666, dtype=dlm.DLM_BF16),
])
def test_workspace_bytes_is_monotonic_in_rows(dims):
    # the split-K slice buffers depend on the planner's choice for each row
    # count; the size query must cover every row count up to max_rows, so it
    # can never shrink as max_rows grows
    _lib_or_skip()
    m = _load(_cfg(**dims))
    prev = 0
    for n in range(1, 1100):
        w = dlm.workspace_bytes(m, n, 8)
        assert w >= prev, n
        prev = w
    dlm.model_destroy(m)


def test_engine_request_block_bookkeeping():
    from paper_2606_29094_amd.engine import Request
    r = Request(np.arange(10), 70, 32, 0.9)
    assert (r.seq_len, r.block_start, r.block_len) == (80, 10, 32)
    r.k = 2
    assert (r.block_start, r.block_len) == (74, 6)      # short last block
    assert not r.done
    r.k = 3
    assert r.done


def test_profile_sample_validation():
    _lib_or_skip()
    m = _load()
    try:
        dlm.profile_sample(m, 1)
        dlm.profile_sample(m, 31)
        with pytest.raises(dlm.DlmError) as e:
            dlm.profile_sample(m, 0)
        assert e.value.status == dlm.DLM_EINVAL and "every" in dlm.last_error()
        dlm.profile_enable(m, True, "gemm_gate_up_swiglu")
        assert dlm.profile_read(m) == {}
        dlm.profile_enable(m, False)
    finally:
        dlm.model_destroy(m)
    with pytest.raises(dlm.DlmError):
        dlm.profile_sample(None, 2)


def test_debug_gemm_validation_on_host():
    """Tile-configuration queries and the GEMM hook's argument checks run on
    the host: malformed launches are rejected before anything is enqueued."""
    L = _lib_or_skip()
    bm, bn, subs = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
    assert L.dlm_debug_gemm_info(6, ctypes.byref(bm), ctypes.byref(bn), ctypes.byref(subs)) == 0
    assert (bm.value, bn.value, subs.value) == (256, 256, 6)      # halves and quarters
    assert L.dlm_debug_gemm_info(65, ctypes.byref(bm), ctypes.byref(bn), ctypes.byref(subs)) == 0
    assert (bm.value, bn.value, subs.value) == (384, 256, 0)
    assert L.dlm_debug_gemm_info(70, ctypes.byref(bm), ctypes.byref(bn), ctypes.byref(subs)) == 0
    assert (bm.value, bn.value, subs.value) == (256, 224, 8)      # seven fragments: no SwiGLU
    assert L.dlm_debug_gemm_info(999, None, None, None) == dlm.DLM_EINVAL
    F = FAKE

    def call(cfg=6, epi=0, sub=0, tail=0, group=0, a=F, b=F, c=F, M=300, N=832, K=320, splits=1):
        return L.dlm_debug_gemm(cfg, epi, sub, tail, group, splits, a, b, c, M, N, K, None)
    assert call(cfg=999) == dlm.DLM_EINVAL
    assert call(a=None) == dlm.DLM_EINVAL
    assert call(K=100) == dlm.DLM_EINVAL
    assert call(M=0) == dlm.DLM_EINVAL
    assert call(epi=3) == dlm.DLM_EINVAL
    assert call(epi=1, N=80) == dlm.DLM_EINVAL           # width 40 not a multiple of 16
    assert call(cfg=62, epi=1, N=96) == dlm.DLM_EINVAL   # 32x32 tiles: width 48 not a multiple of 32
    assert call(cfg=70, epi=1) == dlm.DLM_EINVAL          # odd fragment count: no SwiGLU
    assert "SwiGLU" in dlm.last_error()
    assert call(sub=3, tail=1) == dlm.DLM_EINVAL
    assert call(cfg=65, sub=2, tail=1) == dlm.DLM_EINVAL  # no sub-tiles for 384x256
    assert call(sub=4, tail=10 ** 6) == dlm.DLM_EINVAL
    assert call(tail=-1) == dlm.DLM_EINVAL
    assert "n_tail" in dlm.last_error()
    assert call(splits=0) == dlm.DLM_EINVAL
    assert call(splits=2) == dlm.DLM_EINVAL               # 5 k-tiles do not split in two
    assert "splits" in dlm.last_error()
    assert call(epi=2, splits=5) == dlm.DLM_EINVAL        # slices of the plain store only
