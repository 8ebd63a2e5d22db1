"""The identical-input checker (tests/kernel_checks.py) on the CPU: a layer
trace simulated in float32 arithmetic with bf16 (or fp32) storage, as the GPU
kernels compute it, must pass; the same trace with a planted mistake (a
dropped K term, a transposed head, a rotary angle of the wrong position, a
key beyond the sequence read by attention, a missing residual) must fail."""
import copy

import numpy as np
import pytest

import oracle
from kernel_checks import check_head_unmask, check_layer

f32 = np.float32


class Cfg:
    def __init__(self, dtype):
        self.dtype = dtype
        self.n_q_heads, self.n_kv_heads, self.head_dim = 4, 2, 64
        self.d_model, self.d_ffn, self.vocab = 128, 96, 300
        self.rms_eps, self.rope_theta, self.mask_id = 1e-5, 10000.0, 299


def _st(dtype, x):
    return oracle.round_bf16(x) if dtype == "bf16" else np.asarray(x, f32).astype(np.float64)


def _norm32(h, g, eps):
    h = h.astype(f32)
    ms = np.mean(h * h, axis=-1, keepdims=True, dtype=f32)
    return (h / np.sqrt(ms + f32(eps)) * g.astype(f32)).astype(np.float64)


def _simulate(dtype, seed=0):
    """A two-request step: request 0 recomputes all of its 40 positions,
    request 1 (a cache step) recomputes positions [24, 40) of 56."""
    c = Cfg(dtype)
    rng = np.random.default_rng(seed)
    d, hq, hkv, dh, F = c.d_model, c.n_q_heads, c.n_kv_heads, c.head_dim, c.d_ffn
    w = lambda *s: _st(dtype, rng.standard_normal(s) * 0.05)
    lw = {"wq": w(hq * dh, d), "wk": w(hkv * dh, d), "wv": w(hkv * dh, d), "wo": w(d, hq * dh),
          "wg": w(F, d), "wu": w(F, d), "wd": w(d, F),
          "attn_norm": np.ones(d), "ffn_norm": np.ones(d)}
    rows = [(0, 40), (24, 40)]
    seq = [40, 56]
    n = sum(b - a for a, b in rows)
    h_in = rng.standard_normal((n, d)).astype(f32).astype(np.float64)
    a1 = _st(dtype, _norm32(h_in, lw["attn_norm"], c.rms_eps))
    W = np.concatenate([lw["wq"], lw["wk"], lw["wv"]]).astype(f32)
    half = d // 2
    s0 = (a1[:, :half].astype(f32) @ W[:, :half].T).astype(np.float64)
    s1 = (a1[:, half:].astype(f32) @ W[:, half:].T).astype(np.float64)
    xs = (s0.astype(f32) + s1.astype(f32)).astype(np.float64)
    pos = np.concatenate([np.arange(a, b) for a, b in rows])
    qd, kd = hq * dh, hkv * dh
    q = _st(dtype, oracle.rope(xs[:, :qd].reshape(n, hq, dh), pos, c.rope_theta)).reshape(n, qd)
    k = _st(dtype, oracle.rope(xs[:, qd:qd + kd].reshape(n, hkv, dh), pos, c.rope_theta))
    v = _st(dtype, xs[:, qd + kd:].reshape(n, hkv, dh))
    caches = []
    off = 0
    for (a, b), L in zip(rows, seq):
        K = _st(dtype, rng.standard_normal((L, hkv, dh)) * 0.5)
        V = _st(dtype, rng.standard_normal((L, hkv, dh)) * 0.5)
        K[a:b], V[a:b] = k[off:off + b - a], v[off:off + b - a]
        caches.append((K, V))
        off += b - a
    ao = np.empty((n, hq, dh))
    off = 0
    for (a, b), (K, V) in zip(rows, caches):
        qq = q[off:off + b - a].reshape(-1, hq, dh).astype(f32)
        for h in range(hq):
            s = qq[:, h] @ K[:, h // 2].astype(f32).T / f32(np.sqrt(dh))
            p = np.exp(s - s.max(axis=1, keepdims=True))
            p = p / p.sum(axis=1, keepdims=True, dtype=f32)
            ao[off:off + b - a, h] = (p @ V[:, h // 2].astype(f32)).astype(np.float64)
        off += b - a
    ao = _st(dtype, ao).reshape(n, qd)
    h_mid = (h_in.astype(f32) + (ao.astype(f32) @ lw["wo"].astype(f32).T)).astype(np.float64)
    a2 = _st(dtype, _norm32(h_mid, lw["ffn_norm"], c.rms_eps))
    g = a2.astype(f32) @ lw["wg"].astype(f32).T
    u = a2.astype(f32) @ lw["wu"].astype(f32).T
    act = _st(dtype, (g / (f32(1) + np.exp(-g)) * u).astype(np.float64))
    h_out = (h_mid.astype(f32) + (act.astype(f32) @ lw["wd"].astype(f32).T)).astype(np.float64)
    tr = {"h_in": h_in, "a_attn": a1, "qkv": np.stack([s0, s1]), "q": q, "attn_out": ao,
          "h_mid": h_mid, "a_ffn": a2, "act": act, "h_out": h_out}
    return c, lw, tr, rows, caches, seq


def _check(c, lw, tr, rows, caches, seq):
    return check_layer(c, lw, tr, rows, [0, 1], seq, lambda slot, L: caches[slot], 1,
                       n_sample=24, seed=3)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_simulated_trace_passes(dtype):
    log = _check(*_simulate(dtype))
    assert {n for n, _, _ in log} >= {"attn_norm", "rope_q", "rope_k", "v_write", "attention",
                                      "gemm_o+residual", "ffn_norm", "swiglu",
                                      "gemm_down+residual"}


def _plant(dtype, how):
    c, lw, tr, rows, caches, seq = _simulate(dtype)
    tr = copy.deepcopy(tr)
    caches = [(K.copy(), V.copy()) for K, V in caches]
    if how == "dropped_k_term":
        W = np.concatenate([lw["wq"], lw["wk"], lw["wv"]])
        tr["qkv"][1] -= np.outer(tr["a_attn"][:, 100], W[:, 100])
    elif how == "rope_position":
        lw2 = dict(lw)
        xs = tr["qkv"][0] + tr["qkv"][1]
        n = xs.shape[0]
        qd = c.n_q_heads * c.head_dim
        pos = np.concatenate([np.arange(a, b) for a, b in rows]) + 1
        tr["q"] = _st(dtype, oracle.rope(xs[:, :qd].reshape(n, c.n_q_heads, c.head_dim), pos,
                                         c.rope_theta)).reshape(n, qd)
    elif how == "head_swap":
        q = tr["attn_out"].reshape(len(tr["attn_out"]), c.n_q_heads, -1)
        tr["attn_out"] = q[:, [1, 0, 2, 3]].reshape(len(q), -1)
    elif how == "missing_residual":
        tr["h_mid"] = tr["h_mid"] - tr["h_in"]
    elif how == "swiglu_swapped":
        a2 = tr["a_ffn"].astype(f32)
        g = a2 @ lw["wg"].astype(f32).T
        u = a2 @ lw["wu"].astype(f32).T
        tr["act"] = _st(dtype, (u / (f32(1) + np.exp(-u)) * g).astype(np.float64))
    elif how == "value_not_written":
        K, V = caches[1]
        V[30] = 0.0
    elif how == "norm_eps":
        tr["a_ffn"] = _st(dtype, _norm32(tr["h_mid"], lw["ffn_norm"], 1.0))
    return c, lw, tr, rows, caches, seq


@pytest.mark.parametrize("how", ["dropped_k_term", "rope_position", "head_swap",
                                 "missing_residual", "swiglu_swapped", "value_not_written",
                                 "norm_eps"])
def test_planted_mistakes_fail(how):
    with pytest.raises(AssertionError):
        _check(*_plant("bf16", how))


def test_head_unmask_rules():
    """Decisions from the GPU's own logits: exact away from the threshold,
    the forced single unmask among the tied top, and a wrong decision fails."""
    rng = np.random.default_rng(0)
    z = rng.standard_normal((8, 50)) * 3
    z[2, 7] += 12                                   # a confident position
    conf, tok = oracle.confidence(z)
    s = 100
    masked = np.arange(s, s + 8)
    gamma = 0.9
    sel = oracle.select_unmask(conf, gamma)
    out = {"n": int(sel.sum()), "pos": np.zeros(64, np.int64), "tok": np.zeros(64, np.int64),
           "conf": np.zeros(64), "block_conf": np.full(64, -1.0), "block_tok": np.zeros(64, np.int64)}
    out["pos"][:out["n"]] = masked[sel]
    out["tok"][:out["n"]] = tok[sel]
    out["conf"][:out["n"]] = conf[sel]
    out["block_conf"][:8] = conf
    out["block_tok"][:8] = tok
    counts = {}
    check_head_unmask(z, out, s, masked, gamma, counts)
    assert counts["checked"] == 8
    bad = copy.deepcopy(out)
    bad["n"] = 2
    bad["pos"][1] = s + 5
    with pytest.raises(AssertionError):
        check_head_unmask(z, bad, s, masked, gamma, {})
    # nothing passes: exactly the top one, and only it
    zf = rng.standard_normal((8, 50))
    cf, tf = oracle.confidence(zf)
    top = int(np.argmax(cf))
    forced = {"n": 1, "pos": np.full(64, s + top), "tok": np.full(64, tf[top]),
              "conf": np.full(64, cf[top]), "block_conf": np.r_[cf, -np.ones(56)],
              "block_tok": np.r_[tf, np.zeros(56, np.int64)]}
    c2 = {}
    check_head_unmask(zf, forced, s, masked, gamma, c2)
    wrong = copy.deepcopy(forced)
    other = (top + 1) % 8
    wrong["pos"][:] = s + other
    wrong["tok"][:] = tf[other]
    wrong["conf"][:] = cf[other]
    if cf[top] - cf[other] > 1e-3:
        with pytest.raises(AssertionError):
            check_head_unmask(zf, wrong, s, masked, gamma, {})
