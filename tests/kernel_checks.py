"""Kernel-level parity on identical inputs.

Every kernel of a traced layer (dlm_debug_trace) is compared with the
oracle's operation applied to the exact values that kernel was given on the
GPU, so the comparison measures the kernel alone and not the drift of the
whole forward. The LM head and the unmask rule are checked the same way: the
oracle's confidence and selection applied to the GPU's own logits of the step
(dlm_debug_logits / the trace's logits) against the GPU step's outputs.

Tolerances come from the arithmetic of each kernel, not from end-to-end
drift. With u = 2^-24 (fp32 unit roundoff):

* stored values (bf16 storage, or fp32 for the fp32 model): the GPU computes
  in fp32 and rounds once, so its value lies within half an ulp of the storage
  type plus the fp32 error of the computation (``slack``) from the exact
  result of the same inputs;
* GEMMs: bf16 products are exact in fp32 and each 16x16x32 MFMA adds 32 of
  them to an fp32 accumulator, so the accumulated error is bounded by
  (K/32 + S + 2) u sum_k |a_k w_k| (S = K-split slices summed afterwards);
  the fp32 model's 16x16x4 MFMAs round every product: (K/2 + S + 2) u;
* attention: P enters the PV product as two bf16 terms (hi + lo, 16
  significant bits: |P - hi - lo| <= 2^-18 P), exp2 and the folded scale add
  a few fp32 ulps, sums over L keys (L/16) u: slack (2^-15 + (L/16) u) max|v|;
* SwiGLU: the GEMM bounds of g and u propagated through silu(g) u
  (|silu'| <= 1.1) plus 8 u for exp and the hardware reciprocal.
"""
from __future__ import annotations

import numpy as np

import oracle

U = 2.0 ** -24
CONF_TOL = 1e-3


def half_ulp(x, dtype):
    """Half the spacing of the storage type at |x| (bf16: 8 significant bits;
    fp32: 24)."""
    a = np.maximum(np.abs(np.asarray(x, np.float64)), 2.0 ** -126)
    e = np.floor(np.log2(a))
    return 2.0 ** (e - (8 if dtype == "bf16" else 24))


def check_stored(name, got, ref, slack, dtype, log):
    """got: stored GPU values; ref: exact result of the same inputs (fp64)."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    bound = half_ulp(ref, dtype) + np.asarray(slack, np.float64) + 1e-30
    err = np.abs(got - ref)
    worst = float((err / bound).max()) if err.size else 0.0
    if dtype == "bf16":
        rounded = oracle.round_bf16(ref)
    else:
        rounded = ref.astype(np.float32).astype(np.float64)
    differ = float(np.mean(got != rounded)) if err.size else 0.0
    log.append((name, worst, differ))
    assert worst <= 1.0, (name, worst, float(err.max()))
    if dtype == "bf16":
        # bf16 values off the correctly rounded result are those within the
        # fp32 slack of a rounding boundary: a small share (in fp32 storage the
        # slack is comparable to the half ulp itself)
        assert differ <= 0.02, (name, differ)


def check_close(name, got, ref, tol, log):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    err = np.abs(got - ref)
    worst = float((err / (np.asarray(tol) + 1e-30)).max()) if err.size else 0.0
    log.append((name, worst, None))
    assert worst <= 1.0, (name, worst, float(err.max()))


def gemm_tol(a, w, splits, dtype):
    """Accumulation bound of rows a [n, K] times w [N, K]^T."""
    K = a.shape[1]
    c = (K / 32.0 if dtype == "bf16" else K / 2.0) + splits + 2
    return c * U * (np.abs(a) @ np.abs(w).T)


def sample_rows(n, k, seed, must=()):
    """Up to k packed rows: the first and last few, the given ones, and a
    seeded sample of the rest."""
    rng = np.random.default_rng(seed)
    base = set(range(min(4, n))) | set(range(max(0, n - 4), n)) | {m for m in must if 0 <= m < n}
    rest = np.setdiff1d(np.arange(n), np.array(sorted(base), dtype=np.int64))
    extra = rng.choice(rest, size=min(len(rest), max(0, k - len(base))), replace=False) \
        if len(rest) else np.zeros(0, np.int64)
    return np.array(sorted(base | set(int(x) for x in extra)), dtype=np.int64)


def packed_rows(rows):
    """rows: [(r0, r1)] per request -> list of (first packed row, r0, r1)."""
    out, off = [], 0
    for r0, r1 in rows:
        out.append((off, r0, r1))
        off += r1 - r0
    return out


def check_layer(cfg, lw, tr, rows, slots, seq_lens, read_kv, layer, n_sample=48, seed=0,
                embed=None, ids=None):
    """Check one traced layer kernel by kernel. tr: host float64 arrays of the
    trace; rows: [(r0, r1)] per request; slots / seq_lens per request;
    read_kv(slot, L) -> (K, V) [L, Hkv, dh] of this layer after the step's
    writes; embed / ids (layer 0): the embedding matrix and, per request, the
    embedding id of every position ([MASK] where masked).
    Returns the log [(check, worst error / bound, share off the rounded result)]."""
    dt = cfg.dtype
    hq, hkv, dh, d = cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, cfg.d_model
    qd, kd = hq * dh, hkv * dh
    log = []
    pk = packed_rows(rows)
    n = pk[-1][0] + pk[-1][2] - pk[-1][1]
    must = [p for p, _, _ in pk] + [p + (r1 - r0) - 1 for p, r0, r1 in pk]
    S = sample_rows(n, n_sample, seed, must)
    req_of = np.searchsorted(np.array([p for p, _, _ in pk]), S, side="right") - 1
    pos = np.array([pk[r][1] + (s - pk[r][0]) for s, r in zip(S, req_of)])

    h_in = tr["h_in"][S]
    if layer == 0 and ids is not None:
        emb = np.asarray(embed, np.float64)[[int(ids[r][p]) for r, p in zip(req_of, pos)]]
        assert np.array_equal(h_in, emb), "embedding rows"
        log.append(("embed", 0.0, 0.0))
    a1 = tr["a_attn"][S]
    ref = oracle.rmsnorm(h_in, lw["attn_norm"], cfg.rms_eps)
    check_stored("attn_norm", a1, ref, 1e-5 * np.abs(ref), dt, log)

    # QKV projection, each K-split slice over its own K range
    wqkv = np.concatenate([lw["wq"], lw["wk"], lw["wv"]]).astype(np.float64)
    slices = tr["qkv"][:, S]
    ns = slices.shape[0]
    kw = d // ns
    for s in range(ns):
        a_s, w_s = a1[:, s * kw:(s + 1) * kw], wqkv[:, s * kw:(s + 1) * kw]
        check_close(f"gemm_qkv[{s}/{ns}]", slices[s], a_s @ w_s.T, gemm_tol(a_s, w_s, 0, dt), log)
    xs = slices[0].astype(np.float32)
    for s in range(1, ns):
        xs = xs + slices[s].astype(np.float32)          # the consumer's order
    xs = xs.astype(np.float64)

    # rotary embedding and the key/value write
    def rope_check(name, got, x):
        x = x.reshape(len(S), -1, dh)
        ref = oracle.rope(x, pos, cfg.rope_theta)
        mag = np.abs(x[..., :dh // 2]) + np.abs(x[..., dh // 2:])
        slack = 4 * U * np.concatenate([mag, mag], axis=-1)
        check_stored(name, got.reshape(ref.shape), ref, slack, dt, log)

    rope_check("rope_q", tr["q"][S], xs[:, :qd])
    kv_cache = {}
    for r in sorted(set(req_of.tolist())):
        kv_cache[r] = read_kv(slots[r], seq_lens[r])
    k_got = np.stack([kv_cache[r][0][p] for r, p in zip(req_of, pos)])
    v_got = np.stack([kv_cache[r][1][p] for r, p in zip(req_of, pos)])
    rope_check("rope_k", k_got, xs[:, qd:qd + kd])
    v_ref = oracle.storage(dt)(xs[:, qd + kd:].reshape(len(S), hkv, dh))
    assert np.array_equal(v_got, v_ref), "value rows differ from the rounded projection"
    log.append(("v_write", 0.0, 0.0))

    # attention over every key of the slot, from the GPU's own queries/keys/values
    q = tr["q"][S].reshape(len(S), hq, dh)
    o_ref = np.empty((len(S), hq, dh))
    slack = np.empty((len(S), hq, dh))
    for r in sorted(set(req_of.tolist())):
        sel = req_of == r
        K, V = kv_cache[r]
        o_ref[sel] = oracle.attention(q[sel], K, V)
        L = K.shape[0]
        vmax = np.abs(V).max(axis=(0, 2))                     # per kv head
        grp = hq // hkv
        vm = np.repeat(vmax, grp)[None, :, None]
        c = (2.0 ** -15 if dt == "bf16" else 0.0) + (L / 16.0 + 16) * U
        slack[sel] = c * vm
    check_stored("attention", tr["attn_out"][S].reshape(o_ref.shape), o_ref, slack, dt, log)

    # output projection + residual
    ao = tr["attn_out"][S]
    wo = np.asarray(lw["wo"], np.float64)
    h_mid = tr["h_mid"][S]
    tol = gemm_tol(ao, wo, 8, dt) + 9 * U * (np.abs(h_in) + np.abs(h_mid))
    check_close("gemm_o+residual", h_mid - h_in, ao @ wo.T, tol, log)

    a2 = tr["a_ffn"][S]
    ref = oracle.rmsnorm(h_mid, lw["ffn_norm"], cfg.rms_eps)
    check_stored("ffn_norm", a2, ref, 1e-5 * np.abs(ref), dt, log)

    # SwiGLU
    wg = np.asarray(lw["wg"], np.float64)
    wu = np.asarray(lw["wu"], np.float64)
    g, u = a2 @ wg.T, a2 @ wu.T
    dg, du = gemm_tol(a2, wg, 0, dt), gemm_tol(a2, wu, 0, dt)
    sg = oracle.silu(g)
    ref = sg * u
    slack = 1.1 * dg * np.abs(u) + np.abs(sg) * du + 8 * U * np.abs(ref)
    check_stored("swiglu", tr["act"][S], ref, slack, dt, log)

    # down projection + residual
    act = tr["act"][S]
    wd = np.asarray(lw["wd"], np.float64)
    h_out = tr["h_out"][S]
    tol = gemm_tol(act, wd, 8, dt) + 9 * U * (np.abs(h_mid) + np.abs(h_out))
    check_close("gemm_down+residual", h_out - h_mid, act @ wd.T, tol, log)
    return log


def check_final_head(cfg, W, tr, rows, blocks, inv_tau, n_sample=16, seed=0):
    """Final norm and logits of the active-block rows (trace of the last
    layer): u against RMSNorm of the GPU's last residual rows, the scaled
    logits against u W_lm^T / tau on the GPU's own u. blocks: (block_start,
    block_len) per request."""
    dt = cfg.dtype
    log = []
    pk = packed_rows(rows)
    brow, prow = [], []
    off = 0
    for (p0, r0, _), (s, bl) in zip(pk, blocks):
        for j in range(bl):
            brow.append(off + j)
            prow.append(p0 + (s + j - r0))
        off += bl
    brow, prow = np.array(brow), np.array(prow)
    pick = sample_rows(len(brow), n_sample, seed)
    u = tr["u"][brow[pick]]
    ref = oracle.rmsnorm(tr["h_out"][prow[pick]], W.globals["final_norm"], cfg.rms_eps)
    check_stored("final_norm", u, ref, 1e-5 * np.abs(ref), dt, log)
    wl = np.asarray(W.globals["lm_head"], np.float64)
    z = np.empty((len(pick), wl.shape[0]))
    tol = np.empty_like(z)
    for c in range(0, wl.shape[0], 32768):
        wc = wl[c:c + 32768]
        z[:, c:c + 32768] = (u @ wc.T) * inv_tau
        tol[:, c:c + 32768] = gemm_tol(u, wc, 0, dt) * inv_tau
    zg = tr["logits"][brow[pick]]
    check_close("logits", zg, z, tol + 2 * U * np.abs(z), log)
    return log


def check_head_unmask(z_blk, out_r, blk_start, masked, gamma, counts):
    """The fused head's confidences/predictions and the unmask decision of one
    request's step against the oracle's confidence() and select_unmask() on
    the GPU's own scaled logits z_blk [block_len, V] of that step.

    masked: the masked block positions at step start. Decisions must be exact
    except at positions whose confidence is within 1e-3 of the threshold, and,
    on a step where nothing passes, among positions within 1e-3 of the top
    confidence (then exactly one of them must be unmasked). counts collects
    checked / exempt positions."""
    A = np.asarray(masked, np.int64)
    n = int(out_r["n"])
    got = set(out_r["pos"][:n].tolist())
    assert len(got) == n, "duplicate positions"
    if len(A) == 0:
        assert n == 0
        return
    assert n >= 1
    conf, tok = oracle.confidence(z_blk[A - blk_start])
    bc = out_r["block_conf"][A - blk_start]
    cerr = np.abs(bc - conf)
    counts["conf_err"] = max(counts.get("conf_err", 0.0), float(cerr.max()))
    assert cerr.max() <= CONF_TOL, cerr.max()
    # predictions: equal unless the two largest logits are within the fp32
    # accumulation-order difference of the fused head and the logits GEMM
    zs = np.sort(z_blk[A - blk_start], axis=1)
    tie = (zs[:, -1] - zs[:, -2]) <= 1e-5 * np.abs(zs).max(axis=1) + 1e-6
    bt = out_r["block_tok"][A - blk_start]
    assert np.all((bt == tok) | tie), "predicted tokens"
    counts["tok_tie"] = counts.get("tok_tie", 0) + int(tie.sum())
    want = set(A[oracle.select_unmask(conf, gamma)].tolist())
    near = set(A[np.abs(conf - gamma) <= CONF_TOL].tolist())
    if np.any(conf > gamma):
        assert (got ^ want) <= near, (sorted(got), sorted(want), sorted(near))
        counts["checked"] = counts.get("checked", 0) + len(A) - len(near)
        counts["near"] = counts.get("near", 0) + len(near)
    else:
        top = A[conf >= conf.max() - CONF_TOL]
        if len(top) == 1 and not near:
            assert got == want, (sorted(got), sorted(want))
            counts["checked"] = counts.get("checked", 0) + len(A)
        else:
            # near-tie of the top confidences, or the top near the threshold:
            # exactly the forced one among the tied top, or positions near the
            # threshold that passed on the GPU
            assert got <= set(top.tolist()) | near, (sorted(got), sorted(top), sorted(near))
            if not (got & near):
                assert n == 1
            counts["checked"] = counts.get("checked", 0) + len(A) - len(set(top.tolist()) | near)
            counts["tie_top"] = counts.get("tie_top", 0) + len(top)
    # the unmasked tokens and confidences are the ones reported for the block
    for p, t, c in zip(out_r["pos"][:n], out_r["tok"][:n], out_r["conf"][:n]):
        assert t == out_r["block_tok"][p - blk_start] and c == out_r["block_conf"][p - blk_start]


# ------------------------------------------------------------ GPU drivers --
class DevArray:
    """A device tensor read on demand: indexing gathers the rows on the device
    and returns them to the host as float64."""

    def __init__(self, t):
        self.t = t

    @property
    def shape(self):
        return tuple(self.t.shape)

    def __getitem__(self, idx):
        import torch
        conv = lambda i: torch.as_tensor(i, device=self.t.device) if isinstance(i, np.ndarray) else i
        idx = tuple(conv(i) for i in idx) if isinstance(idx, tuple) else conv(idx)
        return self.t[idx].double().cpu().numpy()


def host_layer(tensors, cfg, l):
    """One layer's device weights in the oracle's dict layout (float32 host
    copies of the generator's values)."""
    qd, kd = cfg.n_q_heads * cfg.head_dim, cfg.n_kv_heads * cfg.head_dim
    f = lambda t: t.float().cpu().numpy()
    lt = tensors["layers"][l]
    qkv, gu = f(lt["w_qkv"]), f(lt["w_gate_up"])
    return {"wq": qkv[:qd], "wk": qkv[qd:qd + kd], "wv": qkv[qd + kd:], "wo": f(lt["w_o"]),
            "wg": gu[:cfg.d_ffn], "wu": gu[cfg.d_ffn:], "wd": f(lt["w_down"]),
            "attn_norm": f(lt["attn_norm"]), "ffn_norm": f(lt["ffn_norm"])}


def trace_step_and_check(cfg, tensors, eng, reqs, layers, inv_tau, n_sample=48, seed=0,
                         head_rows=16, W_globals=None):
    """Trace the given layers of the step about to run (identical-input checks
    of every kernel), then run the step itself and check the fused head and
    the unmask decision of every request against the oracle's confidence and
    selection on the GPU's own logits. Returns (per-layer logs, counts, step
    outputs)."""
    import oracle as _o
    rows = eng.step_rows(reqs)
    saved = [r.refreshed_block for r in reqs]
    states = [eng.read_state(r) for r in reqs]
    ids = [np.where(m, cfg.mask_id, t) for t, m in states]
    slots = [r.slot for r in reqs]
    seq_lens = [r.seq_len for r in reqs]
    logs = {}
    z = None
    last = cfg.n_layers - 1 if hasattr(cfg, "n_layers") else None
    if W_globals is None:
        f = lambda t: t.float().cpu().numpy()
        W_globals = {"embed": f(tensors["embed"]), "lm_head": f(tensors["lm_head"]),
                     "final_norm": f(tensors["final_norm"])}
    n_layers = len(tensors["layers"])
    for i, l in enumerate(layers):
        want_logits = (l == n_layers - 1) or (i == len(layers) - 1 and z is None)
        buf, splits = eng.debug_trace(reqs, l, logits=want_logits)
        for r, s in zip(reqs, saved):
            r.refreshed_block = s
        tr = {k: DevArray(v) for k, v in buf.items()}
        read_kv = lambda slot, L, l=l: tuple(x.double().numpy() for x in eng.read_kv(l, slot, L))
        lw = host_layer(tensors, cfg, l)
        logs[l] = check_layer(cfg, lw, tr, rows, slots, seq_lens, read_kv, l, n_sample, seed + l,
                              embed=W_globals["embed"], ids=ids)
        if want_logits:
            z = buf["logits"].cpu().numpy()
            if l == n_layers - 1:
                W = _o.Weights(W_globals, layers=[])
                blocks = [(r.block_start, r.block_len) for r in reqs]
                logs["head"] = check_final_head(cfg, W, tr, rows, blocks, inv_tau, head_rows, seed)
        del buf, tr
    starts = [r.block_start for r in reqs]
    lens = [r.block_len for r in reqs]
    eng.step(reqs)
    out = eng.read_outputs(len(reqs))
    counts = {}
    off = 0
    for j, (r, (t, m)) in enumerate(zip(reqs, states)):
        s, L = starts[j], lens[j]
        masked = np.nonzero(m[s:s + L])[0] + s
        check_head_unmask(z[off:off + L], {k: v[j] for k, v in out.items()}, s, masked,
                          r.threshold, counts)
        off += L
    assert counts.get("checked", 0) > 0, counts
    return logs, counts, out


def summarize(logs):
    """worst error / bound per check over the traced layers (for the log)."""
    worst = {}
    for l, lg in logs.items():
        for name, w, _ in lg:
            worst[name] = max(worst.get(name, 0.0), w)
    return {k: round(v, 3) for k, v in worst.items()}
