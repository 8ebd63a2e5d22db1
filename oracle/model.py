"""CPU oracle for one denoising step of a masked-diffusion transformer.

TEST INFRASTRUCTURE. Only the tests, the smoke check and the benchmark's CPU
baseline may import this module; the product path never does. It shares no code
with the HIP library: it receives weights and tokens from the seeded input
generator (``synth``) and computes everything else itself, in float64.

What is computed (paper, "Background and Challenges", Diffusion Language
Models; "Support for Approximate Caching"; "Supporting Approximate KV Caching";
"Implementation"):

* the prompt followed by [MASK] tokens goes through one forward pass of a
  Transformer mask predictor with full bidirectional attention (no causal mask),
  which predicts every masked position at once;
* the confidence of a prediction is its softmax probability; every masked
  position whose confidence exceeds the threshold is unmasked, and when none
  does, the single most confident one is unmasked;
* generation proceeds block by block; with approximate KV caching the keys and
  values of the prompt, completed blocks and still-masked future blocks are
  reused while the current block is denoised, and everything is recomputed once
  a block is fully unmasked (recompute step) before the next block.

The architecture constants the paper leaves open (pre-norm RMSNorm, rotate-half
RoPE, SwiGLU, untied LM head, no biases, [MASK] = last vocabulary id) are the
readings listed with the design notes.

Precision: everything is float64. For bf16 models the value is rounded to bf16
(round-to-nearest-even) exactly where the GPU path stores bf16: the normed GEMM
inputs, Q/K/V after RoPE, the attention output, the SwiGLU product and the
final-normed LM-head input. The fp32 model is computed in float64 throughout.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Callable, List, Optional

import numpy as np


# ---------------------------------------------------------------- rounding --
def round_bf16(x) -> np.ndarray:
    """Round to the nearest bf16 value (ties to even) and return float64.

    Values are first rounded to fp32 (nearest-even, numpy's cast), then the low
    16 bits of the fp32 pattern are dropped with round-half-to-even."""
    f = np.asarray(x, dtype=np.float64).astype(np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    low = u & np.uint64(0xFFFF)
    high = u >> np.uint64(16)
    half = np.uint64(0x8000)
    odd = (high & np.uint64(1)) == np.uint64(1)
    up = (low > half) | ((low == half) & odd)
    high = high + up.astype(np.uint64)
    return (high << np.uint64(16)).astype(np.uint32).view(np.float32).astype(np.float64)


def storage(dtype: str) -> Callable[[np.ndarray], np.ndarray]:
    """Storage rounding of the model's activation type."""
    if dtype == "bf16":
        return round_bf16
    if dtype == "f32":
        return lambda x: np.asarray(x, dtype=np.float64)
    raise ValueError(dtype)


# ------------------------------------------------------------ primitives --
def rmsnorm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * g over the last axis."""
    x = np.asarray(x, np.float64)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * np.asarray(g, np.float64)


def rope(x: np.ndarray, pos: np.ndarray, theta: float) -> np.ndarray:
    """Rotary embedding, rotate-half form.

    x: [n, heads, dh]; pos: [n] absolute positions. Pair (i, i + dh/2) for
    i < dh/2 is rotated by the angle pos * theta^(-2i/dh)."""
    x = np.asarray(x, np.float64)
    dh = x.shape[-1]
    half = dh // 2
    freq = theta ** (-np.arange(half, dtype=np.float64) * 2.0 / dh)
    ang = np.asarray(pos, np.float64)[:, None] * freq[None, :]      # [n, half]
    c = np.cos(ang)[:, None, :]
    s = np.sin(ang)[:, None, :]
    x1 = x[..., :half]
    x2 = x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def softmax(z: np.ndarray) -> np.ndarray:
    z = np.asarray(z, np.float64)
    e = np.exp(z - z.max(axis=-1, keepdims=True))
    return e / e.sum(axis=-1, keepdims=True)


def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray) -> np.ndarray:
    """Bidirectional (non-causal) attention over every key.

    q: [nq, Hq, dh]; k, v: [L, Hkv, dh]. Query head h reads key/value head
    h // (Hq / Hkv). Returns [nq, Hq, dh]."""
    nq, hq, dh = q.shape
    hkv = k.shape[1]
    group = hq // hkv
    out = np.empty((nq, hq, dh), np.float64)
    scale = 1.0 / np.sqrt(dh)
    for h in range(hq):
        kh = k[:, h // group, :]
        vh = v[:, h // group, :]
        p = softmax((q[:, h, :] @ kh.T) * scale)
        out[:, h, :] = p @ vh
    return out


def confidence(z: np.ndarray):
    """Confidence and predicted token of each row of scaled logits z [M, V].

    The prediction is the most probable token (lowest id among equal maxima) and
    its confidence is its softmax probability, 1 / sum_v exp(z_v - max z)."""
    z = np.asarray(z, np.float64)
    m = z.max(axis=1)
    s = np.exp(z - m[:, None]).sum(axis=1)
    return 1.0 / s, np.argmax(z, axis=1).astype(np.int64)


def select_unmask(conf: np.ndarray, gamma: float) -> np.ndarray:
    """Boolean selection over masked positions (ascending position order).

    Positions whose confidence exceeds gamma (strictly) are selected; if none
    does and at least one position is masked, the most confident one (lowest
    position on ties) is selected alone."""
    conf = np.asarray(conf, np.float64)
    sel = conf > gamma
    if conf.size and not sel.any():
        sel[int(np.argmax(conf))] = True
    return sel


# ---------------------------------------------------------------- model --
class Weights:
    """Weight provider: ``layer(l)`` returns the dict of layer l and
    ``globals`` the embedding / LM head / final gain (float arrays, [out, in])."""

    def __init__(self, globals_: dict, layers: Optional[list] = None,
                 layer_fn: Optional[Callable[[int], dict]] = None, n_layers: int = 0):
        self.globals = globals_
        self._layers = layers
        self._fn = layer_fn
        self.n_layers = len(layers) if layers is not None else n_layers

    def layer(self, l: int) -> dict:
        if self._layers is not None:
            return self._layers[l]
        return self._fn(l)

    @staticmethod
    def from_dict(w: dict) -> "Weights":
        g = {k: w[k] for k in ("embed", "lm_head", "final_norm")}
        return Weights(g, layers=list(w["layers"]))


@dataclass
class Request:
    """State of one request: prompt then masked generation positions."""
    tokens: np.ndarray          # int64 [L]
    mask: np.ndarray            # bool [L], True = [MASK]
    prompt_len: int
    gen_len: int
    block: int
    gamma: float
    k: int = 0                  # index of the active block
    cache_k: Optional[list] = None   # per layer [L, Hkv, dh]
    cache_v: Optional[list] = None
    cache_block: Optional[int] = None  # block start at the last refresh

    @property
    def seq_len(self) -> int:
        return self.prompt_len + self.gen_len

    @property
    def block_bounds(self):
        s = self.prompt_len + self.k * self.block
        return s, min(s + self.block, self.seq_len)

    @property
    def done(self) -> bool:
        return self.k * self.block >= self.gen_len

    @staticmethod
    def new(prompt: np.ndarray, gen_len: int, block: int, gamma: float,
            mask_id: int) -> "Request":
        P = len(prompt)
        toks = np.concatenate([np.asarray(prompt, np.int64),
                               np.full(gen_len, mask_id, np.int64)])
        mask = np.zeros(P + gen_len, bool)
        mask[P:] = True
        return Request(toks, mask, P, gen_len, block, gamma)


def recompute_rows(req: Request, mode: str, refresh: bool):
    """Rows whose keys/values and hidden states a step recomputes.

    No cache or a recompute step: the whole sequence. Dual cache: the active
    block only. Prefix cache: the active block and everything after it."""
    L = req.seq_len
    s, e = req.block_bounds
    if mode == "none" or refresh:
        return 0, L
    if mode == "dual":
        return s, e
    if mode == "prefix":
        return s, L
    raise ValueError(mode)


def embed_rows(cfg, W: Weights, req: Request, r0: int, r1: int) -> np.ndarray:
    ids = np.where(req.mask[r0:r1], cfg.mask_id, req.tokens[r0:r1])
    return np.asarray(W.globals["embed"], np.float64)[ids]


def layer_forward(cfg, lw: dict, h: np.ndarray, r0: int, r1: int,
                  cache_k: np.ndarray, cache_v: np.ndarray) -> np.ndarray:
    """One pre-norm transformer layer for rows [r0, r1) of a request.

    The rows' post-RoPE keys and values overwrite cache rows [r0, r1); attention
    then reads every cached position. Returns the updated residual stream."""
    st = storage(cfg.dtype)
    n = r1 - r0
    hq, hkv, dh = cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
    pos = np.arange(r0, r1)
    a = st(rmsnorm(h, lw["attn_norm"], cfg.rms_eps))
    q = a @ np.asarray(lw["wq"], np.float64).T
    k = a @ np.asarray(lw["wk"], np.float64).T
    v = a @ np.asarray(lw["wv"], np.float64).T
    q = st(rope(q.reshape(n, hq, dh), pos, cfg.rope_theta))
    k = st(rope(k.reshape(n, hkv, dh), pos, cfg.rope_theta))
    v = st(v.reshape(n, hkv, dh))
    cache_k[r0:r1] = k
    cache_v[r0:r1] = v
    o = st(attention(q, cache_k, cache_v)).reshape(n, hq * dh)
    h = h + o @ np.asarray(lw["wo"], np.float64).T
    a = st(rmsnorm(h, lw["ffn_norm"], cfg.rms_eps))
    g = a @ np.asarray(lw["wg"], np.float64).T
    u = a @ np.asarray(lw["wu"], np.float64).T
    act = st(silu(g) * u)
    return h + act @ np.asarray(lw["wd"], np.float64).T


def head_logits(cfg, W: Weights, h_rows: np.ndarray, inv_tau: float) -> np.ndarray:
    """Scaled logits z = RMSNorm(h) W_lm^T * (1/tau) of the given rows."""
    st = storage(cfg.dtype)
    u = st(rmsnorm(h_rows, W.globals["final_norm"], cfg.rms_eps))
    return (u @ np.asarray(W.globals["lm_head"], np.float64).T) * float(inv_tau)


def ensure_cache(cfg, req: Request, n_layers: int):
    if req.cache_k is None:
        L = req.seq_len
        req.cache_k = [np.zeros((L, cfg.n_kv_heads, cfg.head_dim)) for _ in range(n_layers)]
        req.cache_v = [np.zeros((L, cfg.n_kv_heads, cfg.head_dim)) for _ in range(n_layers)]


def needs_refresh(req: Request, mode: str) -> bool:
    """In cache modes the first step of every block recomputes everything."""
    if mode == "none":
        return True
    return req.cache_block != req.block_bounds[0]


@dataclass
class StepResult:
    positions: np.ndarray       # unmasked positions, ascending
    tokens: np.ndarray          # their new tokens
    conf: np.ndarray            # their confidences
    masked_positions: np.ndarray  # masked active-block positions at step start
    masked_conf: np.ndarray     # confidence of each of them
    masked_tok: np.ndarray      # prediction of each of them
    logits: Optional[np.ndarray] = None   # scaled logits of the masked rows
    refresh: bool = False
    rows: tuple = (0, 0)


def step_forward(cfg, W: Weights, req: Request, mode: str,
                 refresh: Optional[bool] = None) -> tuple:
    """Run the forward of one step; returns (hidden rows, (r0, r1), refresh)."""
    if refresh is None:
        refresh = needs_refresh(req, mode)
    ensure_cache(cfg, req, W.n_layers)
    r0, r1 = recompute_rows(req, mode, refresh)
    h = embed_rows(cfg, W, req, r0, r1)
    for l in range(W.n_layers):
        h = layer_forward(cfg, W.layer(l), h, r0, r1, req.cache_k[l], req.cache_v[l])
    if refresh:
        req.cache_block = req.block_bounds[0]
    return h, (r0, r1), refresh


def finish_step(cfg, W: Weights, req: Request, h: np.ndarray, rows, refresh: bool,
                inv_tau: float, gamma: Optional[float] = None,
                keep_logits: bool = False, apply: bool = True) -> StepResult:
    """Confidence, unmask decision and state update from the step's hidden rows."""
    r0, _ = rows
    s, e = req.block_bounds
    A = np.nonzero(req.mask[s:e])[0] + s
    gamma = req.gamma if gamma is None else gamma
    if len(A):
        z = head_logits(cfg, W, h[A - r0], inv_tau)
        conf, tok = confidence(z)
    else:
        z = np.zeros((0, cfg.vocab))
        conf, tok = np.zeros(0), np.zeros(0, np.int64)
    sel = select_unmask(conf, gamma)
    res = StepResult(A[sel], tok[sel], conf[sel], A, conf, tok,
                     z if keep_logits else None, refresh, rows)
    if apply:
        req.tokens[res.positions] = res.tokens
        req.mask[res.positions] = False
        # advance past every block that is now fully unmasked
        while not req.done:
            s, e = req.block_bounds
            if req.mask[s:e].any():
                break
            req.k += 1
    return res


def denoise_step(cfg, W: Weights, req: Request, mode: str, inv_tau: float,
                 keep_logits: bool = False) -> StepResult:
    """One denoising step of one request (requests in a batch are independent)."""
    h, rows, refresh = step_forward(cfg, W, req, mode)
    return finish_step(cfg, W, req, h, rows, refresh, inv_tau, keep_logits=keep_logits)


def generate(cfg, W: Weights, prompts: List[np.ndarray], gen_lens: List[int],
             gammas: List[float], block: int, mode: str, inv_tau: float):
    """Denoise a batch to completion. Returns (requests, per-step trace).

    One batched step advances every unfinished request by one step."""
    reqs = [Request.new(p, g, block, gm, cfg.mask_id)
            for p, g, gm in zip(prompts, gen_lens, gammas)]
    trace = []
    while not all(r.done for r in reqs):
        step = []
        for i, r in enumerate(reqs):
            if r.done:
                continue
            res = denoise_step(cfg, W, r, mode, inv_tau)
            step.append((i, res))
        trace.append(step)
    return reqs, trace
