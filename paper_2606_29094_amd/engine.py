"""Host driver of the denoising step: device buffers, request bookkeeping and
the block-by-block generation loop around ``dlm_denoise_step``.

Block protocol (paper, "Support for Approximate Caching" and "Supporting
Approximate KV Caching"): the generation positions are split into blocks that
are denoised in order; with a cache, the first step of every block is a
recompute step that rewrites the request's slot, the following steps of the
block are cache steps; a request moves to the next block once its active block
has no [MASK] left, and is done after its last block. The host learns how many
positions a step unmasked from one small device-to-host copy per step.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional

import numpy as np
import torch

from . import dlm


# ------------------------------------------------------------------ model
@dataclass
class ModelShape:
    n_layers: int
    d_model: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    d_ffn: int
    vocab: int
    dtype: str                 # "f32" | "bf16"
    rms_eps: float = 1e-5
    rope_theta: float = 10000.0
    mask_id: Optional[int] = None

    @property
    def qkv_dim(self):
        return (self.n_q_heads + 2 * self.n_kv_heads) * self.head_dim

    @property
    def torch_dtype(self):
        return torch.bfloat16 if self.dtype == "bf16" else torch.float32

    @staticmethod
    def of(cfg) -> "ModelShape":
        return ModelShape(cfg.n_layers, cfg.d_model, cfg.n_q_heads, cfg.n_kv_heads,
                          cfg.head_dim, cfg.d_ffn, cfg.vocab, cfg.dtype, cfg.rms_eps,
                          cfg.rope_theta, cfg.vocab - 1)


class DeviceModel:
    """Caller-owned device weights plus the library's model handle.

    ``tensors``: embed, lm_head, final_norm and ``layers`` (list of dicts with
    attn_norm, w_qkv, w_o, ffn_norm, w_gate_up, w_down), torch CUDA tensors in
    the layouts of include/dlm.h."""

    def __init__(self, shape: ModelShape, tensors: dict, inv_tau: float):
        self.shape = shape
        self.tensors = tensors
        self.inv_tau = float(inv_tau)
        self._layer_arr = (dlm.DlmLayerWeights * shape.n_layers)(*[
            dlm.DlmLayerWeights(l["attn_norm"].data_ptr(), l["w_qkv"].data_ptr(),
                                l["w_o"].data_ptr(), l["ffn_norm"].data_ptr(),
                                l["w_gate_up"].data_ptr(), l["w_down"].data_ptr())
            for l in tensors["layers"]])
        self.weights = dlm.DlmWeights(tensors["embed"].data_ptr(), tensors["lm_head"].data_ptr(),
                                      tensors["final_norm"].data_ptr(),
                                      self._layer_arr)
        mask_id = shape.vocab - 1 if shape.mask_id is None else shape.mask_id
        self.config = dlm.DlmConfig(shape.n_layers, shape.d_model, shape.n_q_heads,
                                    shape.n_kv_heads, shape.head_dim, shape.d_ffn, shape.vocab,
                                    mask_id, shape.rms_eps, shape.rope_theta, self.inv_tau,
                                    dlm.DLM_BF16 if shape.dtype == "bf16" else dlm.DLM_F32)
        self.handle = dlm.load_weights(self.config, self.weights)

    def close(self):
        if self.handle:
            dlm.model_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


# ---------------------------------------------------------------- requests
@dataclass
class Request:
    prompt: np.ndarray
    gen_len: int
    block: int
    threshold: float
    slot: int = -1
    tok_offset: int = 0
    k: int = 0                         # active block index
    masked_in_block: int = 0
    refreshed_block: int = -1          # block_start of the last recompute step
    steps: int = 0
    unmasked: int = 0

    def __post_init__(self):
        # fixed for the request's life and read for every request of every
        # step: plain attributes keep the host's per-step work short
        self.prompt_len = len(self.prompt)
        self.seq_len = self.prompt_len + self.gen_len

    @property
    def block_start(self):
        return self.prompt_len + self.k * self.block

    @property
    def block_len(self):
        return min(self.block, self.seq_len - self.block_start)

    @property
    def done(self):
        return self.k * self.block >= self.gen_len


def advance(r: Request, unmasked: int) -> None:
    """Host bookkeeping after a step that unmasked `unmasked` positions of r's
    active block: a block is done when none of its positions is masked, and
    the next step of the request is then the recompute step of the next block."""
    r.steps += 1
    r.unmasked += unmasked
    r.masked_in_block -= unmasked
    if r.masked_in_block <= 0:
        r.k += 1
        if not r.done:
            r.masked_in_block = r.block_len


class Engine:
    """Slots, workspace and packed token/mask buffers for a fixed set of slots."""

    def __init__(self, model: DeviceModel, n_slots: int, max_seq_len: int, mode: str,
                 max_rows: Optional[int] = None, device="cuda:0", stats: bool = False):
        self.model = model
        self.mode = mode
        self.mode_id = dlm.MODES[mode]
        self.device = torch.device(device)
        self.n_slots = n_slots
        self.max_seq_len = max_seq_len
        _, need = dlm.kv_cache_alloc(model.handle, n_slots, max_seq_len)
        self.cache_buf = torch.empty(need, dtype=torch.uint8, device=self.device)
        self.cache, _ = dlm.kv_cache_alloc(model.handle, n_slots, max_seq_len, self.cache_buf,
                                           need)
        if max_rows is None:
            max_rows = n_slots * max_seq_len
        self.max_rows = max_rows
        ws = dlm.workspace_bytes(model.handle, max_rows, min(n_slots, dlm.DLM_MAX_REQ))
        self.workspace = torch.empty(ws, dtype=torch.uint8, device=self.device)
        self.tokens = torch.zeros(n_slots * max_seq_len, dtype=torch.int32, device=self.device)
        self.mask = torch.zeros(n_slots * max_seq_len, dtype=torch.uint8, device=self.device)
        # confidence each position was unmasked with, and the per-request
        # statistics of those of the output tokens (Step Predictor features)
        self.tok_conf = (torch.zeros(n_slots * max_seq_len, dtype=torch.float32,
                                     device=self.device) if stats else None)
        R = n_slots
        B = dlm.DLM_MAX_BLOCK
        self.n_unmasked = torch.zeros(R, dtype=torch.int32, device=self.device)
        self.out_pos = torch.zeros(R * B, dtype=torch.int32, device=self.device)
        self.out_tok = torch.zeros(R * B, dtype=torch.int32, device=self.device)
        self.out_conf = torch.zeros(R * B, dtype=torch.float32, device=self.device)
        self.block_conf = torch.zeros(R * B, dtype=torch.float32, device=self.device)
        self.block_tok = torch.zeros(R * B, dtype=torch.int32, device=self.device)
        self.stats = (torch.zeros(R * dlm.DLM_NSTATS, dtype=torch.float32, device=self.device)
                      if stats else None)
        self.host_n = torch.zeros(R, dtype=torch.int32).pin_memory()
        self.step_out = dlm.make_step_out(self.n_unmasked, self.out_pos, self.out_tok,
                                          self.out_conf, self.block_conf, self.block_tok,
                                          self.stats)
        self.free_slots = list(range(n_slots))[::-1]

    def close(self):
        if getattr(self, "cache", None):
            dlm.cache_destroy(self.cache)
            self.cache = None

    # ---- admission
    def admit(self, req: Request, mask_id: int):
        if req.seq_len > self.max_seq_len:
            raise ValueError("request longer than a slot")
        req.slot = self.free_slots.pop()
        req.tok_offset = req.slot * self.max_seq_len
        toks = np.concatenate([np.asarray(req.prompt, np.int32),
                               np.full(req.gen_len, mask_id, np.int32)])
        msk = np.concatenate([np.zeros(req.prompt_len, np.uint8), np.ones(req.gen_len, np.uint8)])
        o = req.tok_offset
        self.tokens[o:o + req.seq_len].copy_(torch.from_numpy(toks))
        self.mask[o:o + req.seq_len].copy_(torch.from_numpy(msk))
        req.k = 0
        req.masked_in_block = req.block_len
        req.refreshed_block = -1
        dlm.cache_invalidate(self.cache, req.slot)

    def release(self, req: Request):
        self.free_slots.append(req.slot)
        req.slot = -1

    def set_state(self, req: Request, tokens: np.ndarray, mask: np.ndarray, k: int,
                  tok_conf: Optional[np.ndarray] = None):
        """Overwrite a request's tokens/mask/block (teacher forcing in tests)."""
        o = req.tok_offset
        self.tokens[o:o + req.seq_len].copy_(torch.from_numpy(np.asarray(tokens, np.int32)))
        self.mask[o:o + req.seq_len].copy_(torch.from_numpy(np.asarray(mask, np.uint8)))
        if tok_conf is not None:
            self.tok_conf[o:o + req.seq_len].copy_(
                torch.from_numpy(np.asarray(tok_conf, np.float32)))
        req.k = k
        if not req.done:
            s = req.block_start
            req.masked_in_block = int(np.asarray(mask[s:s + req.block_len]).sum())

    # ---- one step
    def dlm_reqs(self, reqs: List[Request], force_refresh: bool = False):
        # runs between a step's read-back and the next step's launch, while
        # the GPU waits: one pass, no property calls
        all_refresh = force_refresh or self.mode_id == dlm.DLM_CACHE_NONE
        flag = dlm.DLM_REQ_REFRESH
        make = dlm.DlmReq
        out = []
        for r in reqs:
            s = r.prompt_len + r.k * r.block
            n = r.seq_len - s
            out.append(make(r.slot, r.seq_len, r.prompt_len, s, r.block if r.block < n else n,
                            r.tok_offset, flag if all_refresh or r.refreshed_block != s else 0))
        return out

    def enqueue_step(self, reqs: List[Request], stream=None, force_refresh: bool = False):
        """Enqueue one step; force_refresh makes it a refresh (recompute) step
        for every request."""
        dreqs = self.dlm_reqs(reqs, force_refresh)
        batch = dlm.make_batch(dreqs, self.tokens, self.mask, self.mode_id, self.tok_conf)
        dlm.denoise_step(self.model.handle, self.cache, batch, [r.threshold for r in reqs],
                         self.step_out, self.workspace, stream)
        for r, d in zip(reqs, dreqs):
            if d.flags & dlm.DLM_REQ_REFRESH:
                r.refreshed_block = r.block_start
        return dreqs

    def finish_step(self, reqs: List[Request], stream=None):
        """Read the unmask counts back and advance blocks (synchronises)."""
        n = len(reqs)
        self.host_n[:n].copy_(self.n_unmasked[:n], non_blocking=True)
        torch.cuda.current_stream().synchronize() if stream is None else \
            torch.cuda.ExternalStream(stream).synchronize()
        counts = self.host_n[:n].tolist()
        for r, c in zip(reqs, counts):
            advance(r, c)
        return counts

    def step(self, reqs: List[Request], stream=None):
        self.enqueue_step(reqs, stream)
        return self.finish_step(reqs, stream)

    def debug_logits(self, reqs: List[Request]):
        dreqs = self.dlm_reqs(reqs)
        nblk = sum(d.block_len for d in dreqs)
        out = torch.empty(nblk, self.model.shape.vocab, dtype=torch.float32, device=self.device)
        batch = dlm.make_batch(dreqs, self.tokens, self.mask, self.mode_id)
        dlm.debug_logits(self.model.handle, self.cache, batch, out, self.workspace)
        for r, d in zip(reqs, dreqs):
            if d.flags & dlm.DLM_REQ_REFRESH:
                r.refreshed_block = r.block_start
        return out

    def step_rows(self, reqs: List[Request], force_refresh: bool = False):
        """[r0, r1) of the positions each request's next step recomputes, in
        the packed row order of the step."""
        rows = []
        for r, d in zip(reqs, self.dlm_reqs(reqs, force_refresh)):
            if d.flags & dlm.DLM_REQ_REFRESH:
                rows.append((0, r.seq_len))
            elif self.mode == "dual":
                rows.append((r.block_start, r.block_start + r.block_len))
            else:
                rows.append((r.block_start, r.seq_len))
        return rows

    def debug_trace(self, reqs: List[Request], layer: int, logits: bool = True,
                    qkv_cap: int = 8):
        """Intermediates of layer `layer` of the forward of the step about to
        run (dlm_debug_trace; cache writes as the step's), as device tensors,
        plus the scaled logits and final-normed rows of every active-block
        position when `logits`. Returns (buffers, QKV K-split slices)."""
        sh = self.model.shape
        dt = sh.torch_dtype
        dreqs = self.dlm_reqs(reqs)
        n = sum(r1 - r0 for r0, r1 in self.step_rows(reqs))
        nblk = sum(d.block_len for d in dreqs)
        qd = sh.n_q_heads * sh.head_dim
        dev = self.device
        e = lambda *shape, dtype=torch.float32: torch.empty(*shape, dtype=dtype, device=dev)
        buf = {"h_in": e(n, sh.d_model), "a_attn": e(n, sh.d_model, dtype=dt),
               "qkv": e(qkv_cap, n, sh.qkv_dim), "q": e(n, qd, dtype=dt),
               "attn_out": e(n, qd, dtype=dt), "h_mid": e(n, sh.d_model),
               "a_ffn": e(n, sh.d_model, dtype=dt), "act": e(n, sh.d_ffn, dtype=dt),
               "h_out": e(n, sh.d_model)}
        if logits:
            buf["u"] = e(nblk, sh.d_model, dtype=dt)
            buf["logits"] = e(nblk, sh.vocab)
        batch = dlm.make_batch(dreqs, self.tokens, self.mask, self.mode_id)
        splits = dlm.debug_trace(self.model.handle, self.cache, batch, layer, buf, qkv_cap,
                                 self.workspace)
        for r, d in zip(reqs, dreqs):
            if d.flags & dlm.DLM_REQ_REFRESH:
                r.refreshed_block = r.block_start
        buf["qkv"] = buf["qkv"][:splits]
        return buf, splits

    def read_kv(self, layer: int, slot: int, length: int):
        """Keys and values of positions [0, length) of a slot at one layer, as
        [length, n_kv_heads, head_dim] float tensors on the host, read from the
        cache layout of dlm_kv_cache_alloc (per layer a key region
        [slot][kv_head][pos][head_dim] then a value region
        [slot][kv_head][head_dim][pos], slots of max_seq_len rounded up to 64)."""
        sh = self.model.shape
        dt = sh.torch_dtype
        s_max = (self.max_seq_len + 63) // 64 * 64
        per = self.n_slots * sh.n_kv_heads * s_max * sh.head_dim
        region = self.cache_buf.view(dt)
        k = region[(2 * layer) * per:(2 * layer + 1) * per].view(
            self.n_slots, sh.n_kv_heads, s_max, sh.head_dim)[slot, :, :length]
        v = region[(2 * layer + 1) * per:(2 * layer + 2) * per].view(
            self.n_slots, sh.n_kv_heads, sh.head_dim, s_max)[slot, :, :, :length]
        return (k.permute(1, 0, 2).float().cpu(), v.permute(2, 0, 1).float().cpu())

    def refresh(self, reqs: List[Request]):
        dreqs = self.dlm_reqs(reqs, force_refresh=True)
        batch = dlm.make_batch(dreqs, self.tokens, self.mask, self.mode_id)
        dlm.cache_refresh(self.model.handle, self.cache, batch, self.workspace)
        for r in reqs:
            r.refreshed_block = r.block_start

    def read_state(self, req: Request):
        o = req.tok_offset
        return (self.tokens[o:o + req.seq_len].cpu().numpy().astype(np.int64),
                self.mask[o:o + req.seq_len].cpu().numpy().astype(bool))

    def read_outputs(self, n_req: int):
        B = dlm.DLM_MAX_BLOCK
        out = {
            "n": self.n_unmasked[:n_req].cpu().numpy(),
            "pos": self.out_pos[:n_req * B].view(n_req, B).cpu().numpy(),
            "tok": self.out_tok[:n_req * B].view(n_req, B).cpu().numpy(),
            "conf": self.out_conf[:n_req * B].view(n_req, B).cpu().numpy(),
            "block_conf": self.block_conf[:n_req * B].view(n_req, B).cpu().numpy(),
            "block_tok": self.block_tok[:n_req * B].view(n_req, B).cpu().numpy(),
        }
        if self.stats is not None:
            out["stats"] = self.stats[:n_req * dlm.DLM_NSTATS].view(n_req, dlm.DLM_NSTATS).cpu().numpy()
        return out

    def save_state(self, req: Request):
        """Host copy of what a request needs to resume elsewhere (tokens, mask,
        token confidences, block index): a few bytes per position, no KV."""
        toks, msk = self.read_state(req)
        tc = None if self.tok_conf is None else self.read_tok_conf(req)
        return (toks, msk.astype(np.uint8), tc, req.k)

    def restore_state(self, req: Request, state) -> None:
        """After admit(): put a saved request back; its next step is a recompute."""
        toks, msk, tc, k = state
        self.set_state(req, toks, msk, k, tc)

    def read_tok_conf(self, req: Request) -> np.ndarray:
        o = req.tok_offset
        return self.tok_conf[o:o + req.seq_len].cpu().numpy()
