"""Plain float64 CPU oracle of the masked-diffusion denoising step.

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, by ``__graft_entry__.smoke``
and by the CPU-baseline leg of ``bench.py``. The HIP library never calls it and
shares no code with it.

Parity status of each function (what pins it is in ``tests/test_oracle_*.py``):
every function here is pinned by closed forms, invariants, brute force or an
independent library formulation; the full-scale bf16 trajectories are compared
with the GPU only (parity unpinned beyond the per-function pins).
"""
from .model import (round_bf16, storage, rmsnorm, rope, silu, softmax, attention,
                    confidence, select_unmask, Weights, Request, recompute_rows,
                    embed_rows, layer_forward, head_logits, needs_refresh,
                    step_forward, finish_step, denoise_step, generate, StepResult,
                    ensure_cache)
from .calibrate import calibrate, tau_star, top_prob

__all__ = [
    "round_bf16", "storage", "rmsnorm", "rope", "silu", "softmax", "attention",
    "confidence", "select_unmask", "Weights", "Request", "recompute_rows",
    "embed_rows", "layer_forward", "head_logits", "needs_refresh", "step_forward",
    "finish_step", "denoise_step", "generate", "StepResult", "ensure_cache",
    "calibrate", "tau_star", "top_prob",
]
