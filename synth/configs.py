"""Model shapes and workload recipes for the synthetic denoising workloads.

Pure data: no arithmetic of the method lives here. The shapes are the ones the
benchmarks name (a tiny fp32 model, an LLaDA-8B-shaped MHA model and a
Dream-7B-shaped GQA model); the paper itself names only the two open models
(Evaluation, Experimental Setup) and the block size 32 / threshold 0.9 defaults.
"""
from __future__ import annotations

from dataclasses import dataclass, field, asdict
from typing import Optional, Tuple


@dataclass(frozen=True)
class ModelConfig:
    name: str
    n_layers: int
    d_model: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    d_ffn: int
    vocab: int
    dtype: str            # "f32" or "bf16": storage type of weights and activations
    rms_eps: float = 1e-5
    rope_theta: float = 10000.0
    weight_std: float = 0.02
    weight_seed: int = 0

    @property
    def mask_id(self) -> int:
        # [MASK] is the last vocabulary entry.
        return self.vocab - 1

    @property
    def qkv_dim(self) -> int:
        return (self.n_q_heads + 2 * self.n_kv_heads) * self.head_dim

    @property
    def layer_params(self) -> int:
        d, dh = self.d_model, self.head_dim
        return (d * self.qkv_dim + self.n_q_heads * dh * d + 3 * d * self.d_ffn)

    def to_dict(self):
        return asdict(self)


TINY_FP32 = ModelConfig("tiny-fp32", 2, 256, 4, 4, 64, 688, 2048, "f32")
MHA_8B = ModelConfig("mha-8b", 32, 4096, 32, 32, 128, 12288, 126464, "bf16")
GQA_7B = ModelConfig("gqa-7b", 28, 3584, 28, 4, 128, 18944, 152064, "bf16")

MODELS = {m.name: m for m in (TINY_FP32, MHA_8B, GQA_7B)}


@dataclass(frozen=True)
class Workload:
    name: str
    model: ModelConfig
    batch: int
    prompt_len: int           # fixed prompt length (0 when drawn per request)
    gen_len: int              # fixed generation length (0 when drawn per request)
    block: int
    cache_mode: str           # "none" | "prefix" | "dual"
    threshold: float
    # heterogeneous recipe (continuous-batching workload)
    prompt_range: Optional[Tuple[int, int]] = None
    gen_choices: Optional[Tuple[int, ...]] = None
    threshold_choices: Optional[Tuple[float, ...]] = None
    request_seed_base: int = 1000


C1 = Workload("tiny-fp32-nocache", TINY_FP32, 1, 64, 64, 32, "none", 0.9)
C2 = Workload("mha8b-b1-p256-g256-nocache", MHA_8B, 1, 256, 256, 32, "none", 0.9)
C3_DUAL = Workload("mha8b-b8-p1024-g256-dual", MHA_8B, 8, 1024, 256, 32, "dual", 0.9)
C3_PREFIX = Workload("mha8b-b8-p1024-g256-prefix", MHA_8B, 8, 1024, 256, 32, "prefix", 0.9)
C4 = Workload("mha8b-b32-hetero-dual", MHA_8B, 32, 0, 0, 32, "dual", 0.9,
              prompt_range=(128, 2048), gen_choices=(128, 256),
              threshold_choices=(0.7, 0.8, 0.9, 0.95))
C5 = Workload("gqa7b-b64-p512-g512-dual", GQA_7B, 64, 512, 512, 64, "dual", 0.9,
              threshold_choices=(0.5, 0.7, 0.9, 0.99))

WORKLOADS = {w.name: w for w in (C1, C2, C3_DUAL, C3_PREFIX, C4, C5)}
