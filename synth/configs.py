"""Model shapes and workload recipes for the phase-split decoder forward pass.

This module only describes shapes and seeds; it holds no arithmetic of the
forward pass.  The model family is a pre-norm LLaMA-style decoder (RMSNorm,
rotate-half RoPE, grouped-query attention, SwiGLU MLP, untied LM head).  The
paper fixes the phase split -- a prefill over the prompt (q_len > 1) followed
by single-token decode steps against a populated KV cache (Sec. 2.1 and the
appendix "Deployment Kernel Families") -- but no model hyper-parameters, so
the shapes below define the workloads.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, Optional, Tuple


@dataclasses.dataclass(frozen=True)
class ModelConfig:
    name: str
    seed: int                 # workload number s; every random stream is keyed by it
    dtype: str                # "f32" or "bf16": storage type of weights, KV cache and GEMM inputs
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    ffn_dim: int
    vocab: int
    rms_eps: float = 1e-5
    rope_theta: float = 10000.0
    out_proj_scale: float = 1.0   # extra std factor of W_o and W_down
    batch: int = 1
    prompt_len: Optional[int] = None            # fixed prompt length, or
    prompt_range: Optional[Tuple[int, int]] = None  # ragged lengths uniform in [lo, hi]
    prompt_list: Optional[Tuple[int, ...]] = None   # explicit lengths (small test workloads)
    n_decode: int = 1
    init_std: float = 0.02

    @property
    def group(self) -> int:
        return self.n_heads // self.n_kv_heads

    @property
    def q_dim(self) -> int:
        return self.n_heads * self.head_dim

    @property
    def kv_dim(self) -> int:
        return self.n_kv_heads * self.head_dim

    def linear_params_per_layer(self) -> int:
        d = self.d_model
        return d * (self.q_dim + 2 * self.kv_dim) + self.q_dim * d + 3 * d * self.ffn_dim

    def replace(self, **kw) -> "ModelConfig":
        return dataclasses.replace(self, **kw)


# The five workloads.  Names say what each one is.
CONFIGS: Dict[str, ModelConfig] = {
    # 2-layer fp32 decoder; the oracle finishes it in well under a second.
    "tiny-f32": ModelConfig(
        name="tiny-f32", seed=1, dtype="f32", n_layers=2, d_model=256, n_heads=4, n_kv_heads=4,
        head_dim=64, ffn_dim=1024, vocab=1024, batch=1, prompt_len=32, n_decode=16),
    # 125M-class MHA decoder; output projections scaled by 1/sqrt(2 * layers).
    "125m": ModelConfig(
        name="125m", seed=2, dtype="bf16", n_layers=12, d_model=768, n_heads=12, n_kv_heads=12,
        head_dim=64, ffn_dim=2048, vocab=32000, out_proj_scale=1.0 / math.sqrt(24.0),
        batch=1, prompt_len=512, n_decode=128),
    # 1.1B-class GQA decoder (32 query heads over 4 KV heads), batch 8.
    "1b-gqa": ModelConfig(
        name="1b-gqa", seed=3, dtype="bf16", n_layers=22, d_model=2048, n_heads=32, n_kv_heads=4,
        head_dim=64, ffn_dim=5632, vocab=32000, batch=8, prompt_len=1024, n_decode=256),
    # 7B-class MHA decoder, head_dim 128; output projections scaled by 1/sqrt(64).
    "7b-mha": ModelConfig(
        name="7b-mha", seed=4, dtype="bf16", n_layers=32, d_model=4096, n_heads=32, n_kv_heads=32,
        head_dim=128, ffn_dim=11008, vocab=32000, out_proj_scale=1.0 / 8.0,
        batch=1, prompt_len=2048, n_decode=256),
    # 8B-class GQA decoder (32 over 8), 128256 vocab, theta 5e5, 32 ragged prompts in [1024, 4096].
    "8b-gqa": ModelConfig(
        name="8b-gqa", seed=5, dtype="bf16", n_layers=32, d_model=4096, n_heads=32, n_kv_heads=8,
        head_dim=128, ffn_dim=14336, vocab=128256, rope_theta=500000.0,
        batch=32, prompt_range=(1024, 4096), n_decode=128),
}

# Small workloads for parity tests: several tiles per GEMM, ragged tails, GQA and head_dim 128,
# yet small enough for the fp64 oracle to finish in seconds.  Seeds 11.. keep them apart from the
# five workloads above.
TEST_CONFIGS: Dict[str, ModelConfig] = {
    "t-gqa-hd64": ModelConfig(
        name="t-gqa-hd64", seed=11, dtype="bf16", n_layers=2, d_model=512, n_heads=8, n_kv_heads=2,
        head_dim=64, ffn_dim=1408, vocab=4096, batch=4, prompt_list=(77, 1, 130, 64), n_decode=6),
    "t-gqa-hd128": ModelConfig(
        name="t-gqa-hd128", seed=12, dtype="bf16", n_layers=2, d_model=512, n_heads=4, n_kv_heads=2,
        head_dim=128, ffn_dim=768, vocab=2048, rope_theta=500000.0,
        batch=3, prompt_list=(200, 33, 129), n_decode=5),
    "t-f32-ragged": ModelConfig(
        name="t-f32-ragged", seed=13, dtype="f32", n_layers=2, d_model=256, n_heads=4, n_kv_heads=2,
        head_dim=64, ffn_dim=512, vocab=1024, batch=3, prompt_list=(19, 65, 2), n_decode=4),
    "t-b32-hd128": ModelConfig(
        name="t-b32-hd128", seed=14, dtype="bf16", n_layers=1, d_model=256, n_heads=2, n_kv_heads=1,
        head_dim=128, ffn_dim=512, vocab=1024, batch=32, prompt_range=(1, 40), n_decode=3),
}


def get_config(name: str) -> ModelConfig:
    if name in CONFIGS:
        return CONFIGS[name]
    if name in TEST_CONFIGS:
        return TEST_CONFIGS[name]
    raise KeyError(f"unknown config {name!r}; known: {sorted(CONFIGS) + sorted(TEST_CONFIGS)}")
