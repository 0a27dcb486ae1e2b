"""Shapes, seeds and synthetic weights of the RG-LRU (Griffin recurrent block) workloads.

Only draws numbers; holds no arithmetic of the forward pass.  The paper's recurrent case
(appendix "Deployment Kernel Families", Table A.4) is RecurrentGemma's RG-LRU; Table 1 quotes
RecurrentGemma-2B.  rglru-2b has that model's layer shapes (26 residual blocks, d 2560, RG-LRU
width 2560 in 10 blocks of 256, MLP 2 x 7680, conv 4, vocab 256000) with every temporal block
recurrent (RecurrentGemma puts a local-attention block in every third position).

Tensors per layer (names of the recurrent block), fan-in scaled so that every stage carries
O(1) values and the recurrence moves the logits:
  norm_t, norm_c  [d]                  RMSNorm offsets w (gain 1 + w)
  linear_y/_x     [W, d]               workload dtype, N(0, 1/d); biases fp32 N(0, 0.05^2)
  conv_w          [W, d_conv]          fp32, N(0, 1/d_conv); conv_b [W] fp32 N(0, 0.05^2)
  gate_a, gate_x  [H, bw, bw]          workload dtype, N(0, 1/bw) ([head][out][in]); biases
                                       [H, bw] fp32 N(0, 0.05^2)
  lambda          [W]                  fp32, softplus^-1(-log a0), a0 = sqrt(U[0.81, 0.998])
  linear_out      [d, W]               workload dtype, N(0, 1/(2 L W)); bias fp32 N(0, 0.05^2)
  mlp_gate/_up    [F, d]               workload dtype, N(0, 1/d); biases fp32 N(0, 0.05^2)
  mlp_down        [d, F]               workload dtype, N(0, 1/(2 L F)); bias fp32 N(0, 0.05^2)
and embed [V, d] (workload dtype, N(0, init_std^2); the LM head is tied to it) and
final_norm [d].  RMSNorm offsets are zero unless norm_std > 0; then they are multiples of
2^-7 in [-0.49, 0.49], so that 1 + w is exact in bf16 as well.
Random tensor j draws from default_rng([s, 3, j]) in the order embed, final_norm, then per
layer in the order of layer_specs.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional, Tuple

import numpy as np

from .gen import round_to_bf16


@dataclasses.dataclass(frozen=True)
class RGConfig:
    name: str
    seed: int
    dtype: str
    n_layers: int
    d_model: int
    lru_width: int
    n_heads: int
    mlp_width: int
    d_conv: int
    vocab: int
    rms_eps: float = 1e-6
    logit_cap: float = 30.0
    batch: int = 1
    prompt_len: Optional[int] = None
    prompt_range: Optional[Tuple[int, int]] = None
    prompt_list: Optional[Tuple[int, ...]] = None
    n_decode: int = 1
    init_std: float = 0.02   # embedding
    norm_std: float = 0.0
    family: str = "rglru"

    @property
    def block_width(self) -> int:
        return self.lru_width // self.n_heads

    @property
    def embed_scale(self) -> float:
        """sqrt(d_model) rounded to bf16 (RecurrentGemma keeps this constant in bf16)."""
        return float(round_to_bf16(np.array([math.sqrt(self.d_model)], np.float32))[0])

    def linear_params_per_layer(self) -> int:
        W, d, F = self.lru_width, self.d_model, self.mlp_width
        return 3 * W * d + 2 * W * self.block_width + 3 * F * d

    def replace(self, **kw) -> "RGConfig":
        return dataclasses.replace(self, **kw)


RG_CONFIGS: Dict[str, RGConfig] = {
    "rglru-2b": RGConfig(
        name="rglru-2b", seed=61, dtype="bf16", n_layers=26, d_model=2560, lru_width=2560,
        n_heads=10, mlp_width=7680, d_conv=4, vocab=256000, batch=1, prompt_len=1024,
        n_decode=128),
}

RG_TEST_CONFIGS: Dict[str, RGConfig] = {
    # ragged prompts incl. a 1-token one; blocks of 64 (gate groups narrower than 256 columns)
    "t-rg": RGConfig(
        name="t-rg", seed=71, dtype="bf16", n_layers=2, d_model=128, lru_width=128, n_heads=2,
        mlp_width=256, d_conv=4, vocab=512, batch=3, prompt_list=(37, 1, 70), n_decode=5,
        norm_std=0.1),
    "t-rg-f32": RGConfig(
        name="t-rg-f32", seed=72, dtype="f32", n_layers=2, d_model=128, lru_width=256, n_heads=4,
        mlp_width=384, d_conv=4, vocab=512, batch=2, prompt_list=(19, 130), n_decode=4,
        norm_std=0.1),
    # a conv of width 2 (one row of conv state) and blocks of 128
    "t-rg-k2": RGConfig(
        name="t-rg-k2", seed=74, dtype="f32", n_layers=2, d_model=128, lru_width=256, n_heads=2,
        mlp_width=256, d_conv=2, vocab=512, batch=3, prompt_list=(1, 40, 150), n_decode=4,
        norm_std=0.1),
    # long ragged prompts (several scan chunks) and 20 sequences (decode GEMMs above 16 rows)
    "t-rg-long": RGConfig(
        name="t-rg-long", seed=73, dtype="bf16", n_layers=2, d_model=256, lru_width=512,
        n_heads=2, mlp_width=512, d_conv=4, vocab=1024, batch=20, prompt_range=(1, 400),
        n_decode=3),
}


def layer_specs(cfg: RGConfig) -> List[Tuple[str, Tuple[int, ...], str]]:
    d, W, H, bw, F, K = (cfg.d_model, cfg.lru_width, cfg.n_heads, cfg.block_width,
                         cfg.mlp_width, cfg.d_conv)
    return [("norm_t", (d,), "norm"), ("linear_y", (W, d), "mat"), ("linear_y_b", (W,), "bias"),
            ("linear_x", (W, d), "mat"), ("linear_x_b", (W,), "bias"),
            ("conv_w", (W, K), "conv"), ("conv_b", (W,), "bias"),
            ("gate_a", (H, bw, bw), "mat"), ("gate_a_b", (H, bw), "bias"),
            ("gate_x", (H, bw, bw), "mat"), ("gate_x_b", (H, bw), "bias"),
            ("lambda", (W,), "lambda"),
            ("linear_out", (d, W), "out"), ("linear_out_b", (d,), "bias"),
            ("norm_c", (d,), "norm"), ("mlp_gate", (F, d), "mat"), ("mlp_gate_b", (F,), "bias"),
            ("mlp_up", (F, d), "mat"), ("mlp_up_b", (F,), "bias"),
            ("mlp_down", (d, F), "out"), ("mlp_down_b", (d,), "bias")]


def tensor_specs(cfg: RGConfig) -> List[Tuple[str, int, Tuple[int, ...], str]]:
    """[(name, j, shape, kind)] of every tensor in stream order."""
    out = [("embed", 0, (cfg.vocab, cfg.d_model), "embed"),
           ("final_norm", 1, (cfg.d_model,), "norm")]
    j = 2
    for layer in range(cfg.n_layers):
        for name, shape, kind in layer_specs(cfg):
            out.append((f"layers.{layer}.{name}", j, shape, kind))
            j += 1
    return out


def _draw(cfg: RGConfig, j: int, shape, kind: str) -> np.ndarray:
    if kind == "norm" and cfg.norm_std == 0.0:
        return np.zeros(shape, dtype=np.float32)
    rng = np.random.default_rng([cfg.seed, 3, j])
    if kind == "norm":
        w = np.round(rng.standard_normal(shape) * cfg.norm_std * 128.0) / 128.0
        return np.clip(w, -0.49, 0.49).astype(np.float32)
    if kind == "lambda":
        a0 = np.sqrt(rng.uniform(0.81, 0.998, shape))
        return np.log(np.expm1(-np.log(a0))).astype(np.float32)
    w = rng.standard_normal(shape, dtype=np.float32)
    fan_in = shape[-1]
    std = {"embed": cfg.init_std, "mat": fan_in ** -0.5, "conv": cfg.d_conv ** -0.5,
           "bias": 0.05, "out": (2 * cfg.n_layers * fan_in) ** -0.5}[kind]
    w *= np.float32(std)
    if kind in ("embed", "mat", "out") and cfg.dtype == "bf16":
        w = round_to_bf16(w)
    return w


def weights(cfg: RGConfig) -> Dict[str, np.ndarray]:
    """Every tensor as an fp32 array (bf16-exact values for the bf16 matrices)."""
    return {name: _draw(cfg, j, shape, kind) for name, j, shape, kind in tensor_specs(cfg)}


def get_rg_config(name: str) -> RGConfig:
    if name in RG_CONFIGS:
        return RG_CONFIGS[name]
    if name in RG_TEST_CONFIGS:
        return RG_TEST_CONFIGS[name]
    raise KeyError(name)
