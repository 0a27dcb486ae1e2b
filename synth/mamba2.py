"""Shapes, seeds and synthetic weights of the Mamba2 (state-space duality) workloads.

Only draws numbers; holds no arithmetic of the forward pass.  The paper's Mamba2 case
(appendix "Deployment Kernel Families", Table A.4) keeps the mixer sequence of input
projection, depthwise convolution, split into hidden / state parameters, recurrent scan, gated
RMSNorm and output projection; mamba2-130m has the Mamba2-130M layer shape of the paper's
Table 1 (the paper gives no hyper-parameters).

Tensors per layer (names of the standard Mamba2 mixer), fan-in scaled like synth.mamba:
  norm      [d]                      RMSNorm gain (ones)
  in_proj   [2 di + 2 G N + H, d]    workload dtype, N(0, 1/d); rows: z | x | B | C | dt
  conv_w    [di + 2 G N, d_conv]     fp32, N(0, 1/d_conv)   over the x | B | C channels
  conv_b    [di + 2 G N]             fp32, N(0, 0.02^2)
  dt_b      [H]                      fp32, softplus^-1 of dt log-uniform in [dt_min, dt_max]
  A_log     [H]                      fp32, log of U[1, 16] (A = -exp(A_log), one per head)
  D         [H]                      fp32, ones
  gnorm     [di]                     gated RMSNorm gain (ones), workload dtype
  out_proj  [d, di]                  workload dtype, N(0, 1/(2 L di))
and embed [V, d] (workload dtype, N(0, init_std^2); the LM head is tied to it) and
final_norm [d].  di = expand * d, H = di / head_dim heads, G groups of B and C.
Random tensor j draws from default_rng([s, 2, j]) in the order embed, then per layer
(in_proj, conv_w, conv_b, dt_b, A_log, out_proj).
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional, Tuple

import numpy as np

from .gen import round_to_bf16


@dataclasses.dataclass(frozen=True)
class Mamba2Config:
    name: str
    seed: int
    dtype: str
    n_layers: int
    d_model: int
    d_inner: int
    d_state: int
    head_dim: int
    n_groups: int
    d_conv: int
    vocab: int
    rms_eps: float = 1e-5
    batch: int = 1
    prompt_len: Optional[int] = None
    prompt_range: Optional[Tuple[int, int]] = None
    prompt_list: Optional[Tuple[int, ...]] = None
    n_decode: int = 1
    init_std: float = 0.02   # embedding
    dt_min: float = 1e-3
    dt_max: float = 1e-1
    family: str = "mamba2"

    @property
    def n_heads(self) -> int:
        return self.d_inner // self.head_dim

    @property
    def conv_dim(self) -> int:
        return self.d_inner + 2 * self.n_groups * self.d_state

    @property
    def in_dim(self) -> int:
        return self.d_inner + self.conv_dim + self.n_heads

    def linear_params_per_layer(self) -> int:
        return self.in_dim * self.d_model + self.d_model * self.d_inner

    def replace(self, **kw) -> "Mamba2Config":
        return dataclasses.replace(self, **kw)


MAMBA2_CONFIGS: Dict[str, Mamba2Config] = {
    # The Mamba2-130M layer shape: 24 layers, d 768, expand 2, state 128, head dim 64 (24
    # heads), one B/C group, conv 4; vocab 50304 (GPT-NeoX vocabulary padded to 32).
    "mamba2-130m": Mamba2Config(
        name="mamba2-130m", seed=41, dtype="bf16", n_layers=24, d_model=768, d_inner=1536,
        d_state=128, head_dim=64, n_groups=1, d_conv=4, vocab=50304, batch=1, prompt_len=1024,
        n_decode=128),
}

MAMBA2_TEST_CONFIGS: Dict[str, Mamba2Config] = {
    # ragged prompts incl. a 1-token one; two B/C groups
    "t-mamba2": Mamba2Config(
        name="t-mamba2", seed=51, dtype="bf16", n_layers=2, d_model=128, d_inner=256,
        d_state=64, head_dim=32, n_groups=2, d_conv=4, vocab=512, batch=3,
        prompt_list=(37, 1, 70), n_decode=5),
    "t-mamba2-f32": Mamba2Config(
        name="t-mamba2-f32", seed=52, dtype="f32", n_layers=2, d_model=128, d_inner=256,
        d_state=128, head_dim=64, n_groups=1, d_conv=4, vocab=512, batch=2,
        prompt_list=(19, 130), n_decode=4),
    # the smallest and largest state sizes the scan kernel takes (N = 32, N = 256)
    "t-mamba2-n32": Mamba2Config(
        name="t-mamba2-n32", seed=54, dtype="bf16", n_layers=2, d_model=128, d_inner=256,
        d_state=32, head_dim=64, n_groups=2, d_conv=4, vocab=512, batch=3,
        prompt_list=(50, 3, 200), n_decode=4),
    "t-mamba2-n256": Mamba2Config(
        name="t-mamba2-n256", seed=55, dtype="f32", n_layers=2, d_model=128, d_inner=256,
        d_state=256, head_dim=32, n_groups=1, d_conv=4, vocab=512, batch=2,
        prompt_list=(40, 300), n_decode=4),
    # long prompts (several scan chunks) and 6 sequences (decode above 4 rows)
    "t-mamba2-long": Mamba2Config(
        name="t-mamba2-long", seed=53, dtype="bf16", n_layers=2, d_model=256, d_inner=512,
        d_state=128, head_dim=64, n_groups=1, d_conv=4, vocab=1024, batch=6,
        prompt_range=(1, 700), n_decode=3),
}


def tensor_specs(cfg: Mamba2Config) -> List[Tuple[str, int, Tuple[int, ...], str]]:
    """[(name, j, shape, kind)] of the random tensors in stream order."""
    d, H = cfg.d_model, cfg.n_heads
    out = [("embed", 0, (cfg.vocab, d), "embed")]
    j = 1
    for layer in range(cfg.n_layers):
        for name, shape, kind in (("in_proj", (cfg.in_dim, d), "mat"),
                                  ("conv_w", (cfg.conv_dim, cfg.d_conv), "conv"),
                                  ("conv_b", (cfg.conv_dim,), "bias"), ("dt_b", (H,), "dtb"),
                                  ("A_log", (H,), "alog"), ("out_proj", (d, cfg.d_inner), "out")):
            out.append((f"layers.{layer}.{name}", j, shape, kind))
            j += 1
    return out


def _draw(cfg: Mamba2Config, j: int, shape, kind: str) -> np.ndarray:
    rng = np.random.default_rng([cfg.seed, 2, j])
    if kind == "dtb":
        u = rng.random(shape)
        dt = np.exp(u * (math.log(cfg.dt_max) - math.log(cfg.dt_min)) + math.log(cfg.dt_min))
        return (dt + np.log(-np.expm1(-dt))).astype(np.float32)
    if kind == "alog":
        return np.log(rng.uniform(1.0, 16.0, shape)).astype(np.float32)
    w = rng.standard_normal(shape, dtype=np.float32)
    std = {"embed": cfg.init_std, "mat": shape[-1] ** -0.5, "conv": cfg.d_conv ** -0.5,
           "bias": 0.02, "out": (2 * cfg.n_layers * shape[-1]) ** -0.5}[kind]
    w *= np.float32(std)
    if kind in ("embed", "mat", "out") and cfg.dtype == "bf16":
        w = round_to_bf16(w)
    return w


def weights(cfg: Mamba2Config) -> Dict[str, np.ndarray]:
    """Every tensor as an fp32 array (bf16-exact values for the bf16 matrices)."""
    out = {name: _draw(cfg, j, shape, kind) for name, j, shape, kind in tensor_specs(cfg)}
    for layer in range(cfg.n_layers):
        out[f"layers.{layer}.norm"] = np.ones(cfg.d_model, dtype=np.float32)
        out[f"layers.{layer}.gnorm"] = np.ones(cfg.d_inner, dtype=np.float32)
        out[f"layers.{layer}.D"] = np.ones(cfg.n_heads, dtype=np.float32)
    out["final_norm"] = np.ones(cfg.d_model, dtype=np.float32)
    return out


def get_mamba2_config(name: str) -> Mamba2Config:
    if name in MAMBA2_CONFIGS:
        return MAMBA2_CONFIGS[name]
    if name in MAMBA2_TEST_CONFIGS:
        return MAMBA2_TEST_CONFIGS[name]
    raise KeyError(name)
