"""Shapes, seeds and synthetic weights of the selective state-space (Mamba) workloads.

Like the decoder workloads, this module only draws numbers; it holds no arithmetic of the
forward pass.  The paper's Mamba-family cases (appendix "Deployment Kernel Families",
Table A.4) are a prefill recurrent scan and a single-token decode that updates the
convolution and SSM state of an existing cache; the paper gives no hyper-parameters, so the
shapes below define the workloads (mamba-130m has the Mamba-130M layer shape of the paper's
Table 1).

Tensors per layer (names of the standard Mamba mixer), fan-in scaled so that every stage of
the mixer works on O(1) values and the mixers, not the token embedding, make up the residual
stream (otherwise the tied LM head would mostly see the input token's own embedding and the
scan would barely move the logits):
  norm      [d]            RMSNorm gain (ones)
  in_proj   [2 di, d]      workload dtype, N(0, 1/d)
  conv_w    [di, d_conv]   fp32, N(0, 1/d_conv)        depthwise causal convolution taps
  conv_b    [di]           fp32, N(0, 0.02^2)
  x_proj    [R + 2 N, di]  workload dtype, N(0, 1/di)
  dt_w      [di, R]        fp32, N(0, 1/R)             dt projection
  dt_b      [di]           fp32, softplus^-1 of dt log-uniform in [dt_min, dt_max]
  A_log     [di, N]        fp32, log(1 .. N) in every row (A = -exp(A_log))
  D         [di]           fp32, ones
  out_proj  [d, di]        workload dtype, N(0, 1/(2 L di))
and embed [V, d] (workload dtype, N(0, init_std^2); the LM head is tied to it) and
final_norm [d] (ones).
Random tensor j draws from default_rng([s, 2, j]) in the order embed, then per layer
(in_proj, conv_w, conv_b, x_proj, dt_w, dt_b, out_proj); prompts use the streams of gen.py.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional, Tuple

import numpy as np

from .gen import round_to_bf16


@dataclasses.dataclass(frozen=True)
class MambaConfig:
    name: str
    seed: int
    dtype: str            # storage of the embedding and projection matrices ("bf16" or "f32")
    n_layers: int
    d_model: int
    d_inner: int
    d_state: int
    d_conv: int
    dt_rank: int
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
    family: str = "mamba"

    @property
    def xdbl_dim(self) -> int:
        return self.dt_rank + 2 * self.d_state

    def linear_params_per_layer(self) -> int:
        return (2 * self.d_inner * self.d_model + self.xdbl_dim * self.d_inner +
                self.d_model * self.d_inner)

    def replace(self, **kw) -> "MambaConfig":
        return dataclasses.replace(self, **kw)


MAMBA_CONFIGS: Dict[str, MambaConfig] = {
    # The Mamba-130M layer shape: 24 layers, d 768, expand 2, state 16, conv 4, dt rank 48;
    # vocab 50304 (the GPT-NeoX vocabulary padded to a multiple of 32 for the LM-head tiles).
    "mamba-130m": MambaConfig(
        name="mamba-130m", seed=21, dtype="bf16", n_layers=24, d_model=768, d_inner=1536,
        d_state=16, d_conv=4, dt_rank=48, vocab=50304, batch=1, prompt_len=1024, n_decode=128),
}

MAMBA_TEST_CONFIGS: Dict[str, MambaConfig] = {
    # ragged prompts incl. a 1-token one, fp32 and bf16
    "t-mamba": MambaConfig(
        name="t-mamba", seed=31, dtype="bf16", n_layers=2, d_model=128, d_inner=256,
        d_state=16, d_conv=4, dt_rank=8, vocab=512, batch=3, prompt_list=(37, 1, 70),
        n_decode=5),
    "t-mamba-f32": MambaConfig(
        name="t-mamba-f32", seed=32, dtype="f32", n_layers=2, d_model=128, d_inner=256,
        d_state=16, d_conv=4, dt_rank=8, vocab=512, batch=2, prompt_list=(19, 66),
        n_decode=4),
    # dt rank above 64 (x_proj width 112) and prompts long enough for scan chunks of several
    # 16-step stages
    "t-mamba-wide": MambaConfig(
        name="t-mamba-wide", seed=35, dtype="bf16", n_layers=2, d_model=256, d_inner=512,
        d_state=16, d_conv=4, dt_rank=80, vocab=1024, batch=2, prompt_list=(3000, 2500),
        n_decode=3),
    # dt rank 160 (Mamba-2.8B's): the largest rank the scan takes; R + 2N = 192 > 128, so
    # decode takes the unfused path whatever decode_fused says
    "t-mamba-r160": MambaConfig(
        name="t-mamba-r160", seed=36, dtype="f32", n_layers=2, d_model=256, d_inner=512,
        d_state=16, d_conv=4, dt_rank=160, vocab=1024, batch=2, prompt_list=(300, 17),
        n_decode=4),
    # a conv of width 2 (one row of conv state)
    "t-mamba-k2": MambaConfig(
        name="t-mamba-k2", seed=37, dtype="f32", n_layers=2, d_model=128, d_inner=256,
        d_state=16, d_conv=2, dt_rank=16, vocab=512, batch=3, prompt_list=(1, 40, 150),
        n_decode=4),
    # 20 ragged prompts: decode above the fused-step and skinny-GEMM row limits (split-K)
    "t-mamba-b20": MambaConfig(
        name="t-mamba-b20", seed=34, dtype="bf16", n_layers=2, d_model=256, d_inner=512,
        d_state=16, d_conv=4, dt_rank=16, vocab=1024, batch=20, prompt_range=(1, 48),
        n_decode=3),
}


def tensor_specs(cfg: MambaConfig) -> List[Tuple[str, int, Tuple[int, ...], str]]:
    """[(name, j, shape, kind)] of the random tensors in stream order."""
    di, d, R, N = cfg.d_inner, cfg.d_model, cfg.dt_rank, cfg.d_state
    out = [("embed", 0, (cfg.vocab, d), "embed")]
    j = 1
    for layer in range(cfg.n_layers):
        for name, shape, kind in (("in_proj", (2 * di, d), "mat"), ("conv_w", (di, cfg.d_conv), "conv"),
                                  ("conv_b", (di,), "bias"), ("x_proj", (cfg.xdbl_dim, di), "mat"),
                                  ("dt_w", (di, R), "dtw"), ("dt_b", (di,), "dtb"),
                                  ("out_proj", (d, di), "out")):
            out.append((f"layers.{layer}.{name}", j, shape, kind))
            j += 1
    return out


def _draw(cfg: MambaConfig, j: int, shape, kind: str) -> np.ndarray:
    rng = np.random.default_rng([cfg.seed, 2, j])
    if kind == "dtb":
        # dt log-uniform in [dt_min, dt_max]; bias = softplus^-1(dt) = dt + log(-expm1(-dt))
        u = rng.random(shape)
        dt = np.exp(u * (math.log(cfg.dt_max) - math.log(cfg.dt_min)) + math.log(cfg.dt_min))
        return (dt + np.log(-np.expm1(-dt))).astype(np.float32)
    w = rng.standard_normal(shape, dtype=np.float32)
    std = {"embed": cfg.init_std, "mat": shape[-1] ** -0.5, "conv": cfg.d_conv ** -0.5,
           "bias": 0.02, "dtw": cfg.dt_rank ** -0.5,
           "out": (2 * cfg.n_layers * shape[-1]) ** -0.5}[kind]
    w *= np.float32(std)
    if kind in ("embed", "mat", "out") and cfg.dtype == "bf16":
        w = round_to_bf16(w)
    return w


def weights(cfg: MambaConfig) -> Dict[str, np.ndarray]:
    """Every tensor as an fp32 array (bf16-exact values for the bf16 matrices)."""
    out = {name: _draw(cfg, j, shape, kind) for name, j, shape, kind in tensor_specs(cfg)}
    a_log = np.log(np.arange(1, cfg.d_state + 1, dtype=np.float32))
    for layer in range(cfg.n_layers):
        out[f"layers.{layer}.norm"] = np.ones(cfg.d_model, dtype=np.float32)
        out[f"layers.{layer}.A_log"] = np.tile(a_log, (cfg.d_inner, 1)).astype(np.float32)
        out[f"layers.{layer}.D"] = np.ones(cfg.d_inner, dtype=np.float32)
    out["final_norm"] = np.ones(cfg.d_model, dtype=np.float32)
    return out


def get_mamba_config(name: str) -> MambaConfig:
    if name in MAMBA_CONFIGS:
        return MAMBA_CONFIGS[name]
    if name in MAMBA_TEST_CONFIGS:
        return MAMBA_TEST_CONFIGS[name]
    raise KeyError(name)
