"""Seeded synthetic inputs: prompt lengths, prompt tokens and weights.

Shared by the oracle and by the HIP path's tests and benchmark.  Nothing in
here computes any part of the forward pass: it only draws numbers and stores
them in the workload's storage type.

Streams (s = workload seed):
  ragged lengths   default_rng([s, 0]).integers(lo, hi, endpoint=True)
  prompt tokens    default_rng([s, 1]).integers(0, vocab, size=T), packed in sequence order
  weight tensor j  default_rng([s, 2, j]).standard_normal(shape, float32) * std_j, then
                   round-to-nearest-even to bf16 for bf16 workloads
  gain vector j    1.0, or 1 + 0.1 * default_rng([s, 3, j]).standard_normal(d) when asked for
Tensor order j: embedding, then per layer (W_q, W_k, W_v, W_o, W_gate, W_up, W_down), then LM head.
"""
from __future__ import annotations

import hashlib
from typing import Dict, Iterator, List, Tuple

import numpy as np

from .configs import ModelConfig

LAYER_TENSORS = ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down")


def prompt_lengths(cfg: ModelConfig) -> List[int]:
    if cfg.prompt_list is not None:
        assert len(cfg.prompt_list) == cfg.batch
        return [int(x) for x in cfg.prompt_list]
    if cfg.prompt_range is not None:
        lo, hi = cfg.prompt_range
        rng = np.random.default_rng([cfg.seed, 0])
        return [int(x) for x in rng.integers(lo, hi, size=cfg.batch, endpoint=True)]
    return [int(cfg.prompt_len)] * cfg.batch


def prompt_tokens(cfg: ModelConfig) -> Tuple[List[int], np.ndarray]:
    """(lengths, packed int32 token ids of all sequences in order)."""
    lens = prompt_lengths(cfg)
    rng = np.random.default_rng([cfg.seed, 1])
    toks = rng.integers(0, cfg.vocab, size=sum(lens)).astype(np.int32)
    return lens, toks


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """fp32 -> nearest bf16 (ties to even), returned as fp32 holding the bf16 value exactly."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    b = x.view(np.uint32)
    rounded = (b + np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))) & np.uint32(0xFFFF0000)
    return rounded.view(np.float32)


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """Upper 16 bits of fp32 values that are exactly bf16 (as stored on the device)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    return (x.view(np.uint32) >> np.uint32(16)).astype(np.uint16)


def tensor_shapes(cfg: ModelConfig) -> List[Tuple[str, int, Tuple[int, int], float]]:
    """[(name, j, shape, std)] in stream order."""
    d, f = cfg.d_model, cfg.ffn_dim
    out = [("embed", 0, (cfg.vocab, d), cfg.init_std)]
    j = 1
    for layer in range(cfg.n_layers):
        shapes = {
            "wq": (cfg.q_dim, d), "wk": (cfg.kv_dim, d), "wv": (cfg.kv_dim, d), "wo": (d, cfg.q_dim),
            "w_gate": (f, d), "w_up": (f, d), "w_down": (d, f),
        }
        for name in LAYER_TENSORS:
            std = cfg.init_std * (cfg.out_proj_scale if name in ("wo", "w_down") else 1.0)
            out.append((f"layers.{layer}.{name}", j, shapes[name], std))
            j += 1
    out.append(("lm_head", j, (cfg.vocab, d), cfg.init_std))
    return out


def draw_tensor(cfg: ModelConfig, j: int, shape: Tuple[int, int], std: float) -> np.ndarray:
    rng = np.random.default_rng([cfg.seed, 2, j])
    w = rng.standard_normal(shape, dtype=np.float32)
    w *= np.float32(std)
    if cfg.dtype == "bf16":
        w = round_to_bf16(w)
    return w


def iter_weights(cfg: ModelConfig) -> Iterator[Tuple[str, np.ndarray]]:
    """Yield (name, fp32 array) one tensor at a time (keeps peak memory at one tensor)."""
    for name, j, shape, std in tensor_shapes(cfg):
        yield name, draw_tensor(cfg, j, shape, std)


def iter_weights_parallel(cfg: ModelConfig, workers: int = 8) -> Iterator[Tuple[str, np.ndarray]]:
    """Same tensors and order as iter_weights, drawn on `workers` threads (numpy's generator
    releases the GIL), with at most 2 * workers tensors in flight."""
    import collections
    from concurrent.futures import ThreadPoolExecutor
    specs = tensor_shapes(cfg)
    with ThreadPoolExecutor(max_workers=workers) as ex:
        pending = collections.deque()
        for name, j, shape, std in specs:
            pending.append((name, ex.submit(draw_tensor, cfg, j, shape, std)))
            if len(pending) >= 2 * workers:
                n, f = pending.popleft()
                yield n, f.result()
        while pending:
            n, f = pending.popleft()
            yield n, f.result()


def gains(cfg: ModelConfig, random_gains: bool = False) -> Dict[str, np.ndarray]:
    """RMSNorm gain vectors: attn_norm/mlp_norm per layer and final_norm."""
    names = []
    for layer in range(cfg.n_layers):
        names += [f"layers.{layer}.attn_norm", f"layers.{layer}.mlp_norm"]
    names.append("final_norm")
    out = {}
    for j, name in enumerate(names):
        if random_gains:
            g = 1.0 + 0.1 * np.random.default_rng([cfg.seed, 3, j]).standard_normal(
                cfg.d_model, dtype=np.float32)
            if cfg.dtype == "bf16":
                g = round_to_bf16(g)
            out[name] = g.astype(np.float32)
        else:
            out[name] = np.ones(cfg.d_model, dtype=np.float32)
    return out


def weights(cfg: ModelConfig, random_gains: bool = False) -> Dict[str, np.ndarray]:
    """All tensors as fp32 arrays (bf16-exact values for bf16 workloads)."""
    big = cfg.n_layers * cfg.linear_params_per_layer() > 50_000_000
    out = dict(iter_weights_parallel(cfg) if big else iter_weights(cfg))
    out.update(gains(cfg, random_gains))
    return out


def sha256(arr: np.ndarray) -> str:
    return hashlib.sha256(np.ascontiguousarray(arr).tobytes()).hexdigest()
