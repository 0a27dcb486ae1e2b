"""fp64 CPU oracle of the phase-split decoder forward pass.

TEST INFRASTRUCTURE.  Only the tests, the smoke check and the benchmark's
CPU-baseline leg may import this module.  It shares no code with the HIP path;
the only thing both sides use is the seeded input generator in ``synth``.

What is computed.  The paper's method exists to speed up an autoregressive
inference script with two phases (Sec. 2.1 "Motivating Evidence"; Sec. 3.1
"Hotspot Discovery and Phase-Aware Extraction"): a *prefill* over the prompt,
where attention sees a block of queries (q_len > 1), and *decode* steps that
each run one query (q_len = 1) against a populated KV cache and append one
entry to it (appendix "Deployment Kernel Families", Table A.4).  Attention is
causal softmax attention with grouped-query heads, where the KV head of a query
head follows from the head grouping (same appendix).  The paper prints no layer
equations, so every layer below is the plain textbook definition of a pre-norm
LLaMA-style decoder, evaluated in float64 on the exact stored weight values.

Readings of points the paper leaves open (each identical on the GPU side):
  * RMSNorm: x / sqrt(mean(x^2) + eps) * g, eps inside the root, mean over d_model.
  * RoPE: rotate-half pairing (i, i + hd/2), frequency theta^(-2i/hd), angle = pos * freq,
    positions start at 0 in every sequence.
  * GQA: query head h reads KV head h // (H_q / H_kv) (contiguous groups).
  * Attention scale 1/sqrt(head_dim); no biases, no QK-norm, no logit cap, no embedding scale.
  * Pre-norm residual blocks; a final RMSNorm before an untied LM head.
  * Greedy choice: argmax with the lowest index winning ties.
"""
from __future__ import annotations

from typing import Dict, List, Sequence

import numpy as np


# --------------------------------------------------------------------------------------------
# Per-op definitions
# --------------------------------------------------------------------------------------------

def rmsnorm(x: np.ndarray, gain: np.ndarray, eps: float) -> np.ndarray:
    """Root-mean-square normalisation over the last axis, times the gain vector."""
    x = np.asarray(x, dtype=np.float64)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * np.asarray(gain, dtype=np.float64)


def rope_frequencies(head_dim: int, theta: float) -> np.ndarray:
    """freq_i = theta^(-2i/head_dim) for i = 0 .. head_dim/2 - 1."""
    i = np.arange(head_dim // 2, dtype=np.float64)
    return np.power(float(theta), -2.0 * i / head_dim)


def apply_rope(x: np.ndarray, positions: np.ndarray, theta: float) -> np.ndarray:
    """Rotate-half rotary embedding.

    x: [T, H, hd]; positions: [T].  Dimension i pairs with i + hd/2 and the pair is turned by
    the angle positions * freq_i:  (a, b) -> (a cos - b sin, b cos + a sin).
    """
    x = np.asarray(x, dtype=np.float64)
    hd = x.shape[-1]
    half = hd // 2
    ang = np.asarray(positions, dtype=np.float64)[:, None] * rope_frequencies(hd, theta)[None, :]
    cos = np.cos(ang)[:, None, :]
    sin = np.sin(ang)[:, None, :]
    a = x[..., :half]
    b = x[..., half:]
    return np.concatenate([a * cos - b * sin, b * cos + a * sin], axis=-1)


def softmax(s: np.ndarray) -> np.ndarray:
    """Row softmax; -inf entries get probability 0 (the row maximum is subtracted first)."""
    m = np.max(s, axis=-1, keepdims=True)
    e = np.exp(s - m)
    return e / np.sum(e, axis=-1, keepdims=True)


def causal_gqa_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray,
                         q_pos: np.ndarray, k_pos: np.ndarray) -> np.ndarray:
    """o_i = sum_j softmax_j(q_i . k_j / sqrt(hd)) v_j over keys with k_pos[j] <= q_pos[i].

    q: [Tq, Hq, hd]; k, v: [Tk, Hkv, hd].  Query head h reads KV head h // (Hq / Hkv).
    Returns [Tq, Hq, hd].
    """
    tq, hq, hd = q.shape
    hkv = k.shape[1]
    group = hq // hkv
    allowed = np.asarray(k_pos)[None, :] <= np.asarray(q_pos)[:, None]
    out = np.empty((tq, hq, hd), dtype=np.float64)
    for h in range(hq):
        g = h // group
        s = (q[:, h, :] @ k[:, g, :].T) / np.sqrt(hd)
        s = np.where(allowed, s, -np.inf)
        out[:, h, :] = softmax(s) @ v[:, g, :]
    return out


def silu(z: np.ndarray) -> np.ndarray:
    return z / (1.0 + np.exp(-z))


def swiglu(gate: np.ndarray, up: np.ndarray) -> np.ndarray:
    return silu(gate) * up


def argmax_lowest(logits: np.ndarray) -> np.ndarray:
    """Index of the maximum along the last axis; the lowest index wins ties.  NaN is an error."""
    logits = np.asarray(logits)
    if np.isnan(logits).any():
        raise ValueError("NaN logits")
    return np.argmax(logits, axis=-1)   # numpy returns the first occurrence of the maximum


def top2_margin(logits: np.ndarray) -> np.ndarray:
    """Largest minus second-largest logit, per row."""
    part = np.partition(np.asarray(logits, dtype=np.float64), -2, axis=-1)
    return part[..., -1] - part[..., -2]


# --------------------------------------------------------------------------------------------
# The model
# --------------------------------------------------------------------------------------------

class OracleModel:
    """Decoder forward pass with an explicit per-sequence KV cache.

    ``weights`` maps the tensor names of ``synth.gen`` to arrays; they are upcast to float64
    (exact for bf16 and fp32 storage).  Linear layers use the [out, in] layout: y = x @ W^T.
    """

    def __init__(self, cfg, weights: Dict[str, np.ndarray], keep_f64: bool = True):
        self.cfg = cfg
        self.keep_f64 = keep_f64
        self.w = {k: (np.asarray(v, dtype=np.float64) if keep_f64 else np.asarray(v))
                  for k, v in weights.items()}
        self.reset()

    # -- state ---------------------------------------------------------------------------------
    def reset(self) -> None:
        """Empty every sequence's cache (the batch is defined by the next prefill)."""
        self.k_cache: List[List[np.ndarray]] = []   # [seq][layer] -> [S, Hkv, hd]
        self.v_cache: List[List[np.ndarray]] = []
        self.lengths: List[int] = []

    def _W(self, name: str) -> np.ndarray:
        w = self.w[name]
        return w if w.dtype == np.float64 else w.astype(np.float64)

    # -- one decoder layer over a block of tokens of one sequence -------------------------------
    def _layer(self, layer: int, x: np.ndarray, positions: np.ndarray, seq: int) -> np.ndarray:
        cfg = self.cfg
        p = f"layers.{layer}."
        t = x.shape[0]
        h = rmsnorm(x, self.w[p + "attn_norm"], cfg.rms_eps)
        q = (h @ self._W(p + "wq").T).reshape(t, cfg.n_heads, cfg.head_dim)
        k = (h @ self._W(p + "wk").T).reshape(t, cfg.n_kv_heads, cfg.head_dim)
        v = (h @ self._W(p + "wv").T).reshape(t, cfg.n_kv_heads, cfg.head_dim)
        q = apply_rope(q, positions, cfg.rope_theta)
        k = apply_rope(k, positions, cfg.rope_theta)
        # KV-cache append: the new keys/values land after the ones already cached.
        kc = np.concatenate([self.k_cache[seq][layer], k], axis=0)
        vc = np.concatenate([self.v_cache[seq][layer], v], axis=0)
        self.k_cache[seq][layer] = kc
        self.v_cache[seq][layer] = vc
        k_pos = np.arange(kc.shape[0])
        o = causal_gqa_attention(q, kc, vc, positions, k_pos).reshape(t, cfg.q_dim)
        x = x + o @ self._W(p + "wo").T
        h = rmsnorm(x, self.w[p + "mlp_norm"], cfg.rms_eps)
        a = swiglu(h @ self._W(p + "w_gate").T, h @ self._W(p + "w_up").T)
        return x + a @ self._W(p + "w_down").T

    def _run(self, seq: int, tokens: np.ndarray, start: int, all_logits: bool) -> np.ndarray:
        cfg = self.cfg
        tokens = np.asarray(tokens, dtype=np.int64)
        positions = start + np.arange(tokens.shape[0])
        x = self._W("embed")[tokens] if self.keep_f64 else self.w["embed"][tokens].astype(np.float64)
        for layer in range(cfg.n_layers):
            x = self._layer(layer, x, positions, seq)
        self.lengths[seq] = start + tokens.shape[0]
        rows = x if all_logits else x[-1:]
        hf = rmsnorm(rows, self.w["final_norm"], cfg.rms_eps)
        logits = hf @ self._W("lm_head").T
        return logits if all_logits else logits[0]

    # -- the two phases -------------------------------------------------------------------------
    def prefill(self, prompts: Sequence[np.ndarray], all_logits: bool = False):
        """Prefill phase: run every prompt over an empty cache.

        Returns the logits at each sequence's last prompt position ([B, V]), or, with
        all_logits, a list of [L_b, V] arrays.
        """
        self.reset()
        nl = self.cfg.n_layers
        empty = np.zeros((0, self.cfg.n_kv_heads, self.cfg.head_dim))
        out = []
        for b, toks in enumerate(prompts):
            self.k_cache.append([empty] * nl)
            self.v_cache.append([empty] * nl)
            self.lengths.append(0)
            out.append(self._run(b, toks, 0, all_logits))
        return out if all_logits else np.stack(out)

    def extend(self, chunks: Sequence[np.ndarray]) -> np.ndarray:
        """Prefill phase on a populated cache (a further prompt chunk of every sequence):
        chunk b enters at positions len[b] .. len[b] + len(chunk) - 1, its keys and values are
        appended after the cached ones, and each query attends to every cached position up
        to its own.  Returns the logits at each chunk's last position ([B, V])."""
        assert len(chunks) == len(self.lengths), "a chunk per sequence of the prefill batch"
        return np.stack([self._run(b, np.asarray(c), self.lengths[b], False)
                         for b, c in enumerate(chunks)])

    def decode(self, tokens: Sequence[int]) -> np.ndarray:
        """Decode phase: one token per sequence at position len[b]; returns [B, V] logits."""
        assert len(tokens) == len(self.lengths), "decode batch must match the prefill batch"
        return np.stack([self._run(b, np.array([tokens[b]]), self.lengths[b], False)
                         for b in range(len(self.lengths))])

    def forward_full(self, tokens: np.ndarray) -> np.ndarray:
        """Fresh causal forward over one whole sequence; logits at every position ([L, V])."""
        saved = (self.k_cache, self.v_cache, self.lengths)
        try:
            self.reset()
            nl = self.cfg.n_layers
            empty = np.zeros((0, self.cfg.n_kv_heads, self.cfg.head_dim))
            self.k_cache.append([empty] * nl)
            self.v_cache.append([empty] * nl)
            self.lengths.append(0)
            return self._run(0, tokens, 0, True)
        finally:
            self.k_cache, self.v_cache, self.lengths = saved


def split_prompts(lengths: Sequence[int], packed: np.ndarray) -> List[np.ndarray]:
    out, o = [], 0
    for n in lengths:
        out.append(np.asarray(packed[o:o + n]))
        o += n
    return out


def teacher_forced_run(model: OracleModel, lengths: Sequence[int], packed: np.ndarray,
                       n_decode: int):
    """Prefill, then n_decode steps each fed the oracle's own greedy token.

    Returns (logits [n_decode + 1, B, V], tokens [n_decode + 1, B]): row 0 comes from the
    prefill; row k (k >= 1) from decode step k, whose input is tokens[k - 1].
    """
    logits = [model.prefill(split_prompts(lengths, packed))]
    toks = [argmax_lowest(logits[0])]
    for _ in range(n_decode):
        logits.append(model.decode(toks[-1]))
        toks.append(argmax_lowest(logits[-1]))
    return np.stack(logits), np.stack(toks)
