"""fp64 CPU oracle of a selective state-space (Mamba) language model.

TEST INFRASTRUCTURE.  Only the tests, the smoke check and the benchmark's CPU-baseline leg
may import this module.  It shares no code with the HIP path; both sides use only the seeded
generator in ``synth``.

The paper's Mamba-family cases (appendix "Deployment Kernel Families", Table A.4) name the
mixer's chain -- input projection, depthwise causal convolution, split into the SSM
parameters, recurrent scan, gating, output projection -- and the phase contract: the prefill
runs the recurrent scan over the prompt and leaves convolution and SSM state behind; a decode
step takes one token per sequence, updates both states once and emits the next token.  The
paper prints no equations; the layer below is the plain definition of the standard selective
SSM (Mamba) mixer, evaluated in float64 on the exact stored weights, with the recurrence run
one time step after another.

Readings (identical on the GPU side):
  * block: x += mixer(RMSNorm(x) * g); final RMSNorm; LM head tied to the embedding;
  * conv: causal depthwise, u_t = silu(sum_k w[k] x_{t - (K-1) + k} + b), zeros before a
    sequence's first token;
  * dt = softplus(x_dbl[:, :R] W_dt^T + b_dt); A = -exp(A_log);
  * h_t = exp(dt_t A) * h_{t-1} + dt_t B_t u_t;  y_t = C_t . h_t + D u_t;  y *= silu(z).
"""
from __future__ import annotations

from typing import Dict, List, Sequence

import numpy as np

from .transformer import argmax_lowest, rmsnorm, silu


def softplus(x: np.ndarray) -> np.ndarray:
    """log(1 + e^x), computed without overflow."""
    x = np.asarray(x, dtype=np.float64)
    return np.logaddexp(0.0, x)


def causal_depthwise_conv(x: np.ndarray, w: np.ndarray, b: np.ndarray,
                          past: np.ndarray) -> np.ndarray:
    """out[t, c] = sum_k w[c, k] * xx[t + k, c] + b[c], where xx is the K-1 inputs before the
    block (past [K-1, C], oldest first) followed by the block x [T, C]."""
    K = w.shape[1]
    xx = np.concatenate([past, x], axis=0)
    T = x.shape[0]
    out = np.tile(np.asarray(b, dtype=np.float64), (T, 1))
    for k in range(K):
        out += xx[k:k + T] * w[:, k][None, :]
    return out


def selective_scan(u, dt, A, B, C, D, h0):
    """One time step after another:
        h_t = exp(dt_t[:, None] * A) * h_{t-1} + (dt_t * u_t)[:, None] * B_t[None, :]
        y_t = h_t @ C_t + D * u_t
    u, dt [T, C]; A [C, N]; B, C [T, N]; D [C]; h0 [C, N].  Returns (y [T, C], h_T)."""
    h = np.array(h0, dtype=np.float64)
    T = u.shape[0]
    y = np.empty_like(u, dtype=np.float64)
    for t in range(T):
        h = np.exp(dt[t][:, None] * A) * h + (dt[t] * u[t])[:, None] * B[t][None, :]
        y[t] = h @ C[t] + D * u[t]
    return y, h


class OracleMamba:
    """Mamba language model with explicit per-sequence convolution and SSM state."""

    def __init__(self, cfg, weights: Dict[str, np.ndarray]):
        self.cfg = cfg
        self.w = {k: np.asarray(v, dtype=np.float64) for k, v in weights.items()}
        self.reset()

    def reset(self) -> None:
        self.conv: List[List[np.ndarray]] = []   # [seq][layer] -> [K-1, di] last inputs
        self.ssm: List[List[np.ndarray]] = []    # [seq][layer] -> [di, N]
        self.lengths: List[int] = []

    def _mixer(self, layer: int, h: np.ndarray, seq: int) -> np.ndarray:
        cfg, w = self.cfg, self.w
        p = f"layers.{layer}."
        di, R, N = cfg.d_inner, cfg.dt_rank, cfg.d_state
        xz = h @ w[p + "in_proj"].T
        x, z = xz[:, :di], xz[:, di:]
        past = self.conv[seq][layer]
        u = silu(causal_depthwise_conv(x, w[p + "conv_w"], w[p + "conv_b"], past))
        self.conv[seq][layer] = np.concatenate([past, x], axis=0)[-(cfg.d_conv - 1):]
        xdbl = u @ w[p + "x_proj"].T
        dt = softplus(xdbl[:, :R] @ w[p + "dt_w"].T + w[p + "dt_b"])
        Bm, Cm = xdbl[:, R:R + N], xdbl[:, R + N:R + 2 * N]
        A = -np.exp(w[p + "A_log"])
        y, self.ssm[seq][layer] = selective_scan(u, dt, A, Bm, Cm, w[p + "D"],
                                                 self.ssm[seq][layer])
        return (y * silu(z)) @ w[p + "out_proj"].T

    def _run(self, seq: int, tokens: np.ndarray, all_logits: bool) -> np.ndarray:
        cfg, w = self.cfg, self.w
        x = w["embed"][np.asarray(tokens, dtype=np.int64)]
        for layer in range(cfg.n_layers):
            x = x + self._mixer(layer, rmsnorm(x, w[f"layers.{layer}.norm"], cfg.rms_eps), seq)
        self.lengths[seq] += len(tokens)
        rows = x if all_logits else x[-1:]
        logits = rmsnorm(rows, w["final_norm"], cfg.rms_eps) @ w["embed"].T
        return logits if all_logits else logits[0]

    def _new_seq(self) -> None:
        cfg = self.cfg
        self.conv.append([np.zeros((cfg.d_conv - 1, cfg.d_inner)) for _ in range(cfg.n_layers)])
        self.ssm.append([np.zeros((cfg.d_inner, cfg.d_state)) for _ in range(cfg.n_layers)])
        self.lengths.append(0)

    def prefill(self, prompts: Sequence[np.ndarray], all_logits: bool = False):
        """Prefill: every prompt from empty state; logits at each last position ([B, V])."""
        self.reset()
        out = []
        for b, toks in enumerate(prompts):
            self._new_seq()
            out.append(self._run(b, toks, all_logits))
        return out if all_logits else np.stack(out)

    def extend(self, chunks: Sequence[np.ndarray]) -> np.ndarray:
        """Prefill of a further prompt chunk per sequence on the carried state (the scan and
        the convolution continue from it); logits at each chunk's last token ([B, V])."""
        assert len(chunks) == len(self.lengths), "a chunk per held sequence"
        return np.stack([self._run(b, np.asarray(c), False) for b, c in enumerate(chunks)])

    def decode(self, tokens: Sequence[int]) -> np.ndarray:
        """Decode: one token per sequence on the carried state; [B, V] logits."""
        assert len(tokens) == len(self.lengths)
        return np.stack([self._run(b, np.array([tokens[b]]), False)
                         for b in range(len(self.lengths))])

    def forward_full(self, tokens: np.ndarray) -> np.ndarray:
        """Fresh forward over one whole sequence; logits at every position ([L, V])."""
        saved = (self.conv, self.ssm, self.lengths)
        try:
            self.reset()
            self._new_seq()
            return self._run(0, tokens, True)
        finally:
            self.conv, self.ssm, self.lengths = saved


def teacher_forced_run_mamba(model: OracleMamba, lengths, packed, n_decode: int):
    """Prefill, then n_decode steps fed the oracle's own greedy tokens (as for the decoder)."""
    from .transformer import split_prompts
    logits = [model.prefill(split_prompts(lengths, packed))]
    toks = [argmax_lowest(logits[0])]
    for _ in range(n_decode):
        logits.append(model.decode(toks[-1]))
        toks.append(argmax_lowest(logits[-1]))
    return np.stack(logits), np.stack(toks)
