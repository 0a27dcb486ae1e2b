"""fp64 CPU oracle of a Mamba2 (state-space duality) language model.

TEST INFRASTRUCTURE.  Only the tests, the smoke check and the benchmark's CPU-baseline leg
may import this module.  It shares no code with the HIP path; both sides use only the seeded
generator in ``synth``.

The paper's Mamba2 case (appendix "Deployment Kernel Families", Table A.4) names the mixer
sequence -- input projection, depthwise convolution, split into hidden and state parameters,
recurrent scan, gated RMSNorm, output projection -- and the phase contract of the Mamba family
(state ownership: the prefill leaves convolution and SSM state behind, a decode step updates
both once).  The paper prints no equations; the layer below is the plain definition of the
standard Mamba2 mixer in float64, its recurrence run one time step after another.

Readings (identical on the GPU side):
  * block: x += mixer(RMSNorm(x) * g); final RMSNorm; LM head tied to the embedding;
  * in_proj rows: z (di) | x (di) | B (G N) | C (G N) | dt (H); the causal depthwise conv and
    SiLU run over the x | B | C channels (zeros before a sequence's first token);
  * dt = softplus(dt + dt_bias) per head; A = -exp(A_log), one scalar per head; head h reads
    group h // (H / G) of B and C;
  * per head, state [head_dim, N]: h_t = exp(dt_t A) h_{t-1} + dt_t x_t B_t^T,
    y_t = h_t C_t + D x_t;
  * gated RMSNorm over the whole d_inner vector: RMSNorm(y * silu(z)) * gnorm.
"""
from __future__ import annotations

from typing import Dict, List, Sequence

import numpy as np

from .mamba import causal_depthwise_conv, softplus
from .transformer import argmax_lowest, rmsnorm, silu, split_prompts


def ssd_scan(x, dt, A, B, C, D, h0, group_of_head):
    """One time step after another, all heads at once.
        h_t[h] = exp(dt_t[h] A[h]) h_{t-1}[h] + dt_t[h] x_t[h] (outer) B_t[g(h)]
        y_t[h] = h_t[h] @ C_t[g(h)] + D[h] x_t[h]
    x [T, H, P]; dt [T, H]; A, D [H]; B, C [T, G, N]; h0 [H, P, N].  Returns (y, h_T)."""
    h = np.array(h0, dtype=np.float64)
    y = np.empty_like(x, dtype=np.float64)
    for t in range(x.shape[0]):
        Bt, Ct = B[t][group_of_head], C[t][group_of_head]          # [H, N]
        decay = np.exp(dt[t] * A)[:, None, None]
        h = decay * h + (dt[t][:, None] * x[t])[:, :, None] * Bt[:, None, :]
        y[t] = np.einsum("hpn,hn->hp", h, Ct) + D[:, None] * x[t]
    return y, h


class OracleMamba2:
    """Mamba2 language model with explicit per-sequence convolution and SSM state."""

    def __init__(self, cfg, weights: Dict[str, np.ndarray]):
        self.cfg = cfg
        self.w = {k: np.asarray(v, dtype=np.float64) for k, v in weights.items()}
        H, G = cfg.n_heads, cfg.n_groups
        self.group_of_head = np.arange(H) // (H // G)
        self.reset()

    def reset(self) -> None:
        self.conv: List[List[np.ndarray]] = []   # [seq][layer] -> [K-1, conv_dim]
        self.ssm: List[List[np.ndarray]] = []    # [seq][layer] -> [H, P, N]
        self.lengths: List[int] = []

    def _mixer(self, layer: int, hn: np.ndarray, seq: int) -> np.ndarray:
        cfg, w = self.cfg, self.w
        p = f"layers.{layer}."
        di, H, P, N, G = cfg.d_inner, cfg.n_heads, cfg.head_dim, cfg.d_state, cfg.n_groups
        proj = hn @ w[p + "in_proj"].T
        z = proj[:, :di]
        xbc = proj[:, di:di + cfg.conv_dim]
        dt_raw = proj[:, di + cfg.conv_dim:]
        past = self.conv[seq][layer]
        act = silu(causal_depthwise_conv(xbc, w[p + "conv_w"], w[p + "conv_b"], past))
        self.conv[seq][layer] = np.concatenate([past, xbc], axis=0)[-(cfg.d_conv - 1):]
        T = hn.shape[0]
        x = act[:, :di].reshape(T, H, P)
        Bm = act[:, di:di + G * N].reshape(T, G, N)
        Cm = act[:, di + G * N:].reshape(T, G, N)
        dt = softplus(dt_raw + w[p + "dt_b"])
        A = -np.exp(w[p + "A_log"])
        y, self.ssm[seq][layer] = ssd_scan(x, dt, A, Bm, Cm, w[p + "D"], self.ssm[seq][layer],
                                           self.group_of_head)
        g = rmsnorm(y.reshape(T, di) * silu(z), w[p + "gnorm"], cfg.rms_eps)
        return g @ w[p + "out_proj"].T

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
        self.conv.append([np.zeros((cfg.d_conv - 1, cfg.conv_dim)) for _ in range(cfg.n_layers)])
        self.ssm.append([np.zeros((cfg.n_heads, cfg.head_dim, cfg.d_state))
                         for _ in range(cfg.n_layers)])
        self.lengths.append(0)

    def prefill(self, prompts: Sequence[np.ndarray]) -> np.ndarray:
        """Prefill: every prompt from empty state; logits at each last position ([B, V])."""
        self.reset()
        out = []
        for b, toks in enumerate(prompts):
            self._new_seq()
            out.append(self._run(b, toks, False))
        return np.stack(out)

    def extend(self, chunks: Sequence[np.ndarray]) -> np.ndarray:
        """A further prompt chunk per sequence on the carried state ([B, V])."""
        assert len(chunks) == len(self.lengths), "a chunk per held sequence"
        return np.stack([self._run(b, np.asarray(c), False) for b, c in enumerate(chunks)])

    def decode(self, tokens: Sequence[int]) -> np.ndarray:
        """One token per sequence on the carried state; [B, V] logits."""
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


def teacher_forced_run_mamba2(model: OracleMamba2, lengths, packed, n_decode: int):
    """Prefill, then n_decode steps fed the oracle's own greedy tokens."""
    logits = [model.prefill(split_prompts(lengths, packed))]
    toks = [argmax_lowest(logits[0])]
    for _ in range(n_decode):
        logits.append(model.decode(toks[-1]))
        toks.append(argmax_lowest(logits[-1]))
    return np.stack(logits), np.stack(toks)
