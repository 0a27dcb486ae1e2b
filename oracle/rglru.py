"""fp64 CPU oracle of a language model built from Griffin recurrent blocks (the RG-LRU layer of
RecurrentGemma).

TEST INFRASTRUCTURE.  Only the tests, the smoke check and the benchmark's CPU-baseline leg
may import this module.  It shares no code with the HIP path; both sides use only the seeded
generator in ``synth``.

The paper's recurrent case (appendix "Deployment Kernel Families", Table A.4, and the
paragraph on RecurrentGemma after it) names the RG-LRU's parts -- sigmoid gates, a recurrent
gate derived through a softplus, reset handling, input normalisation and the recurrent scan
whose final state is written once -- and the state-ownership contract of the recurrent
families: the prefill leaves the convolution and recurrent state behind and a decode step
updates both exactly once.  The paper prints no equations; the layer below is the plain
definition of the RG-LRU and of the recurrent block around it, in float64, the recurrence run
one time step after another.

Readings (identical on the GPU side):
  * embedding rows scaled by embed_scale (sqrt(d_model) held in bf16, as RecurrentGemma does);
  * RMSNorm gains are 1 + w;
  * residual block: x += recurrent(norm_t(x)); x += mlp(norm_c(x)); final norm; LM head tied
    to the embedding; logits soft-capped, cap * tanh(logits / cap); greedy argmax;
  * recurrent block: y = gelu_tanh(W_y h + b_y); x = conv(W_x h + b_x) (causal depthwise,
    bias, no activation, zeros before a sequence's first token); out = W_o (rglru(x) * y) + b_o;
  * RG-LRU on channel c of head k (block-diagonal gates, W_a[k], W_i[k] of shape
    [block, block] acting as W x on the head's block of x):
        r_t = sigmoid(W_a x_t + b_a),  i_t = sigmoid(W_i x_t + b_i),
        log a_t = -c * r_t * softplus(lambda),  c = 8,
        h_t = a_t h_{t-1} + sqrt(1 - a_t^2) (i_t x_t)      (later tokens)
        h_t = i_t x_t                                       (a sequence's first token: reset)
    and the block's output is h_t;
  * mlp: W_d (gelu_tanh(W_g h + b_g) * (W_u h + b_u)) + b_d.
"""
from __future__ import annotations

from typing import Dict, List, Sequence

import numpy as np

from .mamba import causal_depthwise_conv, softplus
from .transformer import argmax_lowest, split_prompts

RG_GATE_C = 8.0


def gelu_tanh(x: np.ndarray) -> np.ndarray:
    """The tanh approximation of GELU: x/2 (1 + tanh(sqrt(2/pi) (x + 0.044715 x^3)))."""
    x = np.asarray(x, dtype=np.float64)
    return 0.5 * x * (1.0 + np.tanh(np.sqrt(2.0 / np.pi) * (x + 0.044715 * x ** 3)))


def sigmoid(x: np.ndarray) -> np.ndarray:
    x = np.asarray(x, dtype=np.float64)
    return np.exp(-np.logaddexp(0.0, -x))


def rms_norm_offset(x: np.ndarray, w: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * (1 + w)."""
    x = np.asarray(x, dtype=np.float64)
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * (1.0 + w)


def soft_cap(logits: np.ndarray, cap: float) -> np.ndarray:
    return cap * np.tanh(logits / cap)


def block_diag_apply(x: np.ndarray, W: np.ndarray, b: np.ndarray) -> np.ndarray:
    """Head k's block of x times W[k]^T plus b[k]: x [T, H*bw], W [H, bw_out, bw_in],
    b [H, bw] -> [T, H*bw]."""
    H, bw, _ = W.shape
    xs = x.reshape(x.shape[0], H, bw)
    return (np.einsum("thi,hoi->tho", xs, W) + b[None]).reshape(x.shape[0], H * bw)


def rg_lru(x, Wa, ba, Wi, bi, lam, h0, reset_first: bool):
    """The RG-LRU over T steps of one sequence: x [T, W]; h0 [W].  reset_first: the block's
    first row is the sequence's first token.  Returns (h for every step [T, W], h_T)."""
    r = sigmoid(block_diag_apply(x, Wa, ba))
    i = sigmoid(block_diag_apply(x, Wi, bi))
    log_a = -RG_GATE_C * r * softplus(lam)[None, :]
    a = np.exp(log_a)
    gated = x * i
    h = np.array(h0, dtype=np.float64)
    out = np.empty_like(gated)
    for t in range(x.shape[0]):
        if t == 0 and reset_first:
            h = gated[t]
        else:
            h = a[t] * h + np.sqrt(1.0 - a[t] ** 2) * gated[t]
        out[t] = h
    return out, h


class OracleRG:
    """Griffin recurrent-block language model with explicit per-sequence state."""

    def __init__(self, cfg, weights: Dict[str, np.ndarray]):
        self.cfg = cfg
        self.w = {k: np.asarray(v, dtype=np.float64) for k, v in weights.items()}
        self.reset()

    def reset(self) -> None:
        self.conv: List[List[np.ndarray]] = []   # [seq][layer] -> [K-1, W]
        self.rec: List[List[np.ndarray]] = []    # [seq][layer] -> [W]
        self.lengths: List[int] = []

    def _recurrent(self, layer: int, hn: np.ndarray, seq: int) -> np.ndarray:
        cfg, w = self.cfg, self.w
        p = f"layers.{layer}."
        y = gelu_tanh(hn @ w[p + "linear_y"].T + w[p + "linear_y_b"])
        xb = hn @ w[p + "linear_x"].T + w[p + "linear_x_b"]
        past = self.conv[seq][layer]
        xc = causal_depthwise_conv(xb, w[p + "conv_w"], w[p + "conv_b"], past)
        self.conv[seq][layer] = np.concatenate([past, xb], axis=0)[-(cfg.d_conv - 1):]
        h, self.rec[seq][layer] = rg_lru(xc, w[p + "gate_a"], w[p + "gate_a_b"], w[p + "gate_x"],
                                         w[p + "gate_x_b"], w[p + "lambda"], self.rec[seq][layer],
                                         self.lengths[seq] == 0)
        return (h * y) @ w[p + "linear_out"].T + w[p + "linear_out_b"]

    def _mlp(self, layer: int, hn: np.ndarray) -> np.ndarray:
        w = self.w
        p = f"layers.{layer}."
        g = gelu_tanh(hn @ w[p + "mlp_gate"].T + w[p + "mlp_gate_b"])
        u = hn @ w[p + "mlp_up"].T + w[p + "mlp_up_b"]
        return (g * u) @ w[p + "mlp_down"].T + w[p + "mlp_down_b"]

    def _run(self, seq: int, tokens: np.ndarray, all_logits: bool) -> np.ndarray:
        cfg, w = self.cfg, self.w
        x = w["embed"][np.asarray(tokens, dtype=np.int64)] * cfg.embed_scale
        for layer in range(cfg.n_layers):
            p = f"layers.{layer}."
            x = x + self._recurrent(layer, rms_norm_offset(x, w[p + "norm_t"], cfg.rms_eps), seq)
            x = x + self._mlp(layer, rms_norm_offset(x, w[p + "norm_c"], cfg.rms_eps))
        self.lengths[seq] += len(tokens)
        rows = x if all_logits else x[-1:]
        logits = soft_cap(rms_norm_offset(rows, w["final_norm"], cfg.rms_eps) @ w["embed"].T,
                          cfg.logit_cap)
        return logits if all_logits else logits[0]

    def _new_seq(self) -> None:
        cfg = self.cfg
        self.conv.append([np.zeros((cfg.d_conv - 1, cfg.lru_width)) for _ in range(cfg.n_layers)])
        self.rec.append([np.zeros(cfg.lru_width) for _ in range(cfg.n_layers)])
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
        saved = (self.conv, self.rec, self.lengths)
        try:
            self.reset()
            self._new_seq()
            return self._run(0, tokens, True)
        finally:
            self.conv, self.rec, self.lengths = saved


def teacher_forced_run_rg(model: OracleRG, lengths, packed, n_decode: int):
    """Prefill, then n_decode steps fed the oracle's own greedy tokens."""
    logits = [model.prefill(split_prompts(lengths, packed))]
    toks = [argmax_lowest(logits[0])]
    for _ in range(n_decode):
        logits.append(model.decode(toks[-1]))
        toks.append(argmax_lowest(logits[-1]))
    return np.stack(logits), np.stack(toks)
