"""Pins of the fp64 RG-LRU (Griffin recurrent block) oracle against facts that do not come
from the oracle itself.

* an independent library implementation of the same model: transformers' RecurrentGemma in
  float64 with every temporal block recurrent, run without a cache (its full forward); its
  RG-LRU scan accumulates in fp32, hence the 1e-6-level tolerance;
* library routines for the pieces: torch's tanh-approximated GELU, a dense block-diagonal
  matrix for the per-head gates;
* closed forms of the RG-LRU: constant inputs (geometric series), zero input (pure decay of the
  initial state), softplus(lambda) -> 0 (a = 1: the state keeps the first token's input);
* invariants: incremental decode and chunked continuation == full recompute, causality;
* planted mistakes (no reset of the first token, the sqrt(1 - a^2) factor dropped, gate
  blocks transposed, no soft cap, gate constant 1 instead of 8) each fail the library pin.
"""
import numpy as np
import pytest
import scipy.linalg
import torch

from oracle import rglru as R
from oracle import transformer as T
from synth import gen
from synth import rglru as SR

MICRO = SR.RGConfig(name="micro-rg", seed=131, dtype="f32", n_layers=2, d_model=16,
                    lru_width=24, n_heads=3, mlp_width=20, d_conv=4, vocab=13, batch=2,
                    prompt_list=(6, 3), n_decode=3, init_std=0.3, norm_std=0.2)


def hf_rg(cfg, w):
    from transformers import RecurrentGemmaConfig, RecurrentGemmaForCausalLM
    hc = RecurrentGemmaConfig(vocab_size=cfg.vocab, hidden_size=cfg.d_model,
                              intermediate_size=2 * cfg.mlp_width,
                              num_attention_heads=cfg.n_heads, lru_width=cfg.lru_width,
                              num_hidden_layers=cfg.n_layers, conv1d_width=cfg.d_conv,
                              logits_soft_cap=cfg.logit_cap, rms_norm_eps=cfg.rms_eps,
                              block_types=("recurrent",), hidden_activation="gelu_pytorch_tanh",
                              tie_word_embeddings=True)
    m = RecurrentGemmaForCausalLM(hc).double().eval()
    t = lambda a: torch.tensor(np.asarray(a, dtype=np.float64))
    sd = {"model.embed_tokens.weight": t(w["embed"]), "lm_head.weight": t(w["embed"]),
          "model.final_norm.weight": t(w["final_norm"])}
    for l in range(cfg.n_layers):
        p, q = f"layers.{l}.", f"model.layers.{l}."
        tb = q + "temporal_block."
        sd[q + "temporal_pre_norm.weight"] = t(w[p + "norm_t"])
        sd[q + "channel_pre_norm.weight"] = t(w[p + "norm_c"])
        for mine, theirs in (("linear_y", "linear_y"), ("linear_x", "linear_x"),
                             ("linear_out", "linear_out")):
            sd[tb + theirs + ".weight"] = t(w[p + mine])
            sd[tb + theirs + ".bias"] = t(w[p + mine + "_b"])
        sd[tb + "conv_1d.weight"] = t(w[p + "conv_w"])[:, None, :]
        sd[tb + "conv_1d.bias"] = t(w[p + "conv_b"])
        sd[tb + "rg_lru.recurrent_param"] = t(w[p + "lambda"])
        # the library's gate blocks act as x @ W ([in][out]); ours are [out][in]
        sd[tb + "rg_lru.input_gate_weight"] = t(np.transpose(w[p + "gate_x"], (0, 2, 1)))
        sd[tb + "rg_lru.input_gate_bias"] = t(w[p + "gate_x_b"])
        sd[tb + "rg_lru.recurrent_gate_weight"] = t(np.transpose(w[p + "gate_a"], (0, 2, 1)))
        sd[tb + "rg_lru.recurrent_gate_bias"] = t(w[p + "gate_a_b"])
        for mine, theirs in (("mlp_gate", "gate_proj"), ("mlp_up", "up_proj"),
                             ("mlp_down", "down_proj")):
            sd[q + "mlp_block." + theirs + ".weight"] = t(w[p + mine])
            sd[q + "mlp_block." + theirs + ".bias"] = t(w[p + mine + "_b"])
    missing, unexpected = m.load_state_dict(sd, strict=False)
    assert not unexpected and all("normalizer" in k for k in missing), (missing, unexpected)
    return m


def _rel_err(a, b):
    return float(np.max(np.abs(np.asarray(a) - np.asarray(b))) / np.max(np.abs(b)))


def _hf_logits(cfg, w, toks):
    with torch.no_grad():
        out = hf_rg(cfg, w)(torch.tensor(np.asarray(toks)[None]), use_cache=False)
    return out.logits[0].numpy()


@pytest.mark.parametrize("cfg", [MICRO, SR.RG_TEST_CONFIGS["t-rg"],
                                 SR.RG_TEST_CONFIGS["t-rg-f32"]], ids=lambda c: c.name)
def test_full_forward_matches_library_recurrentgemma(cfg):
    w = SR.weights(cfg)
    toks = np.random.default_rng(3).integers(0, cfg.vocab, size=41)
    ref = _hf_logits(cfg, w, toks)
    got = R.OracleRG(cfg, w).forward_full(toks)
    assert _rel_err(got, ref) < 2e-6


def test_library_normalizer_is_the_bf16_embed_scale():
    cfg = SR.RG_TEST_CONFIGS["t-rg"]          # sqrt(128) = 11.3137... is not a bf16 value
    m = hf_rg(cfg, SR.weights(cfg))
    assert float(m.model.normalizer) == cfg.embed_scale == 11.3125


def test_gelu_tanh_is_torch_gelu_tanh():
    x = np.linspace(-8, 8, 1001)
    ref = torch.nn.functional.gelu(torch.tensor(x), approximate="tanh").numpy()
    np.testing.assert_allclose(R.gelu_tanh(x), ref, rtol=1e-14, atol=1e-15)


def test_block_diag_gates_are_a_dense_block_diagonal_matrix():
    rng = np.random.default_rng(4)
    H, bw, Tn = 3, 5, 7
    W = rng.standard_normal((H, bw, bw))
    b = rng.standard_normal((H, bw))
    x = rng.standard_normal((Tn, H * bw))
    dense = scipy.linalg.block_diag(*W)                 # [out][in]
    np.testing.assert_allclose(R.block_diag_apply(x, W, b), x @ dense.T + b.reshape(-1),
                               rtol=1e-13, atol=1e-13)


def _lru_params(rng, H, bw):
    return (rng.standard_normal((H, bw, bw)) * 0.3, rng.standard_normal((H, bw)) * 0.3,
            rng.standard_normal((H, bw, bw)) * 0.3, rng.standard_normal((H, bw)) * 0.3,
            np.log(np.expm1(rng.uniform(0.01, 0.3, H * bw))))


def test_rg_lru_closed_forms():
    rng = np.random.default_rng(5)
    H, bw, Tn = 2, 4, 19
    Wa, ba, Wi, bi, lam = _lru_params(rng, H, bw)
    # constant input from a reset: h_t = a^t h_0 + b (1 - a^t) / (1 - a), h_0 = i x
    x = np.tile(rng.standard_normal((1, H * bw)), (Tn, 1))
    out, hT = R.rg_lru(x, Wa, ba, Wi, bi, lam, np.zeros(H * bw), True)
    r = 1 / (1 + np.exp(-(R.block_diag_apply(x[:1], Wa, ba)[0])))
    i = 1 / (1 + np.exp(-(R.block_diag_apply(x[:1], Wi, bi)[0])))
    a = np.exp(-8.0 * r * np.log1p(np.exp(lam)))
    b = np.sqrt(1 - a * a) * i * x[0]
    for t in (0, 1, 6, Tn - 1):
        expect = a ** t * (i * x[0]) + b * (1 - a ** t) / (1 - a)
        np.testing.assert_allclose(out[t], expect, rtol=1e-12, atol=1e-14)
    # zero input on a held state: pure decay with r = sigmoid(b_a)
    h0 = rng.standard_normal(H * bw)
    out, hT = R.rg_lru(np.zeros((Tn, H * bw)), Wa, ba, Wi, bi, lam, h0, False)
    a0 = np.exp(-8.0 / (1 + np.exp(-ba.reshape(-1))) * np.log1p(np.exp(lam)))
    np.testing.assert_allclose(hT, a0 ** Tn * h0, rtol=1e-12)
    # softplus(lambda) -> 0: a = 1, the input weight sqrt(1 - a^2) = 0, the state keeps i_0 x_0
    x = rng.standard_normal((Tn, H * bw))
    out, hT = R.rg_lru(x, Wa, ba, Wi, bi, np.full(H * bw, -800.0), np.zeros(H * bw), True)
    i0 = 1 / (1 + np.exp(-(R.block_diag_apply(x[:1], Wi, bi)[0])))
    np.testing.assert_allclose(out, np.tile(i0 * x[0], (Tn, 1)), rtol=1e-12, atol=1e-15)


@pytest.mark.parametrize("split", [1, 4, 11])
def test_incremental_decode_and_continuation_equal_full_recompute(split):
    cfg = MICRO
    w = SR.weights(cfg)
    toks = np.random.default_rng(8).integers(0, cfg.vocab, size=16)
    o = R.OracleRG(cfg, w)
    full = o.forward_full(toks)
    got = [o.prefill([toks[:split]])[0]]
    got.append(o.extend([toks[split:split + 2]])[0])
    for t in toks[split + 2:]:
        got.append(o.decode([t])[0])
    np.testing.assert_allclose(got[0], full[split - 1], rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(got[1], full[split + 1], rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(np.stack(got[2:]), full[split + 2:], rtol=1e-11, atol=1e-12)


def test_batched_prefill_and_decode_match_per_sequence_recompute():
    cfg = MICRO
    w = SR.weights(cfg)
    lens, packed = gen.prompt_tokens(cfg)
    o = R.OracleRG(cfg, w)
    logits, toks = R.teacher_forced_run_rg(o, lens, packed, cfg.n_decode)
    for b, p in enumerate(T.split_prompts(lens, packed)):
        seq = np.concatenate([p, toks[:-1, b]])
        ref = R.OracleRG(cfg, w).forward_full(seq)
        for s in range(cfg.n_decode + 1):
            np.testing.assert_allclose(logits[s, b], ref[len(p) - 1 + s], rtol=1e-11, atol=1e-12)


def test_causality():
    cfg = MICRO
    w = SR.weights(cfg)
    a = np.random.default_rng(10).integers(0, cfg.vocab, size=12)
    b = a.copy()
    b[7:] = (b[7:] + 1) % cfg.vocab
    o = R.OracleRG(cfg, w)
    la, lb = o.forward_full(a), o.forward_full(b)
    np.testing.assert_array_equal(la[:7], lb[:7])
    assert np.abs(la[7:] - lb[7:]).max() > 1e-3


_ORIG_LRU = R.rg_lru


def _no_reset(x, Wa, ba, Wi, bi, lam, h0, reset_first):
    return _ORIG_LRU(x, Wa, ba, Wi, bi, lam, h0, False)


def _no_input_norm(x, Wa, ba, Wi, bi, lam, h0, reset_first):
    r = R.sigmoid(R.block_diag_apply(x, Wa, ba))
    i = R.sigmoid(R.block_diag_apply(x, Wi, bi))
    a = np.exp(-8.0 * r * R.softplus(lam)[None, :])
    h = np.array(h0, dtype=np.float64)
    out = np.empty_like(x)
    for t in range(x.shape[0]):
        h = (0 if (t == 0 and reset_first) else a[t] * h) + i[t] * x[t]
        out[t] = h
    return out, h


def _transposed_blocks(x, Wa, ba, Wi, bi, lam, h0, reset_first):
    return _ORIG_LRU(x, np.transpose(Wa, (0, 2, 1)), ba, np.transpose(Wi, (0, 2, 1)), bi, lam,
                     h0, reset_first)


def _gate_constant_one(x, Wa, ba, Wi, bi, lam, h0, reset_first):
    return _ORIG_LRU(x, Wa, ba, Wi, bi, np.log(np.expm1(R.softplus(lam) / 8.0)), h0, reset_first)


@pytest.mark.parametrize("name,fn", [("rg_lru", _no_reset), ("rg_lru", _no_input_norm),
                                     ("rg_lru", _transposed_blocks),
                                     ("rg_lru", _gate_constant_one),
                                     ("soft_cap", lambda l, c: l)])
def test_planted_mistake_is_caught(monkeypatch, name, fn):
    cfg = MICRO
    w = SR.weights(cfg)
    toks = np.random.default_rng(7).integers(0, cfg.vocab, size=9)
    ref = _hf_logits(cfg, w, toks)
    monkeypatch.setattr(R, name, fn)
    bad = R.OracleRG(cfg, w).forward_full(toks)
    assert _rel_err(bad, ref) > 1e-3
