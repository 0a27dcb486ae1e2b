"""Pins of the fp64 Mamba oracle against facts that do not come from the oracle itself.

* an independent library implementation of the same model (transformers' Mamba in float64 on
  the CPU, its sequential "slow" path; its RMSNorm runs in fp32 internally, hence the
  1e-6-level tolerance);
* brute force: a pure-Python scalar-loop model on a micro configuration;
* closed forms: the scan under constant inputs (geometric series), the scan with a state that
  forgets at once, the convolution's impulse response, softplus limits;
* invariants: incremental decode == full recompute (any split point), causality, batch
  independence;
* planted mistakes in the oracle (sign of A, dropped skip term, reversed taps, missing gate,
  missing softplus) each fail the library pin.
"""
import math

import numpy as np
import pytest
import torch

from oracle import mamba as M
from oracle import transformer as T
from synth import gen
from synth import mamba as SM

MICRO = SM.MambaConfig(name="micro-mamba", seed=111, dtype="f32", n_layers=2, d_model=16,
                       d_inner=32, d_state=4, d_conv=4, dt_rank=3, vocab=13, batch=2,
                       prompt_list=(6, 3), n_decode=3, init_std=0.3)


def micro_weights(cfg=MICRO):
    """The generator's tensors, with gains, skip weights and decay rates also randomised so
    that every term of the mixer visibly moves the logits."""
    w = SM.weights(cfg)
    rng = np.random.default_rng(5)
    for l in range(cfg.n_layers):
        p = f"layers.{l}."
        w[p + "norm"] = 1 + 0.2 * rng.standard_normal(cfg.d_model)
        w[p + "D"] = rng.standard_normal(cfg.d_inner)
        w[p + "A_log"] = w[p + "A_log"] + 0.3 * rng.standard_normal(w[p + "A_log"].shape)
        w[p + "dt_b"] = w[p + "dt_b"] + 1.0
    w["final_norm"] = 1 + 0.2 * rng.standard_normal(cfg.d_model)
    return w


def hf_mamba(cfg, w):
    from transformers import MambaConfig, MambaForCausalLM
    hc = MambaConfig(vocab_size=cfg.vocab, hidden_size=cfg.d_model, state_size=cfg.d_state,
                     num_hidden_layers=cfg.n_layers, layer_norm_epsilon=cfg.rms_eps,
                     expand=cfg.d_inner // cfg.d_model, intermediate_size=cfg.d_inner,
                     conv_kernel=cfg.d_conv, use_bias=False, use_conv_bias=True,
                     hidden_act="silu", time_step_rank=cfg.dt_rank, residual_in_fp32=True,
                     tie_word_embeddings=True)
    m = MambaForCausalLM(hc).double().eval()
    t = lambda a: torch.tensor(np.asarray(a, dtype=np.float64))
    sd = {"backbone.embeddings.weight": t(w["embed"]), "lm_head.weight": t(w["embed"]),
          "backbone.norm_f.weight": t(w["final_norm"])}
    for l in range(cfg.n_layers):
        p, q = f"layers.{l}.", f"backbone.layers.{l}."
        sd[q + "norm.weight"] = t(w[p + "norm"])
        sd[q + "mixer.A_log"] = t(w[p + "A_log"])
        sd[q + "mixer.D"] = t(w[p + "D"])
        sd[q + "mixer.conv1d.weight"] = t(w[p + "conv_w"])[:, None, :]
        sd[q + "mixer.conv1d.bias"] = t(w[p + "conv_b"])
        sd[q + "mixer.in_proj.weight"] = t(w[p + "in_proj"])
        sd[q + "mixer.x_proj.weight"] = t(w[p + "x_proj"])
        sd[q + "mixer.dt_proj.weight"] = t(w[p + "dt_w"])
        sd[q + "mixer.dt_proj.bias"] = t(w[p + "dt_b"])
        sd[q + "mixer.out_proj.weight"] = t(w[p + "out_proj"])
    m.load_state_dict(sd, strict=True)
    return m


def _rel_err(a, b):
    return float(np.max(np.abs(np.asarray(a) - np.asarray(b))) / np.max(np.abs(b)))


def _hf_logits(cfg, w, toks):
    with torch.no_grad():
        return hf_mamba(cfg, w)(torch.tensor(np.asarray(toks)[None])).logits[0].numpy()


# ------------------------------------------------------------------------------------------
# Library implementation
# ------------------------------------------------------------------------------------------

@pytest.mark.parametrize("cfg", [MICRO, SM.MAMBA_TEST_CONFIGS["t-mamba-f32"]],
                         ids=lambda c: c.name)
def test_full_forward_matches_library_mamba(cfg):
    w = micro_weights(cfg) if cfg is MICRO else SM.weights(cfg)
    toks = np.random.default_rng(3).integers(0, cfg.vocab, size=48)
    ref = _hf_logits(cfg, w, toks)
    got = M.OracleMamba(cfg, w).forward_full(toks)
    assert _rel_err(got, ref) < 2e-6


def test_cached_decode_matches_library_mamba():
    """Prefill of a ragged batch and decode steps, each sequence against the library's full
    forward over the same tokens."""
    cfg = MICRO
    w = micro_weights(cfg)
    lens, packed = gen.prompt_tokens(cfg)
    o = M.OracleMamba(cfg, w)
    logits, toks = M.teacher_forced_run_mamba(o, lens, packed, cfg.n_decode)
    for b, p in enumerate(T.split_prompts(lens, packed)):
        seq = np.concatenate([p, toks[:-1, b]])
        ref = _hf_logits(cfg, w, seq)
        for s in range(cfg.n_decode + 1):
            assert _rel_err(logits[s, b], ref[len(p) - 1 + s]) < 2e-6


# ------------------------------------------------------------------------------------------
# Brute force
# ------------------------------------------------------------------------------------------

def _bruteforce_logits(cfg, w, toks):
    """Scalar loops only: no numpy reductions, no library calls beyond math.exp / math.log."""
    d, di, N, K, R = cfg.d_model, cfg.d_inner, cfg.d_state, cfg.d_conv, cfg.dt_rank
    W = {k: np.asarray(v, dtype=np.float64).tolist() for k, v in w.items()}

    def rms(v, g):
        ms = sum(a * a for a in v) / len(v)
        return [a / math.sqrt(ms + cfg.rms_eps) * gi for a, gi in zip(v, g)]

    def mv(mat, v):
        return [sum(mat[i][j] * v[j] for j in range(len(v))) for i in range(len(mat))]

    sig = lambda a: 1.0 / (1.0 + math.exp(-a))
    xs = [list(W["embed"][t]) for t in toks]
    for l in range(cfg.n_layers):
        p = f"layers.{l}."
        hist = [[0.0] * di for _ in range(K - 1)]
        h = [[0.0] * N for _ in range(di)]
        for t in range(len(toks)):
            xz = mv(W[p + "in_proj"], rms(xs[t], W[p + "norm"]))
            xin, z = xz[:di], xz[di:]
            hist.append(xin)
            win = hist[-K:]
            u = []
            for c in range(di):
                a = W[p + "conv_b"][c] + sum(W[p + "conv_w"][c][k] * win[k][c] for k in range(K))
                u.append(a * sig(a))
            xd = mv(W[p + "x_proj"], u)
            y = []
            for c in range(di):
                pre = W[p + "dt_b"][c] + sum(W[p + "dt_w"][c][r] * xd[r] for r in range(R))
                dt = math.log(1.0 + math.exp(pre))
                acc = W[p + "D"][c] * u[c]
                for n in range(N):
                    A = -math.exp(W[p + "A_log"][c][n])
                    h[c][n] = math.exp(dt * A) * h[c][n] + dt * xd[R + n] * u[c]
                    acc += xd[R + N + n] * h[c][n]
                y.append(acc * z[c] * sig(z[c]))
            out = mv(W[p + "out_proj"], y)
            xs[t] = [a + b for a, b in zip(xs[t], out)]
    return np.array([mv(W["embed"], rms(x, W["final_norm"])) for x in xs])


def test_bruteforce_micro_model():
    cfg = MICRO
    w = micro_weights(cfg)
    toks = np.random.default_rng(9).integers(0, cfg.vocab, size=11)
    ref = _bruteforce_logits(cfg, w, toks)
    got = M.OracleMamba(cfg, w).forward_full(toks)
    assert _rel_err(got, ref) < 1e-12


# ------------------------------------------------------------------------------------------
# Closed forms
# ------------------------------------------------------------------------------------------

def test_scan_constant_inputs_geometric_series():
    """Constant dt, u, B, C: h_t = dt u B (1 - a^t) / (1 - a) with a = exp(dt A)."""
    rng = np.random.default_rng(1)
    C_, N, T_ = 5, 4, 37
    A = -np.exp(rng.standard_normal((C_, N)))
    dt = np.exp(rng.uniform(-4, 0, C_))
    u = rng.standard_normal(C_)
    B, Cv, D = rng.standard_normal(N), rng.standard_normal(N), rng.standard_normal(C_)
    y, hT = M.selective_scan(np.tile(u, (T_, 1)), np.tile(dt, (T_, 1)), A, np.tile(B, (T_, 1)),
                             np.tile(Cv, (T_, 1)), D, np.zeros((C_, N)))
    a = np.exp(dt[:, None] * A)
    for t in (1, 2, 17, T_):
        h = (dt * u)[:, None] * B[None] * (1 - a ** t) / (1 - a)
        np.testing.assert_allclose(y[t - 1], h @ Cv + D * u, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(hT, (dt * u)[:, None] * B[None] * (1 - a ** T_) / (1 - a),
                               rtol=1e-12, atol=1e-14)


def test_scan_initial_state_decay_and_instant_forgetting():
    rng = np.random.default_rng(2)
    C_, N, T_ = 3, 4, 6
    A = -np.exp(rng.standard_normal((C_, N)))
    dt = np.full((T_, C_), 0.25)
    h0 = rng.standard_normal((C_, N))
    Cv = rng.standard_normal((T_, N))
    # zero input: y_t = C_t . (exp(t dt A) h0)
    y, _ = M.selective_scan(np.zeros((T_, C_)), dt, A, rng.standard_normal((T_, N)), Cv,
                            np.ones(C_), h0)
    for t in range(T_):
        np.testing.assert_allclose(y[t], (np.exp((t + 1) * 0.25 * A) * h0) @ Cv[t], rtol=1e-12)
    # A -> -inf: the state forgets everything, y_t = dt u (B_t . C_t) + D u
    u = rng.standard_normal((T_, C_))
    Bv = rng.standard_normal((T_, N))
    D = rng.standard_normal(C_)
    y, _ = M.selective_scan(u, dt, np.full((C_, N), -1e4), Bv, Cv, D, h0)
    np.testing.assert_allclose(y, 0.25 * u * np.sum(Bv * Cv, axis=1)[:, None] + D * u,
                               rtol=1e-12)


def test_conv_impulse_response_and_history():
    rng = np.random.default_rng(4)
    C_, K, T_ = 6, 4, 10
    w, b = rng.standard_normal((C_, K)), rng.standard_normal(C_)
    x = np.zeros((T_, C_))
    x[3] = 1.0
    out = M.causal_depthwise_conv(x, w, b, np.zeros((K - 1, C_)))
    for t in range(T_):
        j = t - 3
        expect = b + (w[:, K - 1 - j] if 0 <= j < K else 0.0)
        np.testing.assert_allclose(out[t], expect, rtol=0, atol=1e-15)
    # a block that starts after a history equals the same block inside the longer sequence
    xx = rng.standard_normal((T_, C_))
    full = M.causal_depthwise_conv(xx, w, b, np.zeros((K - 1, C_)))
    tail = M.causal_depthwise_conv(xx[5:], w, b, xx[5 - (K - 1):5])
    np.testing.assert_allclose(tail, full[5:], rtol=1e-14)
    # matches torch's grouped conv1d with left zero padding
    ref = torch.nn.functional.conv1d(torch.tensor(xx.T[None]), torch.tensor(w[:, None, :]),
                                     torch.tensor(b), padding=K - 1, groups=C_)[0, :, :T_].T
    np.testing.assert_allclose(full, ref.numpy(), rtol=1e-13, atol=1e-14)


def test_softplus_limits_and_library():
    x = np.array([-800.0, -30.0, -1.0, 0.0, 1e-3, 2.0, 30.0, 800.0])
    s = M.softplus(x)
    assert s[0] == 0.0 and s[-1] == 800.0
    assert s[3] == math.log(2.0)
    np.testing.assert_allclose(s, torch.nn.functional.softplus(torch.tensor(x)).numpy(),
                               rtol=1e-14, atol=1e-300)
    # inverse used by the weight generator: softplus(softplus^-1(dt)) = dt
    dt = np.exp(np.linspace(math.log(1e-3), math.log(0.1), 7))
    np.testing.assert_allclose(M.softplus(dt + np.log(-np.expm1(-dt))), dt, rtol=1e-12)


# ------------------------------------------------------------------------------------------
# Invariants
# ------------------------------------------------------------------------------------------

@pytest.mark.parametrize("split", [1, 5, 12])
def test_incremental_decode_equals_full_recompute(split):
    cfg = MICRO
    w = micro_weights(cfg)
    toks = np.random.default_rng(8).integers(0, cfg.vocab, size=16)
    o = M.OracleMamba(cfg, w)
    full = o.forward_full(toks)
    got = [o.prefill([toks[:split]])[0]]
    for t in toks[split:]:
        got.append(o.decode([t])[0])
    np.testing.assert_allclose(np.stack(got), full[split - 1:], rtol=1e-11, atol=1e-12)


def test_chunked_prefill_equals_full_recompute():
    """Prefill, a further chunk on the carried state, then decode: every logit equals the full
    forward over the concatenated tokens (chunks shorter than the convolution window too)."""
    cfg = MICRO
    w = micro_weights(cfg)
    rng = np.random.default_rng(12)
    a, b = rng.integers(0, cfg.vocab, size=13), rng.integers(0, cfg.vocab, size=7)
    o = M.OracleMamba(cfg, w)
    fa, fb = o.forward_full(a), o.forward_full(b)
    first = o.prefill([a[:5], b[:2]])
    second = o.extend([a[5:11], b[2:3]])
    third = o.extend([a[11:], b[3:]])
    np.testing.assert_allclose(first, np.stack([fa[4], fb[1]]), rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(second, np.stack([fa[10], fb[2]]), rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(third, np.stack([fa[12], fb[6]]), rtol=1e-11, atol=1e-12)
    assert o.lengths == [13, 7]


def test_causality_and_batch_independence():
    cfg = MICRO
    w = micro_weights(cfg)
    rng = np.random.default_rng(10)
    a = rng.integers(0, cfg.vocab, size=12)
    b = a.copy()
    b[8:] = (b[8:] + 1) % cfg.vocab
    o = M.OracleMamba(cfg, w)
    la, lb = o.forward_full(a), o.forward_full(b)
    np.testing.assert_array_equal(la[:8], lb[:8])
    assert np.abs(la[8:] - lb[8:]).max() > 1e-3
    other = rng.integers(0, cfg.vocab, size=5)
    batched = o.prefill([a, other])
    # same values up to the summation order of the LM-head product over more rows
    np.testing.assert_allclose(batched[0], la[-1], rtol=1e-13, atol=1e-13)
    np.testing.assert_array_equal(M.OracleMamba(cfg, w).prefill([other])[0], batched[1])


# ------------------------------------------------------------------------------------------
# Planted mistakes
# ------------------------------------------------------------------------------------------

_ORIG_SCAN = M.selective_scan
_ORIG_CONV = M.causal_depthwise_conv


def _scan_wrong_sign(u, dt, A, B, C, D, h0):
    return _ORIG_SCAN(u, dt, -A, B, C, D, h0)


def _scan_no_skip(u, dt, A, B, C, D, h0):
    return _ORIG_SCAN(u, dt, A, B, C, np.zeros_like(D), h0)


def _scan_b_c_swapped(u, dt, A, B, C, D, h0):
    return _ORIG_SCAN(u, dt, A, C, B, D, h0)


def _conv_reversed(x, w, b, past):
    return _ORIG_CONV(x, w[:, ::-1], b, past)


def _softplus_identity(x):
    return np.asarray(x, dtype=np.float64)


@pytest.mark.parametrize("name,fn", [
    ("selective_scan", _scan_wrong_sign), ("selective_scan", _scan_no_skip),
    ("selective_scan", _scan_b_c_swapped), ("causal_depthwise_conv", _conv_reversed),
    ("softplus", _softplus_identity), ("silu", T.softmax),
])
def test_planted_mistake_is_caught(monkeypatch, name, fn):
    cfg = MICRO
    w = micro_weights(cfg)
    toks = np.random.default_rng(7).integers(0, cfg.vocab, size=9)
    ref = _hf_logits(cfg, w, toks)
    monkeypatch.setattr(M, name, fn)
    bad = M.OracleMamba(cfg, w).forward_full(toks)
    assert not np.isfinite(bad).all() or _rel_err(bad, ref) > 1e-3


def test_generator_is_deterministic_and_bf16_exact():
    cfg = SM.MAMBA_TEST_CONFIGS["t-mamba"]
    a, b = SM.weights(cfg), SM.weights(cfg)
    assert all(np.array_equal(a[k], b[k]) for k in a)
    for name in ("embed", "layers.0.in_proj", "layers.1.x_proj", "layers.1.out_proj"):
        assert np.array_equal(gen.round_to_bf16(a[name]), a[name])
    dt = M.softplus(a["layers.0.dt_b"].astype(np.float64))
    assert dt.min() >= cfg.dt_min * 0.999 and dt.max() <= cfg.dt_max * 1.001
