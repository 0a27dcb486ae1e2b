"""Pins of the fp64 Mamba2 oracle against facts that do not come from the oracle itself.

* an independent library implementation of the same model: transformers' Mamba2 in float64,
  whose prefill runs the chunked state-space-duality algorithm (block matrices per chunk plus
  a recurrence over chunk states) rather than the step recurrence the oracle uses; its scan
  and RMSNorms compute in fp32 internally, hence the 1e-6-level tolerance;
* a special case that reduces to another routine: a Mamba2 head with one row and the same
  decay for every state is a Mamba selective-scan channel (oracle.mamba, itself pinned);
* closed forms: constant inputs (geometric series), zero input (pure decay);
* invariants: incremental decode and chunked continuation == full recompute, causality;
* planted mistakes (head-to-group map, dropped skip term, decay without dt, SiLU replaced by
  the sigmoid) each fail the library pin.
"""
import numpy as np
import pytest
import torch

from oracle import mamba as M1
from oracle import mamba2 as M2
from oracle import transformer as T
from synth import gen
from synth import mamba2 as S2

MICRO = S2.Mamba2Config(name="micro-mamba2", seed=121, dtype="f32", n_layers=2, d_model=16,
                        d_inner=32, d_state=8, head_dim=8, n_groups=2, d_conv=4, vocab=13,
                        batch=2, prompt_list=(6, 3), n_decode=3, init_std=0.3)


def micro_weights(cfg=MICRO):
    """Generator tensors with gains and skip weights randomised as well."""
    w = S2.weights(cfg)
    rng = np.random.default_rng(6)
    for l in range(cfg.n_layers):
        p = f"layers.{l}."
        w[p + "norm"] = 1 + 0.2 * rng.standard_normal(cfg.d_model)
        w[p + "gnorm"] = 1 + 0.2 * rng.standard_normal(cfg.d_inner)
        w[p + "D"] = rng.standard_normal(cfg.n_heads)
        w[p + "dt_b"] = w[p + "dt_b"] + 1.0
    w["final_norm"] = 1 + 0.2 * rng.standard_normal(cfg.d_model)
    return w


def hf_mamba2(cfg, w):
    from transformers import Mamba2Config, Mamba2ForCausalLM
    hc = Mamba2Config(vocab_size=cfg.vocab, hidden_size=cfg.d_model, state_size=cfg.d_state,
                      num_heads=cfg.n_heads, head_dim=cfg.head_dim,
                      expand=cfg.d_inner // cfg.d_model, n_groups=cfg.n_groups,
                      conv_kernel=cfg.d_conv, use_conv_bias=True, use_bias=False,
                      num_hidden_layers=cfg.n_layers, layer_norm_epsilon=cfg.rms_eps,
                      residual_in_fp32=True, tie_word_embeddings=True, chunk_size=16,
                      time_step_limit=(0.0, float("inf")), rms_norm=True)
    m = Mamba2ForCausalLM(hc).double().eval()
    t = lambda a: torch.tensor(np.asarray(a, dtype=np.float64))
    sd = {"backbone.embeddings.weight": t(w["embed"]), "lm_head.weight": t(w["embed"]),
          "backbone.norm_f.weight": t(w["final_norm"])}
    for l in range(cfg.n_layers):
        p, q = f"layers.{l}.", f"backbone.layers.{l}."
        sd[q + "norm.weight"] = t(w[p + "norm"])
        sd[q + "mixer.in_proj.weight"] = t(w[p + "in_proj"])
        sd[q + "mixer.conv1d.weight"] = t(w[p + "conv_w"])[:, None, :]
        sd[q + "mixer.conv1d.bias"] = t(w[p + "conv_b"])
        sd[q + "mixer.dt_bias"] = t(w[p + "dt_b"])
        sd[q + "mixer.A_log"] = t(w[p + "A_log"])
        sd[q + "mixer.D"] = t(w[p + "D"])
        sd[q + "mixer.norm.weight"] = t(w[p + "gnorm"])
        sd[q + "mixer.out_proj.weight"] = t(w[p + "out_proj"])
    m.load_state_dict(sd, strict=True)
    return m


def _rel_err(a, b):
    return float(np.max(np.abs(np.asarray(a) - np.asarray(b))) / np.max(np.abs(b)))


def _hf_logits(cfg, w, toks):
    with torch.no_grad():
        return hf_mamba2(cfg, w)(torch.tensor(np.asarray(toks)[None])).logits[0].numpy()


@pytest.mark.parametrize("cfg", [MICRO, S2.MAMBA2_TEST_CONFIGS["t-mamba2"],
                                 S2.MAMBA2_TEST_CONFIGS["t-mamba2-f32"]], ids=lambda c: c.name)
def test_full_forward_matches_library_mamba2(cfg):
    w = micro_weights(cfg) if cfg is MICRO else S2.weights(cfg)
    toks = np.random.default_rng(3).integers(0, cfg.vocab, size=45)
    ref = _hf_logits(cfg, w, toks)
    got = M2.OracleMamba2(cfg, w).forward_full(toks)
    assert _rel_err(got, ref) < 2e-6


def test_cached_decode_matches_library_mamba2():
    cfg = MICRO
    w = micro_weights(cfg)
    lens, packed = gen.prompt_tokens(cfg)
    o = M2.OracleMamba2(cfg, w)
    logits, toks = M2.teacher_forced_run_mamba2(o, lens, packed, cfg.n_decode)
    for b, p in enumerate(T.split_prompts(lens, packed)):
        seq = np.concatenate([p, toks[:-1, b]])
        ref = _hf_logits(cfg, w, seq)
        for s in range(cfg.n_decode + 1):
            assert _rel_err(logits[s, b], ref[len(p) - 1 + s]) < 2e-6


def test_one_row_head_is_a_selective_scan_channel():
    """P = 1, G = H: head h is Mamba channel h with A[h, n] = A_h for every state n."""
    rng = np.random.default_rng(1)
    Tn, H, N = 23, 5, 6
    x = rng.standard_normal((Tn, H, 1))
    dt = np.exp(rng.uniform(-4, 0, (Tn, H)))
    A = -np.exp(rng.standard_normal(H))
    B, C = rng.standard_normal((Tn, H, N)), rng.standard_normal((Tn, H, N))
    D = rng.standard_normal(H)
    h0 = rng.standard_normal((H, 1, N))
    y2, h2 = M2.ssd_scan(x, dt, A, B, C, D, h0, np.arange(H))
    for hh in range(H):
        y1, h1 = M1.selective_scan(x[:, hh, :], dt[:, hh:hh + 1], np.full((1, N), A[hh]),
                                   B[:, hh], C[:, hh], D[hh:hh + 1], h0[hh])
        np.testing.assert_allclose(y2[:, hh], y1, rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(h2[hh], h1, rtol=1e-12, atol=1e-12)


def test_ssd_scan_closed_forms():
    rng = np.random.default_rng(2)
    Tn, H, P, N, G = 29, 4, 3, 5, 2
    goh = np.arange(H) // (H // G)
    x = np.tile(rng.standard_normal((1, H, P)), (Tn, 1, 1))
    dt = np.tile(np.exp(rng.uniform(-3, 0, (1, H))), (Tn, 1))
    A = -np.exp(rng.standard_normal(H))
    B = np.tile(rng.standard_normal((1, G, N)), (Tn, 1, 1))
    C = np.tile(rng.standard_normal((1, G, N)), (Tn, 1, 1))
    D = rng.standard_normal(H)
    y, hT = M2.ssd_scan(x, dt, A, B, C, D, np.zeros((H, P, N)), goh)
    a = np.exp(dt[0] * A)
    for t in (1, 5, Tn):
        geo = (1 - a ** t) / (1 - a)
        h = (dt[0][:, None] * x[0])[:, :, None] * B[0][goh][:, None, :] * geo[:, None, None]
        np.testing.assert_allclose(y[t - 1], np.einsum("hpn,hn->hp", h, C[0][goh]) + D[:, None] * x[0],
                                   rtol=1e-12, atol=1e-12)
    # zero input: pure decay of the initial state
    h0 = rng.standard_normal((H, P, N))
    y, hT = M2.ssd_scan(np.zeros((Tn, H, P)), dt, A, B, C, D, h0, goh)
    np.testing.assert_allclose(hT, np.exp(Tn * dt[0] * A)[:, None, None] * h0, rtol=1e-12)


def _chunked_matrix_form(x, dt, A, B, C, D, h0, goh, Q):
    """The same scan as products over chunks of Q steps (state-space duality form), written
    out independently of the oracle: per chunk and head, with c the running sum of dt,
    y = diag(e^{A c}) C h_in^T + ((C B^T) o L) x + D x, L[t, s] = e^{A (c_t - c_s)} dt_s (s <= t),
    and h_out = e^{A c_last} h_in + x^T diag(dt_s e^{A (c_last - c_s)}) B."""
    Tn, H, P = x.shape
    h = np.array(h0, dtype=np.float64)
    y = np.empty((Tn, H, P))
    for t0 in range(0, Tn, Q):
        q = min(Q, Tn - t0)
        for hh in range(H):
            Bc, Cc = B[t0:t0 + q, goh[hh]], C[t0:t0 + q, goh[hh]]      # [q, N]
            xc, dc = x[t0:t0 + q, hh], dt[t0:t0 + q, hh]                 # [q, P], [q]
            c = np.cumsum(dc)
            L = np.tril(np.exp(A[hh] * (c[:, None] - c[None, :])) * dc[None, :])
            y[t0:t0 + q, hh] = (np.exp(A[hh] * c)[:, None] * (Cc @ h[hh].T)
                                + ((Cc @ Bc.T) * L) @ xc + D[hh] * xc)
            w = dc * np.exp(A[hh] * (c[-1] - c))
            h[hh] = np.exp(A[hh] * c[-1]) * h[hh] + xc.T @ (w[:, None] * Bc)
    return y, h


@pytest.mark.parametrize("Q", [1, 7, 64])
def test_ssd_scan_equals_its_chunked_matrix_form(Q):
    """The identity the GPU's prefill scan of 16-bit models evaluates (chunks of 64 steps as
    matrix products) pinned against the step recurrence: several chunks, a ragged last one,
    two B/C groups and a nonzero incoming state."""
    rng = np.random.default_rng(12)
    Tn, H, P, N, G = 150, 4, 5, 6, 2
    goh = np.arange(H) // (H // G)
    x = rng.standard_normal((Tn, H, P))
    dt = np.exp(rng.uniform(-4, 0, (Tn, H)))
    A = -np.exp(rng.standard_normal(H))
    B, C = rng.standard_normal((Tn, G, N)), rng.standard_normal((Tn, G, N))
    D = rng.standard_normal(H)
    h0 = rng.standard_normal((H, P, N))
    y_ref, h_ref = M2.ssd_scan(x, dt, A, B, C, D, h0, goh)
    y, h = _chunked_matrix_form(x, dt, A, B, C, D, h0, goh, Q)
    np.testing.assert_allclose(y, y_ref, rtol=1e-10, atol=1e-11)
    np.testing.assert_allclose(h, h_ref, rtol=1e-10, atol=1e-11)


@pytest.mark.parametrize("split", [1, 4, 11])
def test_incremental_decode_and_continuation_equal_full_recompute(split):
    cfg = MICRO
    w = micro_weights(cfg)
    toks = np.random.default_rng(8).integers(0, cfg.vocab, size=16)
    o = M2.OracleMamba2(cfg, w)
    full = o.forward_full(toks)
    got = [o.prefill([toks[:split]])[0]]
    got.append(o.extend([toks[split:split + 2]])[0])
    for t in toks[split + 2:]:
        got.append(o.decode([t])[0])
    np.testing.assert_allclose(got[0], full[split - 1], rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(got[1], full[split + 1], rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(np.stack(got[2:]), full[split + 2:], rtol=1e-11, atol=1e-12)


def test_causality():
    cfg = MICRO
    w = micro_weights(cfg)
    a = np.random.default_rng(10).integers(0, cfg.vocab, size=12)
    b = a.copy()
    b[7:] = (b[7:] + 1) % cfg.vocab
    o = M2.OracleMamba2(cfg, w)
    la, lb = o.forward_full(a), o.forward_full(b)
    np.testing.assert_array_equal(la[:7], lb[:7])
    assert np.abs(la[7:] - lb[7:]).max() > 1e-3


_ORIG = M2.ssd_scan


def _wrong_group_map(x, dt, A, B, C, D, h0, goh):
    return _ORIG(x, dt, A, B, C, D, h0, np.arange(len(goh)) % B.shape[1])


def _no_skip(x, dt, A, B, C, D, h0, goh):
    return _ORIG(x, dt, A, B, C, np.zeros_like(D), h0, goh)


def _decay_without_dt(x, dt, A, B, C, D, h0, goh):
    h = np.array(h0, dtype=np.float64)
    y = np.empty_like(x, dtype=np.float64)
    for t in range(x.shape[0]):
        h = np.exp(A)[:, None, None] * h + (dt[t][:, None] * x[t])[:, :, None] * B[t][goh][:, None, :]
        y[t] = np.einsum("hpn,hn->hp", h, C[t][goh]) + D[:, None] * x[t]
    return y, h


def _silu_as_sigmoid(z):
    return 1.0 / (1.0 + np.exp(-z))


@pytest.mark.parametrize("name,fn", [("ssd_scan", _wrong_group_map), ("ssd_scan", _no_skip),
                                     ("ssd_scan", _decay_without_dt), ("silu", _silu_as_sigmoid)])
def test_planted_mistake_is_caught(monkeypatch, name, fn):
    cfg = MICRO
    w = micro_weights(cfg)
    toks = np.random.default_rng(7).integers(0, cfg.vocab, size=9)
    ref = _hf_logits(cfg, w, toks)
    monkeypatch.setattr(M2, name, fn)
    bad = M2.OracleMamba2(cfg, w).forward_full(toks)
    assert _rel_err(bad, ref) > 1e-3
