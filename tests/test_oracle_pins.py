"""Pins of the fp64 oracle against facts that do not come from the oracle itself.

* an independent library implementation of the same decoder (transformers' LLaMA, float64 on
  the CPU; its RMSNorm and rotary tables run in fp32 internally, hence the 1e-6-level tolerance);
* closed forms (RoPE rotation of basis vectors, RMS of RMSNorm output, theta exponents);
* library routines (torch scaled_dot_product_attention, rms_norm, silu in float64);
* brute force: a pure-Python scalar-loop model on a micro configuration;
* invariants: incremental decode == full causal recompute, GQA == MHA with repeated K/V,
  causality, batch independence, softmax rows summing to one.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from oracle import transformer as T
from synth import gen
from synth.configs import ModelConfig

MICRO = ModelConfig(name="micro", seed=101, dtype="f32", n_layers=2, d_model=16, n_heads=4,
                    n_kv_heads=2, head_dim=4, ffn_dim=24, vocab=11, batch=2,
                    prompt_list=(5, 3), n_decode=3, rope_theta=10000.0)


def micro_weights(cfg=MICRO, scale=0.3):
    # Larger std than the workloads so that every term visibly moves the logits.
    w = gen.weights(cfg.replace(init_std=scale), random_gains=True)
    return w


# ------------------------------------------------------------------------------------------
# Library implementation of the whole decoder (transformers LLaMA in float64)
# ------------------------------------------------------------------------------------------

def hf_model(cfg, w):
    from transformers import LlamaConfig, LlamaForCausalLM
    hc = LlamaConfig(vocab_size=cfg.vocab, hidden_size=cfg.d_model, intermediate_size=cfg.ffn_dim,
                     num_hidden_layers=cfg.n_layers, num_attention_heads=cfg.n_heads,
                     num_key_value_heads=cfg.n_kv_heads, head_dim=cfg.head_dim,
                     rms_norm_eps=cfg.rms_eps, rope_theta=cfg.rope_theta,
                     tie_word_embeddings=False, attention_bias=False, mlp_bias=False,
                     max_position_embeddings=4096)
    hc._attn_implementation = "eager"
    m = LlamaForCausalLM(hc).to(torch.float64).eval()
    sd = {"model.embed_tokens.weight": w["embed"], "model.norm.weight": w["final_norm"],
          "lm_head.weight": w["lm_head"]}
    names = {"wq": "self_attn.q_proj", "wk": "self_attn.k_proj", "wv": "self_attn.v_proj",
             "wo": "self_attn.o_proj", "w_gate": "mlp.gate_proj", "w_up": "mlp.up_proj",
             "w_down": "mlp.down_proj", "attn_norm": "input_layernorm",
             "mlp_norm": "post_attention_layernorm"}
    for layer in range(cfg.n_layers):
        for k, v in names.items():
            sd[f"model.layers.{layer}.{v}.weight"] = w[f"layers.{layer}.{k}"]
    m.load_state_dict({k: torch.tensor(np.asarray(v, dtype=np.float64)) for k, v in sd.items()})
    return m


def _rel_err(a, b):
    return float(np.max(np.abs(a - b)) / max(1e-30, np.max(np.abs(b))))


@pytest.mark.parametrize("cfg", [
    MICRO,
    MICRO.replace(name="micro-mha", n_kv_heads=4, seed=102),
    MICRO.replace(name="micro-hd8", n_heads=2, n_kv_heads=1, head_dim=8, seed=103, rope_theta=500000.0),
])
def test_full_forward_matches_library_llama(cfg):
    w = micro_weights(cfg)
    toks = np.random.default_rng(7).integers(0, cfg.vocab, size=9)
    ours = T.OracleModel(cfg, w).forward_full(toks)
    with torch.no_grad():
        ref = hf_model(cfg, w)(torch.tensor(toks[None])).logits[0].numpy()
    assert _rel_err(ours, ref) < 1e-5


def test_cached_decode_matches_library_llama():
    cfg = MICRO
    w = micro_weights(cfg)
    toks = np.random.default_rng(8).integers(0, cfg.vocab, size=6)
    extra = [3, 9, 0]
    om = T.OracleModel(cfg, w)
    ours = [om.prefill([toks])[0]] + [om.decode([t])[0] for t in extra]
    m = hf_model(cfg, w)
    with torch.no_grad():
        out = m(torch.tensor(toks[None]), use_cache=True)
        ref, past = [out.logits[0, -1].numpy()], out.past_key_values
        for t in extra:
            out = m(torch.tensor([[t]]), past_key_values=past, use_cache=True)
            ref.append(out.logits[0, -1].numpy())
            past = out.past_key_values
    assert _rel_err(np.stack(ours), np.stack(ref)) < 1e-5


def test_chunked_prefill_matches_library_llama():
    """A prompt prefilled in chunks on a populated cache (extend) against transformers' LLaMA
    fed the same chunks with its own key/value cache."""
    cfg = MICRO.replace(name="micro-hd8", n_heads=2, n_kv_heads=1, head_dim=8, seed=103)
    w = micro_weights(cfg)
    toks = np.random.default_rng(9).integers(0, cfg.vocab, size=11)
    chunks = [toks[:4], toks[4:5], toks[5:11]]
    om = T.OracleModel(cfg, w)
    ours = [om.prefill([chunks[0]])[0]] + [om.extend([c])[0] for c in chunks[1:]]
    assert om.lengths == [11]
    m = hf_model(cfg, w)
    with torch.no_grad():
        out = m(torch.tensor(chunks[0][None]), use_cache=True)
        ref, past = [out.logits[0, -1].numpy()], out.past_key_values
        for c in chunks[1:]:
            out = m(torch.tensor(c[None]), past_key_values=past, use_cache=True)
            ref.append(out.logits[0, -1].numpy())
            past = out.past_key_values
    assert _rel_err(np.stack(ours), np.stack(ref)) < 1e-5


# ------------------------------------------------------------------------------------------
# Brute force: a scalar-loop model written without numpy linear algebra
# ------------------------------------------------------------------------------------------

def _bf_matvec(W, x):
    return [sum(W[o][i] * x[i] for i in range(len(x))) for o in range(len(W))]


def _bf_rms(x, g, eps):
    ms = sum(v * v for v in x) / len(x)
    r = 1.0 / math.sqrt(ms + eps)
    return [x[i] * r * g[i] for i in range(len(x))]


def _bf_rope(vec, pos, theta):
    hd = len(vec)
    half = hd // 2
    out = list(vec)
    for i in range(half):
        ang = pos * theta ** (-2.0 * i / hd)
        a, b = vec[i], vec[i + half]
        out[i] = a * math.cos(ang) - b * math.sin(ang)
        out[i + half] = b * math.cos(ang) + a * math.sin(ang)
    return out


def bruteforce_logits(cfg, w, tokens):
    """Logits at every position of one sequence, scalar Python loops only."""
    W = {k: np.asarray(v, dtype=np.float64).tolist() for k, v in w.items()}
    hd, hq, hkv = cfg.head_dim, cfg.n_heads, cfg.n_kv_heads
    xs = [list(W["embed"][t]) for t in tokens]
    for layer in range(cfg.n_layers):
        p = f"layers.{layer}."
        ks, vs, qs = [], [], []
        for pos, x in enumerate(xs):
            h = _bf_rms(x, W[p + "attn_norm"], cfg.rms_eps)
            q, k, v = _bf_matvec(W[p + "wq"], h), _bf_matvec(W[p + "wk"], h), _bf_matvec(W[p + "wv"], h)
            qs.append([_bf_rope(q[j * hd:(j + 1) * hd], pos, cfg.rope_theta) for j in range(hq)])
            ks.append([_bf_rope(k[j * hd:(j + 1) * hd], pos, cfg.rope_theta) for j in range(hkv)])
            vs.append([v[j * hd:(j + 1) * hd] for j in range(hkv)])
        new = []
        for i, x in enumerate(xs):
            o = []
            for h_ in range(hq):
                g = h_ * hkv // hq
                sc = [sum(qs[i][h_][d] * ks[j][g][d] for d in range(hd)) / math.sqrt(hd)
                      for j in range(i + 1)]
                mx = max(sc)
                e = [math.exp(s - mx) for s in sc]
                z = sum(e)
                o += [sum(e[j] / z * vs[j][g][d] for j in range(i + 1)) for d in range(hd)]
            ao = _bf_matvec(W[p + "wo"], o)
            x1 = [x[d] + ao[d] for d in range(len(x))]
            h = _bf_rms(x1, W[p + "mlp_norm"], cfg.rms_eps)
            gt, up = _bf_matvec(W[p + "w_gate"], h), _bf_matvec(W[p + "w_up"], h)
            a = [gt[f] / (1.0 + math.exp(-gt[f])) * up[f] for f in range(len(gt))]
            dn = _bf_matvec(W[p + "w_down"], a)
            new.append([x1[d] + dn[d] for d in range(len(x))])
        xs = new
    return np.array([_bf_matvec(W["lm_head"], _bf_rms(x, W["final_norm"], cfg.rms_eps)) for x in xs])


def test_bruteforce_micro_model():
    w = micro_weights()
    toks = [3, 10, 0, 7, 7]
    bf = bruteforce_logits(MICRO, w, toks)
    ours = T.OracleModel(MICRO, w).forward_full(np.array(toks))
    assert np.max(np.abs(ours - bf)) < 1e-12


# ------------------------------------------------------------------------------------------
# Closed forms and library routines, per op
# ------------------------------------------------------------------------------------------

def test_rope_frequencies_closed_form():
    for hd, theta in [(64, 1e4), (128, 5e5), (4, 1e4)]:
        f = T.rope_frequencies(hd, theta)
        assert f.shape == (hd // 2,)
        assert f[0] == 1.0
        assert math.isclose(f[-1], theta ** (-(hd - 2) / hd), rel_tol=1e-15)


def test_rope_basis_vectors_closed_form():
    hd, theta = 8, 10000.0
    for pos in [0, 1, 5, 37]:
        for i in range(hd):
            e = np.zeros((1, 1, hd))
            e[0, 0, i] = 1.0
            r = T.apply_rope(e, np.array([pos]), theta)[0, 0]
            half = hd // 2
            fi = i % half
            ang = pos * theta ** (-2.0 * fi / hd)
            want = np.zeros(hd)
            if i < half:        # e_i -> cos e_i + sin e_{i+half}
                want[i], want[i + half] = math.cos(ang), math.sin(ang)
            else:               # e_{i+half} -> -sin e_i + cos e_{i+half}
                want[i - half], want[i] = -math.sin(ang), math.cos(ang)
            assert np.allclose(r, want, atol=1e-15)


def test_rope_identity_norm_and_relative_position():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((1, 3, 64))
    assert np.array_equal(T.apply_rope(x, np.array([0]), 1e4), x)
    r = T.apply_rope(x, np.array([123]), 1e4)
    assert np.allclose(np.linalg.norm(r, axis=-1), np.linalg.norm(x, axis=-1), rtol=1e-13)
    q, k = rng.standard_normal((1, 1, 64)), rng.standard_normal((1, 1, 64))
    for m, n in [(7, 3), (100, 42), (5, 5)]:
        lhs = np.sum(T.apply_rope(q, np.array([m]), 1e4) * T.apply_rope(k, np.array([n]), 1e4))
        rhs = np.sum(T.apply_rope(q, np.array([m - n]), 1e4) * k)
        assert math.isclose(lhs, rhs, rel_tol=1e-11, abs_tol=1e-12)


def test_rmsnorm_closed_form_and_library():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((5, 32)) * 3.0
    eps = 1e-5
    y = T.rmsnorm(x, np.ones(32), eps)
    ms = np.mean(x * x, axis=-1)
    assert np.allclose(np.sqrt(np.mean(y * y, axis=-1)), np.sqrt(ms / (ms + eps)), rtol=1e-14)
    assert np.allclose(T.rmsnorm(7.5 * x, np.ones(32), 0.0), T.rmsnorm(x, np.ones(32), 0.0), rtol=1e-14)
    g = rng.standard_normal(32)
    ref = torch.nn.functional.rms_norm(torch.tensor(x), (32,), torch.tensor(g), eps).numpy()
    assert np.allclose(T.rmsnorm(x, g, eps), ref, rtol=1e-13, atol=1e-14)


def test_attention_matches_library_sdpa():
    rng = np.random.default_rng(2)
    t, hq, hkv, hd = 13, 8, 2, 16
    q, k, v = (rng.standard_normal((t, h, hd)) for h in (hq, hkv, hkv))
    pos = np.arange(t)
    ours = T.causal_gqa_attention(q, k, v, pos, pos)
    tq = torch.tensor(q).transpose(0, 1)[None]
    tk = torch.tensor(k).transpose(0, 1)[None]
    tv = torch.tensor(v).transpose(0, 1)[None]
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, is_causal=True, enable_gqa=True)
    assert np.allclose(ours, ref[0].transpose(0, 1).numpy(), rtol=1e-12, atol=1e-13)
    # single query at the last position attends to every key
    one = T.causal_gqa_attention(q[-1:], k, v, pos[-1:], pos)
    ref1 = torch.nn.functional.scaled_dot_product_attention(tq[:, :, -1:], tk, tv, enable_gqa=True)
    assert np.allclose(one, ref1[0].transpose(0, 1).numpy(), rtol=1e-12, atol=1e-13)


def test_attention_special_cases():
    rng = np.random.default_rng(3)
    q, k, v = rng.standard_normal((1, 2, 8)), rng.standard_normal((1, 1, 8)), rng.standard_normal((1, 1, 8))
    o = T.causal_gqa_attention(q, k, v, np.array([0]), np.array([0]))
    assert np.array_equal(o[0, 0], v[0, 0]) and np.array_equal(o[0, 1], v[0, 0])
    # equal keys -> the mean of the visible values
    k = np.repeat(rng.standard_normal((1, 1, 8)), 6, axis=0)
    v = rng.standard_normal((6, 1, 8))
    q = rng.standard_normal((6, 1, 8))
    o = T.causal_gqa_attention(q, k, v, np.arange(6), np.arange(6))
    for i in range(6):
        assert np.allclose(o[i, 0], v[:i + 1, 0].mean(axis=0), rtol=1e-13, atol=1e-14)


def test_softmax_rows():
    rng = np.random.default_rng(4)
    s = rng.standard_normal((7, 9)) * 10
    s[np.triu_indices(7, 1, 9)] = -np.inf
    p = T.softmax(s)
    assert np.all(p >= 0)
    assert np.max(np.abs(p.sum(axis=-1) - 1.0)) < 1e-12
    assert np.all(p[np.triu_indices(7, 1, 9)] == 0.0)


def test_silu_library():
    from scipy.special import expit
    z = np.linspace(-30, 30, 301)
    assert np.allclose(T.silu(z), z * expit(z), rtol=1e-14, atol=1e-300)
    assert np.allclose(T.silu(z), torch.nn.functional.silu(torch.tensor(z)).numpy(), rtol=1e-14, atol=1e-300)
    assert T.silu(np.array(0.0)) == 0.0


def test_argmax_lowest_index_and_margin():
    x = np.array([[1.0, 3.0, 3.0, -1.0], [5.0, 5.0, 5.0, 5.0], [0.0, -2.0, 0.5, 0.25]])
    assert T.argmax_lowest(x).tolist() == [1, 0, 2]
    assert np.allclose(T.top2_margin(x), [0.0, 0.0, 0.25])
    with pytest.raises(ValueError):
        T.argmax_lowest(np.array([1.0, np.nan]))


# ------------------------------------------------------------------------------------------
# Invariants of the whole model
# ------------------------------------------------------------------------------------------

def test_incremental_decode_equals_full_recompute():
    cfg = MICRO
    w = micro_weights()
    toks = np.random.default_rng(5).integers(0, cfg.vocab, size=8)
    om = T.OracleModel(cfg, w)
    steps = [om.prefill([toks[:5]])[0]] + [om.decode([t])[0] for t in toks[5:]]
    full = T.OracleModel(cfg, w).forward_full(toks)
    for i, lg in enumerate(steps):
        ref = full[4 + i]
        assert np.max(np.abs(lg - ref)) <= 1e-10 * np.max(np.abs(ref))


def test_chunked_prefill_equals_full_recompute():
    """Prefill chunks of two ragged sequences on populated caches give, at every chunk's
    last position, the logits of a fresh causal forward over the tokens so far."""
    cfg = MICRO
    w = micro_weights()
    rng = np.random.default_rng(6)
    seqs = [rng.integers(0, cfg.vocab, size=9), rng.integers(0, cfg.vocab, size=4)]
    cuts = [[3, 4, 9], [1, 2, 4]]   # chunk ends per sequence (a 1-token chunk included)
    om = T.OracleModel(cfg, w)
    got = [om.prefill([s_[:c[0]] for s_, c in zip(seqs, cuts)])]
    for i in (1, 2):
        got.append(om.extend([s_[c[i - 1]:c[i]] for s_, c in zip(seqs, cuts)]))
    for b, s_ in enumerate(seqs):
        full = T.OracleModel(cfg, w).forward_full(s_)
        for i, end in enumerate(cuts[b]):
            ref = full[end - 1]
            assert np.max(np.abs(got[i][b] - ref)) <= 1e-10 * np.max(np.abs(ref))
    assert om.lengths == [9, 4]


def test_gqa_equals_mha_with_repeated_kv():
    cfg = MICRO
    w = micro_weights()
    mha = cfg.replace(n_kv_heads=cfg.n_heads)
    w2 = dict(w)
    g = cfg.group
    for layer in range(cfg.n_layers):
        for name in ("wk", "wv"):
            W = w[f"layers.{layer}.{name}"].reshape(cfg.n_kv_heads, cfg.head_dim, cfg.d_model)
            w2[f"layers.{layer}.{name}"] = np.repeat(W, g, axis=0).reshape(-1, cfg.d_model)
    toks = np.random.default_rng(6).integers(0, cfg.vocab, size=7)
    a = T.OracleModel(cfg, w).forward_full(toks)
    b = T.OracleModel(mha, w2).forward_full(toks)
    assert np.max(np.abs(a - b)) < 1e-12


def test_causality():
    w = micro_weights()
    toks = np.random.default_rng(9).integers(0, MICRO.vocab, size=8)
    a = T.OracleModel(MICRO, w).forward_full(toks)
    toks2 = toks.copy()
    toks2[5] = (toks2[5] + 1) % MICRO.vocab
    b = T.OracleModel(MICRO, w).forward_full(toks2)
    assert np.array_equal(a[:5], b[:5])
    assert not np.allclose(a[5:], b[5:])


def test_batch_independence():
    w = micro_weights()
    rng = np.random.default_rng(10)
    prompts = [rng.integers(0, MICRO.vocab, size=n) for n in (5, 1, 3)]
    om = T.OracleModel(MICRO, w)
    batched = [om.prefill(prompts)] + [om.decode([1, 2, 3]), om.decode([4, 5, 6])]
    for b, p in enumerate(prompts):
        alone = T.OracleModel(MICRO, w)
        rows = [alone.prefill([p])[0], alone.decode([[1, 2, 3][b]])[0], alone.decode([[4, 5, 6][b]])[0]]
        for step in range(3):
            assert np.max(np.abs(batched[step][b] - rows[step])) < 1e-13


def test_teacher_forced_run_shapes():
    w = micro_weights()
    lens, toks = gen.prompt_tokens(MICRO)
    lg, tk = T.teacher_forced_run(T.OracleModel(MICRO, w), lens, toks, 3)
    assert lg.shape == (4, 2, MICRO.vocab) and tk.shape == (4, 2)
    assert np.array_equal(tk, np.argmax(lg, axis=-1))


# ------------------------------------------------------------------------------------------
# Sensitivity: plausible mistakes planted in the oracle must fail the library pin
# ------------------------------------------------------------------------------------------

def _rope_wrong_sign(x, positions, theta):
    x = np.asarray(x, dtype=np.float64)
    half = x.shape[-1] // 2
    ang = np.asarray(positions, dtype=np.float64)[:, None] * T.rope_frequencies(x.shape[-1], theta)[None]
    c, s = np.cos(ang)[:, None], np.sin(ang)[:, None]
    a, b = x[..., :half], x[..., half:]
    return np.concatenate([a * c + b * s, b * c - a * s], axis=-1)


def _rope_interleaved(x, positions, theta):
    x = np.asarray(x, dtype=np.float64)
    ang = np.asarray(positions, dtype=np.float64)[:, None] * T.rope_frequencies(x.shape[-1], theta)[None]
    c, s = np.cos(ang)[:, None], np.sin(ang)[:, None]
    a, b = x[..., 0::2], x[..., 1::2]
    out = np.empty_like(x)
    out[..., 0::2], out[..., 1::2] = a * c - b * s, b * c + a * s
    return out


def _rms_eps_outside(x, gain, eps):
    x = np.asarray(x, dtype=np.float64)
    return x / (np.sqrt(np.mean(x * x, axis=-1, keepdims=True)) + eps) * gain


def _attn_wrong_group(q, k, v, q_pos, k_pos):
    hkv = k.shape[1]
    kk = np.stack([k[:, h % hkv] for h in range(q.shape[1])], axis=1)
    vv = np.stack([v[:, h % hkv] for h in range(q.shape[1])], axis=1)
    return _ORIG_ATTN(q, kk, vv, q_pos, k_pos)


def _attn_no_scale(q, k, v, q_pos, k_pos):
    return _ORIG_ATTN(q * math.sqrt(q.shape[-1]), k, v, q_pos, k_pos)


def _silu_as_sigmoid(z):
    return 1.0 / (1.0 + np.exp(-z))


_ORIG_ATTN = T.causal_gqa_attention


@pytest.mark.parametrize("name,fn", [
    ("apply_rope", _rope_wrong_sign), ("apply_rope", _rope_interleaved),
    ("rmsnorm", _rms_eps_outside), ("causal_gqa_attention", _attn_wrong_group),
    ("causal_gqa_attention", _attn_no_scale), ("silu", _silu_as_sigmoid),
])
def test_planted_mistake_is_caught(monkeypatch, name, fn):
    cfg = MICRO.replace(rms_eps=0.5) if name == "rmsnorm" else MICRO
    w = micro_weights(cfg)
    toks = np.random.default_rng(7).integers(0, cfg.vocab, size=9)
    with torch.no_grad():
        ref = hf_model(cfg, w)(torch.tensor(toks[None])).logits[0].numpy()
    monkeypatch.setattr(T, name, fn)
    bad = T.OracleModel(cfg, w).forward_full(toks)
    assert _rel_err(bad, ref) > 1e-3


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(11)
    x = np.concatenate([rng.standard_normal(100000).astype(np.float32) * 0.02,
                        np.array([1.00390625, 1.01171875, -3.0e-39, 65504.0, 0.0, -0.0], np.float32)])
    ours = gen.bf16_bits(gen.round_to_bf16(x))
    ref = torch.tensor(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)


def test_generator_is_deterministic():
    cfg = MICRO
    a, b = gen.weights(cfg), gen.weights(cfg)
    assert all(np.array_equal(a[k], b[k]) for k in a)
    l1, t1 = gen.prompt_tokens(cfg)
    l2, t2 = gen.prompt_tokens(cfg)
    assert l1 == l2 and np.array_equal(t1, t2)
    from synth.configs import CONFIGS
    lens = gen.prompt_lengths(CONFIGS["8b-gqa"])
    assert len(lens) == 32 and min(lens) >= 1024 and max(lens) <= 4096
