"""Isolated qualification of each hot-path kernel through the per-kernel C entry points
(include/ll_ops.h), against the oracle's per-op functions on the same rounded inputs.

Floating-point bounds (derived from the arithmetic, not tuned):
  * GEMM with fp32 accumulation of exact products: |c - c64| <= 4 K u (|A| |W|^T), u = 2^-24
    (a-priori dot-product bound, any summation order).
  * RMSNorm: bf16 output rounding 2^-9 |y| plus fp32 noise -> 2^-8 |y| + 1e-6; fp32 1e-5 |y|.
  * Attention, bf16: P is rounded to bf16 (2^-9 relative) before the PV product and the
    output is rounded to bf16: |o - o64| <= 4 * 2^-9 * max|v|.  fp32: 1e-5 * max|v|.
"""
import numpy as np
import pytest

import oracle
from parity import device_tensor, log, rounded

pytestmark = pytest.mark.gpu

U = 2.0 ** -24


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_21836_amd.binding import load_library
    load_library()


def _np(t):
    import torch
    return t.float().cpu().numpy() if t.dtype == torch.bfloat16 else t.cpu().numpy()


@pytest.mark.parametrize("dtype", ["bf16", "f16", "f32"])
@pytest.mark.parametrize("rows,d", [(1, 256), (5, 768), (3, 4096)])
def test_rmsnorm(dtype, rows, d):
    from paper_2608_21836_amd.binding import op_rmsnorm
    import torch
    log(f"rmsnorm {dtype} rows={rows} d={d}")
    rng = np.random.default_rng(rows * 7 + d)
    x = (rng.standard_normal((rows, d)) * 3).astype(np.float32)
    g = rounded(1 + 0.1 * rng.standard_normal(d), dtype)
    y = op_rmsnorm(torch.from_numpy(x).cuda(), device_tensor(g, dtype), 1e-5)
    torch.cuda.synchronize()
    ref = oracle.rmsnorm(x, g, 1e-5)
    rel = {"bf16": 2.0 ** -8, "f16": 2.0 ** -11, "f32": 1e-5}[dtype]
    tol = rel * np.abs(ref) + (1e-6 if dtype != "f32" else 1e-7)
    assert np.all(np.abs(_np(y) - ref) <= tol)


GEMM_SHAPES = [
    # 64 x 128 tiles (short prompts), with M tails
    (0, 1, 256, 64), (0, 130, 384, 768), (0, 300, 128, 192), (0, 257, 256, 1408),
    (0, 512, 2304, 768),
    # enough 256 x 256 tiles for the large-tile kernel, with ragged M tails
    (0, 2000, 6144, 256), (0, 3000, 4096, 1024), (0, 6144, 2048, 128),
    # 128 x 256 tiles (too few 256 x 256 tiles), exact and ragged M
    (0, 2048, 4096, 512), (0, 1530, 4096, 256),
    (1, 1, 32, 64), (1, 1, 256, 768), (1, 15, 96, 192), (1, 16, 256, 512), (1, 17, 64, 64),
    (1, 32, 128, 4096), (1, 33, 64, 256), (1, 70, 96, 128),
]


@pytest.mark.parametrize("dtype", ["bf16", "f16", "f32"])
@pytest.mark.parametrize("path,m,n,k", GEMM_SHAPES)
def test_gemm(dtype, path, m, n, k):
    from paper_2608_21836_amd.binding import op_gemm, op_repack
    import torch
    log(f"gemm path={path} {dtype} m={m} n={n} k={k}")
    rng = np.random.default_rng(m * 1000 + n + k)
    a = rounded(rng.standard_normal((m, k)), dtype)
    w = rounded(rng.standard_normal((n, k)) * 0.05, dtype)
    c0 = rng.standard_normal((m, n)).astype(np.float32)
    A, W = device_tensor(a, dtype), device_tensor(w, dtype)
    wt = op_repack(W)
    c = op_gemm(path, A, wt, n)
    cacc = op_gemm(path, A, wt, n, c=torch.from_numpy(c0).cuda(), accumulate=True)
    torch.cuda.synchronize()
    ref = a.astype(np.float64) @ w.astype(np.float64).T
    bound = 4 * k * U * (np.abs(a).astype(np.float64) @ np.abs(w).astype(np.float64).T) + 1e-30
    assert np.all(np.abs(_np(c) - ref) <= bound)
    assert np.all(np.abs(_np(cacc) - (ref + c0)) <= bound + 2 * U * np.abs(ref + c0))


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("m,n,k", [(300, 1024, 512), (4100, 2048, 256), (64, 256, 1024)])
def test_gemm_swiglu(dtype, m, n, k):
    """The prefill GEMM with the SwiGLU epilogue against silu(a W_g^T) * (a W_u^T) in fp64,
    under the dot-product bound plus the rounding of the output and of silu's inputs."""
    from paper_2608_21836_amd.binding import op_gemm_swiglu, op_repack
    import torch
    log(f"gemm swiglu {dtype} m={m} n={n} k={k}")
    rng = np.random.default_rng(m + n + k)
    f = n // 2
    a = rounded(rng.standard_normal((m, k)), dtype)
    wg = rounded(rng.standard_normal((f, k)) * 0.05, dtype)
    wu = rounded(rng.standard_normal((f, k)) * 0.05, dtype)
    # rows interleaved in blocks of 16: gate 16 u .., then up 16 u .., per 32-row unit
    w = np.empty((n, k), dtype=np.float32)
    for u in range(f // 16):
        w[32 * u:32 * u + 16] = wg[16 * u:16 * u + 16]
        w[32 * u + 16:32 * u + 32] = wu[16 * u:16 * u + 16]
    act = op_gemm_swiglu(device_tensor(a, dtype), op_repack(device_tensor(w, dtype)), n)
    torch.cuda.synchronize()
    a64 = a.astype(np.float64)
    g, up = a64 @ wg.astype(np.float64).T, a64 @ wu.astype(np.float64).T
    ref = g / (1.0 + np.exp(-g)) * up
    bg = 4 * k * U * (np.abs(a64) @ np.abs(wg.astype(np.float64)).T)
    bu = 4 * k * U * (np.abs(a64) @ np.abs(wu.astype(np.float64)).T)
    # d(silu)/dg <= 1.1; the output's own rounding (bf16: 8-bit significand, 2^-8 relative)
    out_u = 2.0 ** -8 if dtype == "bf16" else 2.0 ** -23
    bound = 1.1 * bg * np.abs(up) + np.abs(g) * bu + (out_u + 4e-6) * np.abs(ref) + 1e-30
    assert np.all(np.abs(_np(act).astype(np.float64) - ref) <= bound)


SPLITK_SHAPES = [(17, 128, 64), (32, 512, 256), (32, 4096, 1024), (33, 384, 4096),
                 (64, 256, 14336), (20, 6144, 512),
                 # every compiled slice length: 64 (8B gate/up), 56 (8B down), 32, 40, 48
                 (32, 16384, 4096), (32, 4096, 14336), (32, 4096, 8192), (32, 4096, 10240),
                 (32, 4096, 12288)]


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("m,n,k", SPLITK_SHAPES)
def test_gemm_splitk(dtype, m, n, k):
    from paper_2608_21836_amd.binding import op_gemm_splitk, op_repack
    import torch
    log(f"gemm split-K {dtype} m={m} n={n} k={k}")
    rng = np.random.default_rng(m * 7 + n + k)
    a = rounded(rng.standard_normal((m, k)), dtype)
    w = rounded(rng.standard_normal((n, k)) * 0.05, dtype)
    c0 = rng.standard_normal((m, n)).astype(np.float32)
    A, W = device_tensor(a, dtype), device_tensor(w, dtype)
    wt = op_repack(W)
    c = op_gemm_splitk(A, wt, n)
    cacc = op_gemm_splitk(A, wt, n, c=torch.from_numpy(c0).cuda(), accumulate=True)
    torch.cuda.synchronize()
    ref = a.astype(np.float64) @ w.astype(np.float64).T
    bound = 4 * k * U * (np.abs(a).astype(np.float64) @ np.abs(w).astype(np.float64).T) + 1e-30
    assert np.all(np.abs(_np(c) - ref) <= bound)
    assert np.all(np.abs(_np(cacc) - (ref + c0)) <= bound + 2 * U * np.abs(ref + c0))


# Short prompts: too few 64 x 128 output tiles to fill the CUs, so K is split over blocks
# (125m O and down projections at 512 tokens, ragged row counts, a single row).
PREFILL_SPLITK_SHAPES = [(512, 768, 2048), (512, 768, 768), (300, 768, 768), (200, 1280, 512),
                         (1, 256, 1024), (77, 1024, 4096)]


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("m,n,k", PREFILL_SPLITK_SHAPES)
def test_gemm_prefill_splitk(dtype, m, n, k):
    from paper_2608_21836_amd.binding import load_library, op_gemm_prefill_splitk, op_repack
    import torch
    log(f"gemm prefill split-K {dtype} m={m} n={n} k={k}")
    assert load_library().ll_op_gemm_prefill_splitk_scratch(1 if dtype == "bf16" else 0, m, n, k) > 0
    rng = np.random.default_rng(m * 11 + n + k)
    a = rounded(rng.standard_normal((m, k)), dtype)
    w = rounded(rng.standard_normal((n, k)) * 0.05, dtype)
    c0 = rng.standard_normal((m, n)).astype(np.float32)
    A, W = device_tensor(a, dtype), device_tensor(w, dtype)
    wt = op_repack(W)
    c = op_gemm_prefill_splitk(A, wt, n)
    cacc = op_gemm_prefill_splitk(A, wt, n, c=torch.from_numpy(c0).cuda(), accumulate=True)
    torch.cuda.synchronize()
    ref = a.astype(np.float64) @ w.astype(np.float64).T
    bound = 4 * k * U * (np.abs(a).astype(np.float64) @ np.abs(w).astype(np.float64).T) + 1e-30
    assert np.all(np.abs(_np(c) - ref) <= bound)
    assert np.all(np.abs(_np(cacc) - (ref + c0)) <= bound + 2 * U * np.abs(ref + c0))


def _caches(rng, dtype, batch, hkv, max_ctx, hd, lens):
    """Random caches with every position at or beyond a sequence's length set to NaN, so a
    read of a stale or out-of-range entry poisons the output."""
    k = rounded(rng.standard_normal((batch, hkv, max_ctx, hd)), dtype)
    v = rounded(rng.standard_normal((batch, hkv, max_ctx, hd)), dtype)
    for b, n in enumerate(lens):
        k[b, :, n:] = np.nan
        v[b, :, n:] = np.nan
    return k, v


# P and the output are rounded to the operand type: bf16 8-bit, fp16 11-bit significands
ATTN_TOL = {"bf16": 4 * 2.0 ** -9, "f16": 4 * 2.0 ** -11, "f32": 1e-5}

ATTN_CASES = [
    ("bf16", 64, 8, 2, [1, 63, 64, 65, 200]),
    ("bf16", 128, 4, 1, [130, 7]),
    ("bf16", 128, 8, 8, [96]),
    # several 128-query tiles and 64-key tiles, ragged tails, GQA groups of 4
    ("bf16", 128, 8, 2, [300, 129, 1, 257]),
    ("bf16", 128, 4, 4, [1030]),
    ("bf16", 64, 4, 1, [513, 128, 127]),
    # grouped-query kernel (one block per query tile and KV head) at every group size: groups
    # of 8 at head_dim 64 (32-query tiles), of 4 at 128 (64-query tiles), of 2 (128-query
    # tiles); many ragged sequences so that the work list is cut over the XCDs mid-sequence
    ("bf16", 64, 32, 4, [1024, 77, 1, 33]),
    ("bf16", 64, 16, 2, [300, 31, 32, 257]),
    ("bf16", 128, 32, 8, [1500, 1, 700, 64]),
    ("bf16", 128, 8, 4, [129, 255, 2]),
    ("bf16", 128, 16, 4, [int(x) for x in np.random.default_rng(7).integers(1, 600, 20)]),
    # fp16 operands (a bf16 model with f16_compute): both kernels
    ("f16", 128, 32, 8, [1500, 1, 700, 64]),
    ("f16", 64, 32, 4, [1024, 77, 1, 33]),
    ("f16", 128, 4, 4, [1030]),
    ("f32", 64, 4, 4, [33, 1, 128]),
    ("f32", 128, 4, 2, [70]),
]


@pytest.mark.parametrize("dtype,hd,hq,hkv,lens", ATTN_CASES)
def test_attn_prefill(dtype, hd, hq, hkv, lens):
    from paper_2608_21836_amd.binding import op_attn_prefill
    import torch
    log(f"attn_prefill {dtype} hd={hd} hq={hq} hkv={hkv} lens={lens}")
    rng = np.random.default_rng(hd + hq * 10 + len(lens))
    B, T, max_ctx = len(lens), sum(lens), max(lens) + 3
    q = rounded(rng.standard_normal((T, hq * hd)), dtype)
    k, v = _caches(rng, dtype, B, hkv, max_ctx, hd, lens)
    o = op_attn_prefill(lens, device_tensor(q, dtype), device_tensor(k, dtype),
                        device_tensor(v, dtype), hq, hkv, hd, max_ctx)
    torch.cuda.synchronize()
    o = _np(o)
    t0 = 0
    for b, L in enumerate(lens):
        qb = q[t0:t0 + L].reshape(L, hq, hd).astype(np.float64)
        kb = k[b, :, :L].transpose(1, 0, 2).astype(np.float64)
        vb = v[b, :, :L].transpose(1, 0, 2).astype(np.float64)
        pos = np.arange(L)
        ref = oracle.causal_gqa_attention(qb, kb, vb, pos, pos).reshape(L, hq * hd)
        tol = ATTN_TOL[dtype] * np.abs(vb).max()
        assert np.all(np.abs(o[t0:t0 + L] - ref) <= tol), f"sequence {b}"
        t0 += L


# Prefill chunks on populated caches: (dtype, hd, hq, hkv, new tokens, cached keys) per
# sequence; query i of sequence b sits at position cached[b] + i.
CHUNK_CASES = [
    ("bf16", 64, 8, 2, [1, 63, 64, 130], [100, 1, 64, 0]),
    ("bf16", 128, 32, 8, [200, 17], [1000, 63]),
    ("bf16", 64, 4, 4, [128], [512]),
    ("bf16", 64, 32, 4, [40, 1, 300], [1000, 5, 64]),
    ("bf16", 128, 32, 8, [65, 128], [63, 2000]),
    ("f16", 128, 32, 8, [65, 128], [63, 2000]),
    ("f32", 64, 4, 4, [33, 1, 70], [31, 200, 64]),
    ("f32", 128, 4, 2, [65], [3]),
]


@pytest.mark.parametrize("dtype,hd,hq,hkv,lens,cached", CHUNK_CASES)
def test_attn_prefill_chunk(dtype, hd, hq, hkv, lens, cached):
    from paper_2608_21836_amd.binding import op_attn_prefill
    import torch
    log(f"attn_prefill chunk {dtype} hd={hd} hq={hq} hkv={hkv} lens={lens} cached={cached}")
    rng = np.random.default_rng(hd + hq * 10 + sum(cached))
    B, T = len(lens), sum(lens)
    tot = [c + n for c, n in zip(cached, lens)]
    max_ctx = max(tot) + 5
    q = rounded(rng.standard_normal((T, hq * hd)), dtype)
    k, v = _caches(rng, dtype, B, hkv, max_ctx, hd, tot)
    o = op_attn_prefill(lens, device_tensor(q, dtype), device_tensor(k, dtype),
                        device_tensor(v, dtype), hq, hkv, hd, max_ctx, cached=cached)
    torch.cuda.synchronize()
    o = _np(o)
    t0 = 0
    for b, L in enumerate(lens):
        P0 = cached[b]
        qb = q[t0:t0 + L].reshape(L, hq, hd).astype(np.float64)
        kb = k[b, :, :P0 + L].transpose(1, 0, 2).astype(np.float64)
        vb = v[b, :, :P0 + L].transpose(1, 0, 2).astype(np.float64)
        ref = oracle.causal_gqa_attention(qb, kb, vb, P0 + np.arange(L), np.arange(P0 + L))
        ref = ref.reshape(L, hq * hd)
        tol = ATTN_TOL[dtype] * np.abs(vb).max()
        assert np.all(np.abs(o[t0:t0 + L] - ref) <= tol), f"sequence {b}"
        t0 += L


DEC_CASES = [
    ("bf16", 64, 8, 2, [1, 63, 64, 65, 257, 1000], 1024),
    ("bf16", 128, 32, 8, [4096, 17, 2049], 4224),
    ("bf16", 128, 16, 2, [300], 512),
    ("f16", 128, 32, 8, [4096, 17, 2049], 4224),
    ("bf16", 64, 4, 4, [5, 640], 640),
    ("f32", 64, 4, 4, [48, 2], 48),
    ("f32", 128, 4, 1, [129], 200),
]


@pytest.mark.parametrize("dtype,hd,hq,hkv,lens,max_ctx", DEC_CASES)
def test_attn_decode(dtype, hd, hq, hkv, lens, max_ctx):
    from paper_2608_21836_amd.binding import op_attn_decode
    import torch
    log(f"attn_decode {dtype} hd={hd} hq={hq} hkv={hkv} lens={lens} max_ctx={max_ctx}")
    rng = np.random.default_rng(hd + hq + max_ctx)
    B = len(lens)
    q = rounded(rng.standard_normal((B, hq * hd)), dtype)
    k, v = _caches(rng, dtype, B, hkv, max_ctx, hd, lens)
    ctx = torch.tensor(lens, dtype=torch.int32, device="cuda")
    o = op_attn_decode(device_tensor(q, dtype), device_tensor(k, dtype), device_tensor(v, dtype),
                       ctx, hq, hkv, hd, max_ctx)
    torch.cuda.synchronize()
    o = _np(o)
    for b, L in enumerate(lens):
        qb = q[b].reshape(1, hq, hd).astype(np.float64)
        kb = k[b, :, :L].transpose(1, 0, 2).astype(np.float64)
        vb = v[b, :, :L].transpose(1, 0, 2).astype(np.float64)
        ref = oracle.causal_gqa_attention(qb, kb, vb, np.array([L - 1]), np.arange(L)).reshape(-1)
        tol = ATTN_TOL[dtype] / 2 * np.abs(vb).max()
        assert np.all(np.abs(o[b] - ref) <= tol), f"sequence {b}"


@pytest.mark.parametrize("dtype", ["bf16", "f16", "f32"])
@pytest.mark.parametrize("rows,vocab,k", [(1, 1024, 256), (3, 4096, 768), (33, 32000, 512)])
def test_lmhead_argmax(dtype, rows, vocab, k):
    from paper_2608_21836_amd.binding import op_lmhead_argmax, op_repack
    import torch
    log(f"lmhead_argmax {dtype} rows={rows} vocab={vocab} k={k}")
    rng = np.random.default_rng(rows + vocab + k)
    h = rounded(rng.standard_normal((rows, k)), dtype)
    w = rng.standard_normal((vocab, k)) * 0.02
    # planted exact tie at the top for row 0: two identical weight rows aligned with h[0]
    w[vocab // 3] = w[vocab - 5] = h[0] / np.linalg.norm(h[0])
    w = rounded(w, dtype)
    wt = op_repack(device_tensor(w, dtype))
    nxt, logits = op_lmhead_argmax(device_tensor(h, dtype), wt, vocab)
    nxt2, none = op_lmhead_argmax(device_tensor(h, dtype), wt, vocab, want_logits=False)
    torch.cuda.synchronize()
    lg = logits.cpu().numpy()
    ref = h.astype(np.float64) @ w.astype(np.float64).T
    bound = 4 * k * U * (np.abs(h).astype(np.float64) @ np.abs(w).astype(np.float64).T) + 1e-30
    assert np.all(np.abs(lg - ref) <= bound)
    assert np.array_equal(nxt.cpu().numpy(), np.argmax(lg, axis=-1))
    assert np.array_equal(nxt.cpu().numpy(), nxt2.cpu().numpy())
    assert nxt.cpu().numpy()[0] == vocab // 3


def test_mfma_calibration_loop_runs():
    """The calibration loop (ll_op_mfma_loop) fills its output and rejects bad arguments."""
    import torch
    from paper_2608_21836_amd.binding import LLError, op_mfma_loop
    out = op_mfma_loop(8, 4)
    torch.cuda.synchronize()
    assert out.shape == (32,) and torch.isfinite(out).all()
    with pytest.raises(LLError):
        op_mfma_loop(0, 4)


@pytest.mark.parametrize("n,blocks", [(0, 4), (12, 3), ((1 << 20) + 12, 64), ((1 << 22) + 4, 2048)])
def test_read_stream_calibration_sums_everything_once(n, blocks):
    """The read-stream calibration (ll_op_read_stream) reads every element exactly once: with
    small integers the per-block sums are exact in fp32, so their total equals the buffer's
    sum (the tail past the unrolled rounds included); bad arguments are rejected."""
    import torch
    from paper_2608_21836_amd.binding import LLError, op_read_stream
    src = (torch.arange(n, device="cuda", dtype=torch.int64) % 3).to(torch.float32)
    out = op_read_stream(src, blocks)
    torch.cuda.synchronize()
    assert out.shape == (blocks,)
    assert int(out.double().sum().item()) == int(src.double().sum().item())
    with pytest.raises(LLError):
        op_read_stream(src[:2] if n else torch.empty(2, device="cuda"), blocks)   # n % 4 != 0
    with pytest.raises(LLError):
        op_read_stream(src, 0)
