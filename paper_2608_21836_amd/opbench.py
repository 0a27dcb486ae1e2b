"""Microbenchmark of the per-kernel entry points (include/ll_ops.h) at the workload shapes.

The paper qualifies a kernel in isolation before accepting it inside the model (Sec. 2.2);
this module times each hot-path kernel alone, on the shapes the five workloads run:
  gemm        prefill GEMM (ll_op_gemm path 0), M = the workload's prompt tokens; the
              gate/up shape also with its SwiGLU epilogue (ll_op_gemm_swiglu)
  gemv        decode GEMM, whole-K (ll_op_gemm path 1) and split-K (ll_op_gemm_splitk),
              M = the workload's batch; weights rotate over >= 1 GiB so they stream from HBM
  attn        prefill attention (ll_op_attn_prefill) and decode attention (ll_op_attn_decode)
  vendor      the vendor library's bf16 GEMM (torch.matmul, i.e. hipBLASLt) on the prefill GEMM
              shapes: a reference for what this GPU reaches on the same products, not part of the
              path
Each line: kernel, workload, shape, mean time per call, achieved rate and the fraction of the
MI355X peak (HBM 8 TB/s; fp16 / bf16 MFMA 2.5 PFLOP/s).  Operands are fp16, as the decoder
runs bf16 weights by default (--bf16 for bf16 operands).  Inputs are random; only timing
matters here (numerics are covered by tests/test_kernels_gpu.py).

  python -m paper_2608_21836_amd.opbench [--only gemm,gemv,attn] [--workloads 7b-mha,8b-gqa]
"""
from __future__ import annotations

import argparse
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK = 8.0e12
DT = None   # operand type (torch.float16 or torch.bfloat16), set in main
MFMA_PEAK = 2.5e15


def _timeit(fn, iters: int) -> float:
    """Mean microseconds per call over `iters` calls after 2 warm-up calls."""
    import torch
    for i in range(2):
        fn(i)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(iters):
        fn(i)
    e1.record()
    e1.synchronize()
    return e0.elapsed_time(e1) * 1e3 / iters


def _line(kind, wl, shape, us, work, unit):
    if unit == "flop":
        rate, frac, u = work / us * 1e-6, work / (us * 1e-6) / MFMA_PEAK, "TFLOP/s"
    else:
        rate, frac, u = work / us * 1e-6, work / (us * 1e-6) / HBM_PEAK, "TB/s"
    print(f"{kind:22s} {wl:8s} {shape:34s} {us:10.1f} us {rate:8.2f} {u:8s} {100 * frac:5.1f} %",
          flush=True)


def linear_shapes(cfg):
    nqkv = cfg.q_dim + 2 * cfg.kv_dim
    return [("qkv", nqkv, cfg.d_model), ("o", cfg.d_model, cfg.q_dim),
            ("gate_up", 2 * cfg.ffn_dim, cfg.d_model), ("down", cfg.d_model, cfg.ffn_dim)]


def bench_gemm(cfg, lens, iters):
    import torch
    from paper_2608_21836_amd.binding import op_gemm, op_gemm_swiglu, op_repack
    T = int(sum(lens))
    a = (torch.randn(T, max(k for _, _, k in linear_shapes(cfg)), device="cuda") * 0.5).to(DT)
    for name, n, k in linear_shapes(cfg):
        ak = a[:, :k].contiguous()
        wt = op_repack((torch.randn(n, k, device="cuda") * 0.02).to(DT))
        c = torch.empty(T, n, device="cuda")
        us = _timeit(lambda i: op_gemm(0, ak, wt, n, c=c), iters)
        _line("prefill_gemm", cfg.name, f"{name} M={T} N={n} K={k}", us, 2.0 * T * n * k, "flop")
        if name == "gate_up":   # the workload's own epilogue: SwiGLU, act [M, F] in bf16
            act = torch.empty(T, n // 2, dtype=DT, device="cuda")
            us = _timeit(lambda i: op_gemm_swiglu(ak, wt, n, act=act), iters)
            _line("prefill_gemm_swiglu", cfg.name, f"{name} M={T} N={n} K={k}", us,
                  2.0 * T * n * k, "flop")
            del act
        del ak, wt, c
        torch.cuda.empty_cache()


def bench_gemv(cfg, batch, iters):
    import torch
    from paper_2608_21836_amd.binding import load_library, op_gemm, op_gemm_splitk, op_repack
    lib = load_library()
    for name, n, k in linear_shapes(cfg):
        wbytes = n * k * 2
        reps = max(2, min(64, (1 << 30) // wbytes + 1))
        wts = [op_repack((torch.randn(n, k, device="cuda") * 0.02).to(DT)) for _ in range(reps)]
        a = torch.randn(batch, k, device="cuda").to(DT)
        c = torch.zeros(batch, n, device="cuda")
        work = wbytes + batch * k * 2 + 2 * batch * n * 4
        us = _timeit(lambda i: op_gemm(1, a, wts[i % reps], n, c=c, accumulate=True), 3 * reps)
        _line("decode_gemm_wholek", cfg.name, f"{name} M={batch} N={n} K={k}", us, work, "byte")
        if lib.ll_op_gemm_splitk_scratch(1, batch, n, k):
            us = _timeit(lambda i: op_gemm_splitk(a, wts[i % reps], n, c=c, accumulate=True), 3 * reps)
            _line("decode_gemm_splitk", cfg.name, f"{name} M={batch} N={n} K={k}", us, work, "byte")
        del wts
        torch.cuda.empty_cache()


def bench_vendor(cfg, lens, iters):
    import torch
    M = int(sum(lens))
    for name, n, k in linear_shapes(cfg):
        a = torch.randn(M, k, device="cuda").to(DT)
        w = torch.randn(n, k, device="cuda").to(DT)
        us = _timeit(lambda i: torch.matmul(a, w.t()), iters)
        _line("vendor_gemm", cfg.name, f"{name} M={M} N={n} K={k}", us, 2.0 * M * n * k, "flop")
        del a, w
        torch.cuda.empty_cache()


def bench_attn(cfg, lens, n_decode, iters):
    import torch
    from paper_2608_21836_amd.binding import op_attn_decode, op_attn_prefill
    B, T, hd = len(lens), int(sum(lens)), cfg.head_dim
    max_ctx = max(lens) + n_decode
    q = torch.randn(T, cfg.q_dim, device="cuda").to(DT)
    kc = torch.randn(B, cfg.n_kv_heads, max_ctx, hd, device="cuda").to(DT)
    vc = torch.randn(B, cfg.n_kv_heads, max_ctx, hd, device="cuda").to(DT)
    us = _timeit(lambda i: op_attn_prefill(lens, q, kc, vc, cfg.n_heads, cfg.n_kv_heads, hd, max_ctx),
                 iters)
    flops = 2.0 * hd * cfg.n_heads * sum(x * (x + 1) for x in lens)
    _line("prefill_attention", cfg.name, f"B={B} T={T} H={cfg.n_heads}/{cfg.n_kv_heads}x{hd}", us,
          flops, "flop")
    ctx = torch.tensor([x + n_decode // 2 for x in lens], dtype=torch.int32, device="cuda")
    qd = torch.randn(B, cfg.q_dim, device="cuda").to(DT)
    us = _timeit(lambda i: op_attn_decode(qd, kc, vc, ctx, cfg.n_heads, cfg.n_kv_heads, hd, max_ctx),
                 iters * 10)
    kv = sum(x + n_decode // 2 for x in lens) * 2 * cfg.kv_dim * 2 + B * cfg.q_dim * 2
    _line("decode_attention", cfg.name, f"B={B} ctx~{max(lens) + n_decode // 2} H={cfg.n_heads}/{cfg.n_kv_heads}x{hd}",
          us, kv, "byte")


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--only", default="gemm,gemv,attn")
    ap.add_argument("--workloads", default="1b-gqa,7b-mha,8b-gqa")
    ap.add_argument("--iters", type=int, default=5)
    ap.add_argument("--bf16", action="store_true", help="bf16 operands instead of fp16")
    args = ap.parse_args()
    import torch
    global DT
    DT = torch.bfloat16 if args.bf16 else torch.float16
    from synth import gen, get_config
    kinds = set(args.only.split(","))
    torch.cuda.set_device(0)
    for wl in args.workloads.split(","):
        cfg = get_config(wl)
        if cfg.dtype != "bf16":
            continue
        lens = [int(x) for x in gen.prompt_lengths(cfg)]
        if "gemm" in kinds:
            bench_gemm(cfg, lens, args.iters)
        if "gemv" in kinds:
            bench_gemv(cfg, len(lens), args.iters)
        if "attn" in kinds:
            bench_attn(cfg, lens, cfg.n_decode, args.iters)
        if "vendor" in kinds:
            bench_vendor(cfg, lens, args.iters)
    return 0


if __name__ == "__main__":
    sys.exit(main())
