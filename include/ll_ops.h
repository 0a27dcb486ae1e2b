/*
 * ll_ops.h -- per-kernel entry points of the hot path, for isolated qualification.
 *
 * The paper separates isolated qualification of a kernel (numerical correctness in a
 * standalone harness) from deployment-time acceptance inside the model (Sec. 2.2
 * "Formulation and Implications", first and third evaluation stages).  These calls run the
 * same kernels that ll_prefill / ll_decode_step use, one at a time, so that each can be
 * checked on its own; the model-level calls in ll.h are the acceptance path.
 *
 * All pointers are DEVICE pointers unless named *_host.  Element type "T" is float for
 * LL_F32 and bfloat16 for LL_BF16.  Every call validates sizes first (no enqueue on error),
 * enqueues on `stream` (hipStream_t, NULL = default) and returns without synchronising.
 * The library allocates nothing: a call that needs scratch takes it from the caller.
 */
#ifndef LL_OPS_H
#define LL_OPS_H

#include "ll.h"

#ifdef __cplusplus
extern "C" {
#endif

/* y[r, :] = x[r, :] / sqrt(mean(x[r, :]^2) + eps) * gain   (Sec. 3 model block; RMSNorm).
 * x fp32 [rows, d] row-major, gain T [d], y T [rows, d].  d a multiple of 4. */
ll_status ll_op_rmsnorm(int32_t dtype, int32_t rows, int32_t d, const float *x,
                        const void *gain, float eps, void *y, void *stream);

/* Repack a row-major weight W (T [N, K]) into the tiled layout both GEMM paths stream:
 * 16-row x (32 bf16 | 16 fp32)-column tiles of 1 KiB, each laid out in MFMA operand
 * order, tiles of one 16-row block contiguous along K.  wt must hold N*K*sizeof(T) bytes.
 * N a multiple of 16, K a multiple of 64. */
ll_status ll_op_repack(int32_t dtype, int32_t n, int32_t k, const void *w, void *wt,
                       void *stream);

/* C[M, N] = A[M, K] W^T (accumulate = 0) or C += A W^T (accumulate = 1).
 * A T row-major (lda = K), wt = repacked W, C fp32 row-major (ldc = N).
 * path 0: prefill GEMM (LDS-tiled MFMA, N a multiple of 128);
 * path 1: decode GEMM (weight-streaming MFMA, N a multiple of 32, any M). */
ll_status ll_op_gemm(int32_t path, int32_t dtype, int32_t m, int32_t n, int32_t k,
                     const void *a, const void *wt, float *c, int32_t accumulate, void *stream);

/* The prefill GEMM with the gate/up projection's SwiGLU epilogue: act[m, 16 u + c] =
 * silu(g) * v, where g and v are columns 32 u + c and 32 u + 16 + c (c < 16) of A W^T, i.e. W
 * holds the gate and up rows interleaved in blocks of 16 (gate rows 16 u .. 16 u + 15, then
 * up rows 16 u .. 16 u + 15, for u = 0 .. n / 32 - 1) before ll_op_repack.  A T row-major
 * (lda = K), act T row-major [M, N/2].  N a multiple of 128, K a multiple of 64. */
ll_status ll_op_gemm_swiglu(int32_t dtype, int32_t m, int32_t n, int32_t k, const void *a,
                            const void *wt, void *act, void *stream);

/* Decode GEMM for batches above 16 rows, split over K: C = A W^T (accumulate = 0) or
 * C += A W^T.  Each block of 128 output columns covers a slice of K and stages its slice of
 * A in LDS once for all its columns; fp32 partial sums go to `scratch`, and a second kernel
 * adds them in split order and writes C.  Same A / wt / C layouts as ll_op_gemm.  Requires
 * m > 16, n a multiple of 128, k a multiple of 64, and scratch >= ll_op_gemm_splitk_scratch
 * bytes (LL_ERR_UNSUPPORTED / LL_ERR_WORKSPACE otherwise). */
ll_status ll_op_gemm_splitk(int32_t dtype, int32_t m, int32_t n, int32_t k, const void *a,
                            const void *wt, float *c, int32_t accumulate, void *scratch,
                            size_t scratch_bytes, void *stream);
/* Scratch bytes ll_op_gemm_splitk needs for this shape; 0 if the shape is not supported. */
size_t ll_op_gemm_splitk_scratch(int32_t dtype, int32_t m, int32_t n, int32_t k);

/* Prefill GEMM for prompts too short to fill the GPU with 64 x 128 output tiles, split over
 * K: each block covers a range of K, fp32 partial sums go to `scratch`, and a second kernel
 * adds them in split order and writes C = A W^T (accumulate = 0) or C += A W^T.  Same A / wt /
 * C layouts as ll_op_gemm.  Requires a shape that ll_op_gemm_prefill_splitk_scratch accepts
 * (non-zero: n a multiple of 128, k a multiple of 64, fewer than 96 tiles of 64 x 128) and
 * scratch of at least that many bytes (LL_ERR_UNSUPPORTED / LL_ERR_WORKSPACE otherwise). */
ll_status ll_op_gemm_prefill_splitk(int32_t dtype, int32_t m, int32_t n, int32_t k,
                                    const void *a, const void *wt, float *c, int32_t accumulate,
                                    void *scratch, size_t scratch_bytes, void *stream);
/* Scratch bytes ll_op_gemm_prefill_splitk needs for this shape; 0 if it does not split it. */
size_t ll_op_gemm_prefill_splitk_scratch(int32_t dtype, int32_t m, int32_t n, int32_t k);

/* Causal grouped-query prefill attention over packed ragged sequences (appendix
 * "Deployment Kernel Families", Table A.4: programs over query tiles, KV head from the head
 * grouping with KV loads shared by the heads of a group, causal mask in the score update,
 * fp32 online-softmax statistics).  bf16 with n_heads / n_kv_heads >= 2: one block per (query
 * tile, KV head) covering the whole head group; otherwise one block per (query tile, head).
 * q T [sum(seq_lens), n_heads*head_dim]; kcache/vcache T [batch][n_kv_heads][max_ctx]
 * [head_dim]; o T like q.  Sequence b's queries sit at positions cached_host[b] ..
 * cached_host[b] + seq_lens[b] - 1 (cached_host nullable: all 0) and the cache holds its
 * positions 0 .. cached_host[b] + seq_lens[b] - 1; query i attends to positions
 * 0 .. cached_host[b] + i (a prefill chunk on a populated cache when cached_host[b] > 0).
 * scratch >= ll_op_attn_prefill_scratch(...) bytes (device metadata: offsets, positions and
 * the blocks' work list), 256-byte aligned; LL_ERR_WORKSPACE when smaller. */
ll_status ll_op_attn_prefill(int32_t dtype, int32_t batch, const int32_t *seq_lens_host,
                             const int32_t *cached_host, int32_t n_heads, int32_t n_kv_heads,
                             int32_t head_dim, int32_t max_ctx, const void *q,
                             const void *kcache, const void *vcache, void *o, void *scratch,
                             size_t scratch_bytes, void *stream);

/* Scratch bytes ll_op_attn_prefill needs for these arguments (same meaning); 0 when they are
 * invalid.  Host only. */
size_t ll_op_attn_prefill_scratch(int32_t dtype, int32_t batch, const int32_t *seq_lens_host,
                                  const int32_t *cached_host, int32_t n_heads,
                                  int32_t n_kv_heads, int32_t head_dim, int32_t max_ctx);

/* Decode attention: one query per sequence over ctx_lens_dev[b] cached keys (same
 * appendix: each KV tile loaded once for its whole query-head group; split over the cache
 * length with an fp32 log-sum-exp combine).  q T [batch, n_heads*head_dim]; caches as
 * above; o T [batch, n_heads*head_dim].  1 <= ctx_lens_dev[b] <= max_ctx <= 32768 (larger
 * values are clamped to max_ctx).  scratch >= ll_op_attn_decode_scratch(...) bytes (split
 * partials). */
ll_status ll_op_attn_decode(int32_t dtype, int32_t batch, int32_t n_heads, int32_t n_kv_heads,
                            int32_t head_dim, int32_t max_ctx, const void *q,
                            const void *kcache, const void *vcache, const int32_t *ctx_lens_dev,
                            void *o, void *scratch, size_t scratch_bytes, void *stream);
size_t ll_op_attn_decode_scratch(int32_t batch, int32_t n_heads, int32_t n_kv_heads,
                                 int32_t head_dim, int32_t max_ctx);

/* LM head with fused greedy argmax: logits = h W^T, next[r] = argmax (lowest index on
 * ties).  h T [rows, k], wt repacked [vocab, k], logits fp32 [rows, vocab] (nullable),
 * next int32 [rows].  scratch >= 8 * rows * vocab / 32 bytes (per-block partials). */
ll_status ll_op_lmhead_argmax(int32_t dtype, int32_t rows, int32_t vocab, int32_t k,
                              const void *h, const void *wt, float *logits, int32_t *next,
                              void *scratch, size_t scratch_bytes, void *stream);

/* ll_op_lmhead_argmax for callers that cannot allocate: code under HIP graph capture, tight
 * serving loops, harnesses that forbid allocation.  Same arguments, kernels and results,
 * without the scratch: the per-block partials live in a static device array of 2 MiB that the
 * library holds on each GPU it runs on until the process ends (its address is resolved once
 * per device, on the first call with that device current).  rows * vocab / 32 <= 262144
 * (LL_ERR_CAPACITY otherwise, nothing enqueued).  No allocation of any kind.  Every call on a
 * GPU shares that GPU's array: calls that overlap on one GPU (other streams, other threads)
 * race; each partial is written before it is read, so nothing needs clearing between calls. */
ll_status ll_op_lmhead_argmax_noalloc(int32_t dtype, int32_t rows, int32_t vocab, int32_t k,
                                      const void *h, const void *wt, float *logits,
                                      int32_t *next, void *stream);

/* Calibration, not part of the model: an MFMA-only loop (no memory traffic inside it) that
 * measures the bf16 matrix-core rate this GPU sustains, reported beside the datasheet peak.
 * blocks blocks of 4 waves; each wave runs iters x 8 v_mfma_f32_16x16x32_bf16, i.e.
 * blocks * 4 * iters * 8 * 16384 flops in all; out_dev fp32 [4 * blocks] receives one sum per
 * wave. */
ll_status ll_op_mfma_loop(int32_t blocks, int32_t iters, float *out_dev, void *stream);

/* Calibration, not part of the model: a read-only stream over n fp32 values of src_dev (device,
 * n a multiple of 4, 16-byte aligned) by blocks of 256 threads, block b reading the b-th of
 * `blocks` contiguous, equal ranges with eight non-temporal 16-byte loads in flight per
 * thread; out_dev fp32 [blocks] receives each block's sum of what it read (the sum of all of
 * them is the sum of src).  Measures the HBM read rate this GPU sustains,
 * reported beside the datasheet peak.  LL_ERR_INVALID_ARGUMENT for n < 0, n not a multiple of
 * 4, blocks < 1, a NULL out_dev, or a NULL / misaligned src_dev with n > 0. */
ll_status ll_op_read_stream(const float *src_dev, int64_t n, int32_t blocks, float *out_dev,
                            void *stream);

#ifdef __cplusplus
}
#endif
#endif /* LL_OPS_H */
