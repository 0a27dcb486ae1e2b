/*
 * ll.h -- C ABI of the phase-split decoder forward pass on one MI355X (gfx950).
 *
 * The paper frames inference as a target script with two phases whose kernels must be
 * specialised separately (Sec. 2.1 "Motivating Evidence"; Sec. 3.1 "Hotspot Discovery and
 * Phase-Aware Extraction"; appendix "Deployment Kernel Families", Table A.4):
 *   - prefill: attention over a block of prompt queries (q_len > 1) that builds the KV cache;
 *   - decode:  one query per sequence (q_len = 1) against the populated cache, which
 *              appends exactly one entry per step.
 * The library implements the forward pass of a pre-norm LLaMA-style decoder (RMSNorm,
 * rotate-half RoPE, grouped-query attention, SwiGLU MLP, untied LM head, greedy argmax)
 * for both phases, entirely in HIP kernels.
 *
 * Conventions for every call:
 *   - No exceptions cross the boundary.  Every call validates its host-visible arguments
 *     first and returns a status without enqueuing anything when they are wrong.
 *   - The library never allocates device memory.  The caller passes one workspace buffer
 *     (size from ll_workspace_size) that holds repacked weights, the KV cache, activations
 *     and metadata for the model's lifetime.
 *   - All device work is enqueued on the caller's HIP stream and the calls return without
 *     synchronising; device faults surface at the caller's next synchronisation.
 *   - A model handle is not thread-safe: use one host thread per handle.
 *   - ll_last_error() returns a thread-local description of the last failure.
 */
#ifndef LL_H
#define LL_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ll_model ll_model; /* opaque, library-owned host object */

typedef enum {
  LL_OK = 0,
  LL_ERR_INVALID_ARGUMENT = 1, /* null pointer, non-positive size, bad length */
  LL_ERR_UNSUPPORTED = 2,      /* shape the kernels do not cover (rejected at load) */
  LL_ERR_CAPACITY = 3,         /* batch, token or context limit of the config exceeded */
  LL_ERR_STATE = 4,            /* prefill batch != cached sequences, decode before prefill */
  LL_ERR_WORKSPACE = 5,        /* workspace missing, too small or misaligned */
  LL_ERR_HIP = 6               /* a HIP runtime call or kernel launch failed */
} ll_status;

/* LL_F16 names fp16 operands; it is accepted by the per-kernel entry points (ll_ops.h), while
 * a model's weights are LL_F32 or LL_BF16 and ll_config.f16_compute chooses fp16 operands. */
typedef enum { LL_F32 = 0, LL_BF16 = 1, LL_F16 = 2 } ll_dtype;

/* Model shape and capacity.  Supported: head_dim in {64, 128}; n_heads a multiple of
 * n_kv_heads with n_heads / n_kv_heads in {1, 2, 4, 8}; d_model, n_heads*head_dim and
 * (n_heads + 2 n_kv_heads)*head_dim and 2*ffn_dim multiples of 128; ffn_dim and d_model
 * multiples of 64; vocab a multiple of 32; max_batch <= LL_MAX_BATCH. */
typedef struct {
  int32_t n_layers, d_model, n_heads, n_kv_heads, head_dim, ffn_dim, vocab;
  float rms_eps;        /* RMSNorm epsilon (inside the square root) */
  double rope_theta;    /* RoPE base: freq_i = theta^(-2i/head_dim) */
  int32_t dtype;        /* ll_dtype: storage of weights, KV cache and GEMM inputs */
  int32_t max_batch;          /* sequences per prefill / decode step */
  int32_t max_prefill_tokens; /* total prompt tokens of one prefill */
  int32_t max_ctx;            /* per-sequence cache capacity (prompt + decoded tokens) */
  /* Paged KV cache (vLLM-style block table; the paper's continuous-batching discussion
   * names paging as the missing piece for mixed phases).  kv_page = 0: one contiguous slab
   * of max_ctx positions per (sequence, kv head).  kv_page > 0 (a multiple of 256): the
   * cache of each layer is a pool of kv_pages pages of kv_page positions for every kv head
   * (kv_pages = 0: max_batch * ceil(max_ctx / kv_page)); a sequence holds ceil(len /
   * kv_page) pages, taken from the pool when ll_prefill or ll_decode_step first writes a
   * position in them and returned by ll_kv_reset, so sequences of different lengths share a
   * pool smaller than max_batch full contexts.  The block table lives in the workspace. */
  int32_t kv_page;
  int32_t kv_pages;
  /* LL_BF16 weights only.  0: GEMM inputs, activations and the KV cache in bf16.  1: the
   * weights are converted to fp16 at load -- exact for every bf16 value of magnitude in
   * [2^-17, 65504], since bf16's 8-bit significand fits fp16's 11 (smaller magnitudes round to
   * fp16's subnormal grid of 2^-24; a larger one becomes inf and sets bit 1 of the device
   * flags) -- and GEMM inputs, activations and the KV cache are fp16: the same bytes and the
   * same MFMA rate, with 8x finer rounding of every activation.  Activations must then stay
   * within the fp16 range (|v| <= 65504); the residual stream and all accumulation stay fp32. */
  int32_t f16_compute;
} ll_config;

#define LL_MAX_BATCH 256

/* Weights: DEVICE pointers, element type = cfg.dtype, row-major [out][in] (y = x W^T).
 * Per-layer fields are HOST arrays of n_layers device pointers.  They are read only
 * during ll_model_load (repacked into the workspace); the caller may free them after
 * synchronising the stream that ll_model_load used. */
typedef struct {
  const void *tok_embed;   /* [vocab, d_model] */
  const void *final_norm;  /* [d_model] RMSNorm gain before the LM head */
  const void *lm_head;     /* [vocab, d_model] (untied) */
  const void *const *attn_norm; /* [d_model] */
  const void *const *wq;        /* [n_heads*head_dim, d_model] */
  const void *const *wk;        /* [n_kv_heads*head_dim, d_model] */
  const void *const *wv;        /* [n_kv_heads*head_dim, d_model] */
  const void *const *wo;        /* [d_model, n_heads*head_dim] */
  const void *const *mlp_norm;  /* [d_model] */
  const void *const *w_gate;    /* [ffn_dim, d_model] */
  const void *const *w_up;      /* [ffn_dim, d_model] */
  const void *const *w_down;    /* [d_model, ffn_dim] */
} ll_weights;

/* Bytes of workspace the config needs.  Host only, no HIP call. */
ll_status ll_workspace_size(const ll_config *cfg, size_t *bytes);

/* Validate cfg, repack the weights into `workspace` (device memory, >= ll_workspace_size
 * bytes, 256-byte aligned) and build the RoPE table, all enqueued on `hip_stream`
 * (a hipStream_t; NULL = the default stream).  On success *out owns host state only;
 * the workspace stays the caller's and must outlive the model. */
ll_status ll_model_load(const ll_config *cfg, const ll_weights *w, void *workspace,
                        size_t workspace_bytes, void *hip_stream, ll_model **out);

/* Prefill phase (a block of q_len >= 1 prompt tokens per sequence).
 * batch sequences with host lengths seq_lens_host[batch] (each >= 1); tokens_dev holds the
 * sum(seq_lens) token ids packed in sequence order (device, int32, each in [0, vocab)).
 * On an empty cache this starts `batch` new sequences at position 0.  On a populated cache
 * (after an earlier ll_prefill, possibly followed by decode steps) it is a further prompt
 * chunk of the same `batch` sequences: sequence b's tokens enter at positions len[b] ..
 * len[b] + seq_lens_host[b] - 1 and attend to everything cached before them (chunked
 * prefill).  Writes next_tokens_dev[batch] (device) = argmax of the logits at each
 * sequence's last new position (lowest index on ties) and, if logits_dev is not NULL, the
 * fp32 logits [batch, vocab].  Afterwards len[b] grows by seq_lens_host[b].
 * LL_ERR_STATE if the cache holds a different number of sequences (ll_kv_reset starts new
 * ones); LL_ERR_CAPACITY if batch > max_batch, sum(seq_lens) > max_prefill_tokens, some
 * len[b] + seq_lens_host[b] > max_ctx or (paged cache) the free pages do not cover the new
 * positions; nothing is enqueued and no state changes then. */
ll_status ll_prefill(ll_model *m, int32_t batch, const int32_t *seq_lens_host,
                     const int32_t *tokens_dev, int32_t *next_tokens_dev, float *logits_dev);

/* Decode phase (q_len = 1 against the populated cache): feeds in_tokens_dev[b] at position
 * len[b] of every sequence of the last prefill, appends its key/value, writes
 * next_tokens_dev[b] (and fp32 logits [batch, vocab] if logits_dev is not NULL) and
 * advances every length by one.  in_tokens_dev may equal next_tokens_dev (greedy
 * feedback).  The step runs as one HIP graph replay, captured on first use for each
 * (in, out, logits) pointer triple.  LL_ERR_STATE before a prefill; LL_ERR_CAPACITY when
 * some len[b] + 1 > max_ctx or (paged cache) a sequence entering a new page finds the pool
 * empty.  With a paged cache the new block-table entries are copied to the device on the
 * model's stream before the step. */
ll_status ll_decode_step(ll_model *m, const int32_t *in_tokens_dev, int32_t *next_tokens_dev,
                         float *logits_dev);

/* Forget every sequence (all lengths 0); the next call must be ll_prefill.  With a paged
 * cache every page returns to the pool (the call first synchronises the stream, since
 * block-table copies of earlier steps read host memory that is reused). */
ll_status ll_kv_reset(ll_model *m);

/* Paged cache: pages held by the current sequences and pages in the pool (both 0 for a
 * contiguous cache).  Host only. */
ll_status ll_kv_pages(const ll_model *m, int32_t *used, int32_t *total);

/* The regions of the model's workspace, in address order: writes min(cap, count) entries of
 * byte offset from the workspace start, size in bytes and name (a string owned by the model,
 * valid until ll_model_free: "embed", "layers.<l>.wqkv", "kcache", "x", ...); *n = count.
 * Every region is followed by a gap of at least 256 bytes that no kernel writes, so a caller
 * (a test harness, a debugging allocator) can fill the gaps with a pattern and check after
 * any call that no kernel wrote past a region's end.  Host only. */
ll_status ll_workspace_regions(const ll_model *m, int32_t cap, uint64_t *offsets,
                               uint64_t *bytes, const char **names, int32_t *n);

/* Current host-mirrored sequence lengths: writes min(cap, batch) values, *n = batch. */
ll_status ll_seq_lengths(const ll_model *m, int32_t *out, int32_t cap, int32_t *n);

/* Enable (1, default) or disable (0) HIP-graph replay of decode steps. */
ll_status ll_set_decode_graph(ll_model *m, int32_t enable);

/* Implementation variants of the hot path.  Each option chooses between kernels that compute
 * the same function (results differ only in fp32 summation order); none changes the model.
 * The paper admits such a variant into the deployed model only when the model's own measured
 * latency drops by at least a margin delta (Sec. 3.3, Eq. 3) -- see the package's tuner.
 * Changing an option drops the captured decode graphs (they are captured again on use). */
typedef enum {
  LL_OPT_DECODE_GRAPH = 0,     /* 1 (default): decode steps replay a HIP graph; 0: direct launches
                                  (same as ll_set_decode_graph) */
  LL_OPT_PREFILL_SPLITK = 1,   /* 1 (default): prefill GEMMs whose 64x128 tiles cannot fill the
                                  GPU split K over blocks; 0: never split */
  LL_OPT_DECODE_SPLITK = 2,    /* 1 (default): decode GEMMs above 16 rows split K over blocks of
                                  128 columns; 0: whole-K blocks; 2: as 1, and up to 16 rows the
                                  residual GEMMs split K over two blocks per column block that add
                                  their partial sums with fp32 atomics (more blocks streaming the
                                  weights; the summation order is then not fixed) */
  LL_OPT_PREFILL_TILE = 3,     /* 0 (default): prefill GEMM tile family chosen per shape; 1: 256x256,
                                  2: 128x256, 3: 64x128 (256-column tiles only where the output
                                  width is a multiple of 256; elsewhere the default) */
  LL_OPT_ATTN_DECODE_CHUNK = 4,/* 0 (default): cached keys per decode-attention block from the
                                  load-time plan; 64, 128 or 256 override it (not below the plan's
                                  value: the workspace holds the plan's number of splits) */
  LL_OPT_DECODE_FUSED = 5,     /* Decoder: 0 (default): the decode attention's splits are merged
                                  by a kernel of their own; 1: a decode step of at most 16
                                  sequences whose attention uses 2..16 splits merges them while
                                  the O projection stages its A rows (same arithmetic, same
                                  bits; one launch per layer fewer).  Mamba model (ll_mamba.h):
                                  1 (default): a decode step of at most 4 sequences runs the conv
                                  step in the in_proj epilogue and x_proj inside the scan-step
                                  kernel; 2: as 1, and out_proj with the residual add inside the
                                  scan step too, its 32-channel shares added with fp32 atomics
                                  (the summation order, hence the last bits, can differ between
                                  runs); 0: separate conv, x_proj and scan kernels.  The Mamba2
                                  and RG-LRU models reject it (LL_ERR_UNSUPPORTED) */
  LL_OPT_COUNT = 6
} ll_option;

/* Set / read an option.  LL_ERR_INVALID_ARGUMENT for an unknown option or value,
 * LL_ERR_UNSUPPORTED for a decode-attention chunk below the load-time plan's. */
ll_status ll_set_option(ll_model *m, int32_t option, int32_t value);
ll_status ll_get_option(const ll_model *m, int32_t option, int32_t *value);

/* Synchronise the model's stream and read the device error flags: bit 0 = a token id
 * outside [0, vocab) was seen (it was replaced by 0, never read out of bounds); bit 1 = a
 * weight outside the fp16 range met the conversion of f16_compute. */
ll_status ll_device_flags(ll_model *m, int32_t *flags);

/* Kernel classes of the hot path, for per-module timing.  The paper ranks modules by the
 * time t(m, p) they take in each phase p relative to the phase latency T(p) (Sec. 3,
 * Eq. 1); these classes are the modules of this forward pass. */
typedef enum {
  LL_K_META = 0,        /* prefill metadata (offsets, positions, tile order) */
  LL_K_EMBED = 1,       /* embedding gather */
  LL_K_RMSNORM = 2,     /* RMSNorm kernel (decode batches <= 16 normalise inside the GEMM) */
  LL_K_QKV = 3,         /* fused QKV projection + RoPE + KV-cache append */
  LL_K_ATTN = 4,        /* causal prefill attention, or the per-split decode attention */
  LL_K_ATTN_COMBINE = 5,/* decode attention: merge of the per-split partial results */
  LL_K_O = 6,           /* O projection + residual add */
  LL_K_GATE_UP = 7,     /* gate/up projection + SwiGLU */
  LL_K_DOWN = 8,        /* down projection + residual add */
  LL_K_LM_HEAD = 9,     /* LM head + per-block argmax partials */
  LL_K_ARGMAX = 10,     /* argmax reduction (+ length advance in decode) */
  LL_K_COUNT = 11
} ll_kernel_class;

/* Enable (1) or disable (0) per-launch timing.  While enabled, every kernel of ll_prefill
 * and ll_decode_step is launched with a start/stop HIP event pair stamped by the dispatch
 * itself (hipExtLaunchKernel), and decode steps launch their kernels directly instead of
 * replaying the graph.  Host event objects are created as needed; no device memory. */
ll_status ll_set_kernel_timing(ll_model *m, int32_t enable);

/* Synchronise the model's stream and return the launches and summed kernel milliseconds
 * recorded since the last read, per phase and class: index phase * LL_K_COUNT + class,
 * phase 0 = prefill, 1 = decode.  counts and ms hold 2 * LL_K_COUNT entries. */
ll_status ll_kernel_timing_read(ll_model *m, int32_t *counts, double *ms);

/* Name of a kernel class ("" if out of range). */
const char *ll_kernel_class_name(int32_t cls);

/* Release host state (graphs, handle).  The workspace is the caller's. */
void ll_model_free(ll_model *m);

/* Thread-local text of the last error ("" if none). */
const char *ll_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* LL_H */
