/*
 * ll_rglru.h -- C ABI of a language model of Griffin recurrent blocks (the RG-LRU layer of
 * RecurrentGemma) on one MI355X (gfx950), prefill and single-token decode with explicit
 * convolution and recurrent state.
 *
 * The paper's recurrent case (appendix "Deployment Kernel Families", Table A.4, and the
 * paragraph on RecurrentGemma) fuses sigmoid gates, the softplus-derived recurrent gate, reset
 * handling, input normalisation and the recurrent scan, with the state carried through the
 * sequence and the final state written once; its state-ownership contract is the Mamba
 * family's (ll_mamba.h): the prefill leaves conv and recurrent state behind, a decode step
 * updates both exactly once.  Each residual block (every temporal block is recurrent):
 *   h = RMSNorm(x) * (1 + norm_t),
 *   y = gelu_tanh(linear_y h + b_y),  v = conv(linear_x h + b_x)  (causal depthwise, bias,
 *   no activation),  x += linear_out(rglru(v) * y) + b_out,
 *   rglru per channel j of head k (block-diagonal gate weights [k][out][in]):
 *     r = sigmoid(gate_a v + b_a),  i = sigmoid(gate_x v + b_x'),
 *     log a = -8 r softplus(lambda),
 *     h_t = a h_{t-1} + sqrt(1 - a^2) i v   (a sequence's first token: h = i v),
 *   h = RMSNorm(x) * (1 + norm_c),  x += mlp_down(gelu_tanh(mlp_gate h + b_g) *
 *   (mlp_up h + b_u)) + b_d,
 * with x0 = embed[token] * embed_scale, then RMSNorm * (1 + final_norm), an LM head tied to
 * the embedding, logits soft-capped as cap * tanh(l / cap), greedy argmax.
 *
 * Conventions are those of ll.h (statuses, ll_last_error, no device allocation, work on the
 * caller's stream, one host thread per handle).
 */
#ifndef LL_RGLRU_H
#define LL_RGLRU_H

#include "ll.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ll_rg ll_rg; /* opaque, library-owned host object */

/* Model shape and capacity.  Supported: lru_width = n_heads * block with block a multiple of
 * 64; d_model a multiple of 128; mlp_width a multiple of 64; d_conv in [1, 4]; vocab a
 * multiple of 32; max_batch <= LL_MAX_BATCH.  No context limit: the state has a fixed size. */
typedef struct {
  int32_t n_layers, d_model, lru_width, n_heads, mlp_width, d_conv, vocab;
  float rms_eps;              /* RMSNorm epsilon (inside the square root) */
  float embed_scale;          /* factor of the embedding rows (RecurrentGemma: sqrt(d) in bf16) */
  float logit_cap;            /* soft cap of the logits, > 0 */
  int32_t dtype;              /* ll_dtype of the embedding, norm offsets, matrices, activations */
  int32_t max_batch;          /* sequences per prefill / decode step */
  int32_t max_prefill_tokens; /* total prompt tokens of one prefill call */
} ll_rg_config;

/* Weights: DEVICE pointers.  "T" = cfg.dtype, matrices row-major [out][in]; biases and the
 * recurrence parameters fp32.  Per-layer fields are HOST arrays of n_layers device pointers,
 * read only during ll_rg_load (copied / repacked into the workspace).  W = lru_width,
 * H = n_heads, bw = W / H, F = mlp_width, d = d_model, K = d_conv. */
typedef struct {
  const void *embed;                 /* T [vocab, d]; also the LM head */
  const void *final_norm;            /* T [d] offset (gain 1 + w) */
  const void *const *norm_t;         /* T [d] offset of the temporal pre-norm */
  const void *const *linear_y;       /* T [W, d] */
  const float *const *linear_y_b;    /* [W] */
  const void *const *linear_x;       /* T [W, d] */
  const float *const *linear_x_b;    /* [W] */
  const float *const *conv_w;        /* [W, K]; tap K-1 multiplies the current row */
  const float *const *conv_b;        /* [W] */
  const void *const *gate_a;         /* T [H, bw, bw] recurrence gate blocks, [head][out][in] */
  const float *const *gate_a_b;      /* [H, bw] */
  const void *const *gate_x;         /* T [H, bw, bw] input gate blocks */
  const float *const *gate_x_b;      /* [H, bw] */
  const float *const *lambda;        /* [W] recurrence parameter (a = exp(-8 r softplus)) */
  const void *const *linear_out;     /* T [d, W] */
  const float *const *linear_out_b;  /* [d] */
  const void *const *norm_c;         /* T [d] offset of the MLP pre-norm */
  const void *const *mlp_gate;       /* T [F, d] */
  const float *const *mlp_gate_b;    /* [F] */
  const void *const *mlp_up;         /* T [F, d] */
  const float *const *mlp_up_b;      /* [F] */
  const void *const *mlp_down;       /* T [d, F] */
  const float *const *mlp_down_b;    /* [d] */
} ll_rg_weights;

/* Bytes of workspace the config needs.  Host only, no HIP call. */
ll_status ll_rg_workspace_size(const ll_rg_config *cfg, size_t *bytes);

/* Validate cfg, copy / repack the weights into `workspace` (device, >= ll_rg_workspace_size
 * bytes, 256-byte aligned), enqueued on `hip_stream` (NULL = default stream).  On success *out
 * owns host state only; the workspace stays the caller's and must outlive the model. */
ll_status ll_rg_load(const ll_rg_config *cfg, const ll_rg_weights *w, void *workspace,
                     size_t workspace_bytes, void *hip_stream, ll_rg **out);

/* Prefill: `batch` sequences of seq_lens_host[b] >= 1 tokens (tokens_dev packed in sequence
 * order, int32 in [0, vocab)).  With no sequences held it starts new ones from zero state (the
 * first token of each is the RG-LRU's reset); on held state it is a further chunk of the same
 * sequences (LL_ERR_STATE if batch differs).  Writes next_tokens_dev[batch] = argmax of the
 * logits at each sequence's last new token (lowest index on ties) and, if logits_dev is not
 * NULL, the soft-capped fp32 logits [batch, vocab].  LL_ERR_CAPACITY: batch > max_batch or
 * sum > max_prefill_tokens. */
ll_status ll_rg_prefill(ll_rg *m, int32_t batch, const int32_t *seq_lens_host,
                        const int32_t *tokens_dev, int32_t *next_tokens_dev, float *logits_dev);

/* Decode: one token per held sequence (in_tokens_dev[b], may equal next_tokens_dev), state
 * updated once, next_tokens_dev[b] (and the logits if not NULL) written.  Replays a HIP graph
 * captured per (in, out, logits) pointer triple unless disabled.  LL_ERR_STATE before a
 * prefill. */
ll_status ll_rg_decode_step(ll_rg *m, const int32_t *in_tokens_dev, int32_t *next_tokens_dev,
                            float *logits_dev);

/* Forget every sequence; the next call must be ll_rg_prefill. */
ll_status ll_rg_reset(ll_rg *m);

/* Tokens consumed so far per held sequence: writes min(cap, batch) values, *n = batch. */
ll_status ll_rg_seq_lengths(const ll_rg *m, int32_t *out, int32_t cap, int32_t *n);

/* Options (ids of ll_option in ll.h): LL_OPT_DECODE_GRAPH, LL_OPT_PREFILL_SPLITK,
 * LL_OPT_DECODE_SPLITK, LL_OPT_PREFILL_TILE, with the values ll.h documents; the others give
 * LL_ERR_UNSUPPORTED.  Changing one drops captured decode graphs. */
ll_status ll_rg_set_option(ll_rg *m, int32_t option, int32_t value);
ll_status ll_rg_get_option(const ll_rg *m, int32_t option, int32_t *value);

/* Synchronise the stream and read the device error flags (bit 0: a token id outside
 * [0, vocab) was seen and replaced by 0). */
ll_status ll_rg_device_flags(ll_rg *m, int32_t *flags);

/* Kernel classes of the forward pass for per-module timing (Sec. 3, Eq. 1). */
typedef enum {
  LL_RGK_META = 0,       /* prefill metadata (offsets, chunk list) */
  LL_RGK_EMBED = 1,      /* embedding gather and scale */
  LL_RGK_RMSNORM = 2,    /* RMSNorm kernel (decode batches <= 16 normalise inside the GEMM) */
  LL_RGK_IN_PROJ = 3,    /* linear_y | linear_x GEMM: gelu branch, conv input (decode: + the
                            conv step) */
  LL_RGK_CONV = 4,       /* causal depthwise conv (prefill) */
  LL_RGK_GATES = 5,      /* RG-LRU gate GEMM with the gate, decay and normalisation epilogue
                            (decode: + the recurrence step and the product with the gelu
                            branch) */
  LL_RGK_SCAN_CHUNK = 6, /* prefill scan pass 1: chunk products and end states */
  LL_RGK_SCAN = 7,       /* prefill scan pass 3: rescan, output, final state */
  LL_RGK_OUT_PROJ = 8,   /* linear_out GEMM + bias + residual add */
  LL_RGK_MLP_UP = 9,     /* mlp gate | up GEMM with the GeGLU epilogue */
  LL_RGK_MLP_DOWN = 10,  /* mlp down GEMM + bias + residual add */
  LL_RGK_LM_HEAD = 11,   /* LM head + per-block argmax partials */
  LL_RGK_ARGMAX = 12,    /* argmax reduction */
  LL_RGK_SOFTCAP = 13,   /* soft cap of the returned logits (only when logits are requested) */
  LL_RGK_COUNT = 14
} ll_rg_kernel_class;

/* Per-launch timing as in ll.h.  ll_rg_kernel_timing_read: counts / ms hold 2 * LL_RGK_COUNT
 * entries, phase-major (0 = prefill, 1 = decode). */
ll_status ll_rg_set_kernel_timing(ll_rg *m, int32_t enable);
ll_status ll_rg_kernel_timing_read(ll_rg *m, int32_t *counts, double *ms);
const char *ll_rg_kernel_class_name(int32_t cls);

/* Release host state (graphs, handle).  The workspace is the caller's. */
void ll_rg_free(ll_rg *m);

#ifdef __cplusplus
}
#endif
#endif /* LL_RGLRU_H */
