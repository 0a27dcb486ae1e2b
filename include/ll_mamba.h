/*
 * ll_mamba.h -- C ABI of a selective state-space (Mamba) language model on one MI355X (gfx950),
 * prefill and single-token decode with explicit convolution and SSM state.
 *
 * The paper's Mamba-family cases (appendix "Deployment Kernel Families", Table A.4, and its
 * discussion of state ownership) fix the phase contract: the prefill runs the recurrent scan
 * over the prompt block and leaves the convolution and SSM state of every sequence behind; a
 * decode step takes one token per sequence with that state, updates both exactly once and
 * returns the next token.  Each layer is the standard Mamba mixer behind a pre-norm residual:
 *   x += out_proj( y * silu(z) ),   [xc | z] = in_proj( RMSNorm(x) * g ),
 *   u = silu(causal depthwise conv(xc) + conv_b),   [dt_low | B | C] = x_proj(u),
 *   dt = softplus(dt_w dt_low + dt_b),   A = -exp(A_log),
 *   h_t = exp(dt_t A) * h_{t-1} + dt_t B_t u_t,   y_t = C_t . h_t + D u_t,
 * then a final RMSNorm and an LM head tied to the embedding, greedy argmax.
 *
 * Conventions are those of ll.h: statuses from ll.h, ll_last_error() for the text, no device
 * allocation (one caller workspace), all work enqueued on the caller's stream, one host thread
 * per handle.
 */
#ifndef LL_MAMBA_H
#define LL_MAMBA_H

#include "ll.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ll_mamba ll_mamba; /* opaque, library-owned host object */

/* Model shape and capacity.  Supported: d_state = 16; d_conv in [1, 4]; dt_rank in [1, 160];
 * d_model a multiple of 128; d_inner a multiple of 64; vocab a multiple of 32;
 * max_batch <= LL_MAX_BATCH.  There is no context limit: the state has a fixed size. */
typedef struct {
  int32_t n_layers, d_model, d_inner, d_state, d_conv, dt_rank, vocab;
  float rms_eps;              /* RMSNorm epsilon (inside the square root) */
  int32_t dtype;              /* ll_dtype of the embedding, norms, projections and activations */
  int32_t max_batch;          /* sequences per prefill / decode step */
  int32_t max_prefill_tokens; /* total prompt tokens of one prefill call */
} ll_mamba_config;

/* Weights: DEVICE pointers.  "T" = cfg.dtype; matrices row-major [out][in] (y = x W^T).
 * Per-layer fields are HOST arrays of n_layers device pointers, read only during
 * ll_mamba_load (copied / repacked into the workspace). */
typedef struct {
  const void *embed;            /* T [vocab, d_model]; also the LM head */
  const void *final_norm;       /* T [d_model] */
  const void *const *norm;      /* T [d_model] */
  const void *const *in_proj;   /* T [2 d_inner, d_model]: rows [0, d_inner) -> xc, the rest -> z */
  const float *const *conv_w;   /* fp32 [d_inner, d_conv]; tap d_conv-1 multiplies the current row */
  const float *const *conv_b;   /* fp32 [d_inner] */
  const void *const *x_proj;    /* T [dt_rank + 2 d_state, d_inner] -> dt_low | B | C */
  const float *const *dt_w;     /* fp32 [d_inner, dt_rank] */
  const float *const *dt_b;     /* fp32 [d_inner] */
  const float *const *A_log;    /* fp32 [d_inner, d_state] */
  const float *const *D;        /* fp32 [d_inner] */
  const void *const *out_proj;  /* T [d_model, d_inner] */
} ll_mamba_weights;

/* Bytes of workspace the config needs.  Host only, no HIP call. */
ll_status ll_mamba_workspace_size(const ll_mamba_config *cfg, size_t *bytes);

/* Validate cfg, copy / repack the weights into `workspace` (device, >= ll_mamba_workspace_size
 * bytes, 256-byte aligned), enqueued on `hip_stream` (NULL = default stream).  On success *out
 * owns host state only; the workspace stays the caller's and must outlive the model. */
ll_status ll_mamba_load(const ll_mamba_config *cfg, const ll_mamba_weights *w, void *workspace,
                        size_t workspace_bytes, void *hip_stream, ll_mamba **out);

/* Prefill: `batch` sequences of seq_lens_host[b] >= 1 tokens (tokens_dev packed in sequence
 * order, int32 in [0, vocab)).  With no sequences held it starts new ones from zero state; on
 * held state it is a further chunk of the same sequences, continuing their conv and SSM state
 * (LL_ERR_STATE if batch differs).  Writes next_tokens_dev[batch] = argmax of the logits at
 * each sequence's last new token (lowest index on ties) and, if logits_dev is not NULL, the
 * fp32 logits [batch, vocab].  LL_ERR_CAPACITY: batch > max_batch or sum > max_prefill_tokens. */
ll_status ll_mamba_prefill(ll_mamba *m, int32_t batch, const int32_t *seq_lens_host,
                           const int32_t *tokens_dev, int32_t *next_tokens_dev,
                           float *logits_dev);

/* Decode: one token per held sequence (in_tokens_dev[b], may equal next_tokens_dev), state
 * updated once, next_tokens_dev[b] (and logits [batch, vocab] if not NULL) written.  Replays a
 * HIP graph captured per (in, out, logits) pointer triple unless disabled.  LL_ERR_STATE
 * before a prefill. */
ll_status ll_mamba_decode_step(ll_mamba *m, const int32_t *in_tokens_dev,
                               int32_t *next_tokens_dev, float *logits_dev);

/* Forget every sequence; the next call must be ll_mamba_prefill. */
ll_status ll_mamba_reset(ll_mamba *m);

/* Tokens consumed so far per held sequence: writes min(cap, batch) values, *n = batch. */
ll_status ll_mamba_seq_lengths(const ll_mamba *m, int32_t *out, int32_t cap, int32_t *n);

/* Options (ids of ll_option in ll.h): LL_OPT_DECODE_GRAPH, LL_OPT_PREFILL_SPLITK,
 * LL_OPT_DECODE_SPLITK, LL_OPT_PREFILL_TILE and LL_OPT_DECODE_FUSED, with the values ll.h
 * documents; LL_OPT_ATTN_DECODE_CHUNK gives LL_ERR_UNSUPPORTED.  Changing one drops captured
 * decode graphs. */
ll_status ll_mamba_set_option(ll_mamba *m, int32_t option, int32_t value);
ll_status ll_mamba_get_option(const ll_mamba *m, int32_t option, int32_t *value);

/* Synchronise the stream and read the device error flags (bit 0: a token id outside
 * [0, vocab) was seen and replaced by 0). */
ll_status ll_mamba_device_flags(ll_mamba *m, int32_t *flags);

/* Kernel classes of the Mamba forward pass for per-module timing (Sec. 3, Eq. 1). */
typedef enum {
  LL_MK_META = 0,       /* prefill metadata (offsets, chunk list) */
  LL_MK_EMBED = 1,      /* embedding gather */
  LL_MK_RMSNORM = 2,    /* RMSNorm kernel (decode batches <= 16 normalise inside the GEMM) */
  LL_MK_IN_PROJ = 3,    /* in_proj GEMM -> xc | z (fused decode: + the conv step and SiLU) */
  LL_MK_CONV = 4,       /* causal depthwise conv + SiLU */
  LL_MK_X_PROJ = 5,     /* x_proj GEMM -> dt_low | B | C */
  LL_MK_SCAN_CHUNK = 6, /* prefill scan pass 1: chunk end states */
  LL_MK_SCAN_CARRY = 7, /* prefill scan pass 2: incoming state of each chunk */
  LL_MK_SCAN = 8,       /* scan with output and state update (pass 3; the decode step, which
                           in the fused decode also forms x_proj) */
  LL_MK_OUT_PROJ = 9,   /* out_proj GEMM + residual add */
  LL_MK_LM_HEAD = 10,   /* LM head + per-block argmax partials */
  LL_MK_ARGMAX = 11,    /* argmax reduction */
  LL_MK_COUNT = 12
} ll_mamba_kernel_class;

/* Per-launch timing as in ll.h (hipExtLaunchKernel events; decode then launches directly).
 * ll_mamba_kernel_timing_read: counts / ms hold 2 * LL_MK_COUNT entries, phase-major
 * (0 = prefill, 1 = decode). */
ll_status ll_mamba_set_kernel_timing(ll_mamba *m, int32_t enable);
ll_status ll_mamba_kernel_timing_read(ll_mamba *m, int32_t *counts, double *ms);
const char *ll_mamba_kernel_class_name(int32_t cls);

/* Release host state (graphs, handle).  The workspace is the caller's. */
void ll_mamba_free(ll_mamba *m);

#ifdef __cplusplus
}
#endif
#endif /* LL_MAMBA_H */
