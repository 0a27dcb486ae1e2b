/*
 * ll_mamba2.h -- C ABI of a Mamba2 (state-space duality) language model on one MI355X
 * (gfx950), prefill and single-token decode with explicit convolution and SSM state.
 *
 * The paper's Mamba2 case (appendix "Deployment Kernel Families", Table A.4) keeps the mixer
 * sequence -- input projection, depthwise convolution, split into hidden and state
 * parameters, recurrent scan, gated RMSNorm, output projection -- with the state tile in
 * registers across the scan and B, C shared by the heads; the Mamba family's phase contract
 * (state ownership) is that of ll_mamba.h.  Each layer is a pre-norm residual block:
 *   [z | x B C | dt] = in_proj(RMSNorm(x) * g),  [x | B | C] = silu(causal depthwise conv),
 *   dt = softplus(dt + dt_bias) per head,  A = -exp(A_log) per head,
 *   per head (group h / (H / G) of B, C; state [head_dim][d_state]):
 *     h_t = exp(dt_t A) h_{t-1} + dt_t x_t B_t^T,   y_t = h_t C_t + D x_t,
 *   x += out_proj( RMSNorm(y * silu(z)) * gnorm ),
 * then a final RMSNorm and an LM head tied to the embedding, greedy argmax.
 * Prefill of bf16 models evaluates the scan over chunks of 64 steps in its matrix form
 * (C B^T masked and decayed, times x, plus the incoming state's term) on fp16 MFMAs with fp32
 * accumulation, which is the same recurrence unrolled; fp32 models and decode run the step
 * recurrence in fp32.
 *
 * Conventions are those of ll.h (statuses, ll_last_error, no device allocation, work on the
 * caller's stream, one host thread per handle).
 */
#ifndef LL_MAMBA2_H
#define LL_MAMBA2_H

#include "ll.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ll_mamba2 ll_mamba2; /* opaque, library-owned host object */

/* Model shape and capacity.  Supported: d_state in {32, 64, 128, 256}; head_dim a multiple of
 * 16 dividing d_inner; n_groups dividing the head count; d_conv in [1, 4]; d_model a multiple
 * of 128; d_inner a multiple of 64; vocab a multiple of 32; max_batch <= LL_MAX_BATCH. */
typedef struct {
  int32_t n_layers, d_model, d_inner, d_state, head_dim, n_groups, d_conv, vocab;
  float rms_eps;              /* epsilon of every RMSNorm, the gated one included */
  int32_t dtype;              /* ll_dtype of the embedding, norms and projections */
  int32_t max_batch;          /* sequences per prefill / decode step */
  int32_t max_prefill_tokens; /* total prompt tokens of one prefill call */
} ll_mamba2_config;

/* Weights: DEVICE pointers.  "T" = cfg.dtype; matrices row-major [out][in].  Per-layer fields
 * are HOST arrays of n_layers device pointers, read only during ll_mamba2_load.  With
 * H = d_inner / head_dim and CD = d_inner + 2 n_groups d_state: */
typedef struct {
  const void *embed;            /* T [vocab, d_model]; also the LM head */
  const void *final_norm;       /* T [d_model] */
  const void *const *norm;      /* T [d_model] */
  const void *const *in_proj;   /* T [d_inner + CD + H, d_model]: rows z | x B C | dt */
  const float *const *conv_w;   /* fp32 [CD, d_conv]; tap d_conv-1 multiplies the current row */
  const float *const *conv_b;   /* fp32 [CD] */
  const float *const *dt_b;     /* fp32 [H] */
  const float *const *A_log;    /* fp32 [H] */
  const float *const *D;        /* fp32 [H] */
  const void *const *gnorm;     /* T [d_inner] gated RMSNorm gain */
  const void *const *out_proj;  /* T [d_model, d_inner] */
} ll_mamba2_weights;

ll_status ll_mamba2_workspace_size(const ll_mamba2_config *cfg, size_t *bytes);
ll_status ll_mamba2_load(const ll_mamba2_config *cfg, const ll_mamba2_weights *w, void *workspace,
                         size_t workspace_bytes, void *hip_stream, ll_mamba2 **out);
/* Prefill / continuation / decode / reset: the same contract as the ll_mamba_* calls. */
ll_status ll_mamba2_prefill(ll_mamba2 *m, int32_t batch, const int32_t *seq_lens_host,
                            const int32_t *tokens_dev, int32_t *next_tokens_dev,
                            float *logits_dev);
ll_status ll_mamba2_decode_step(ll_mamba2 *m, const int32_t *in_tokens_dev,
                                int32_t *next_tokens_dev, float *logits_dev);
ll_status ll_mamba2_reset(ll_mamba2 *m);
ll_status ll_mamba2_seq_lengths(const ll_mamba2 *m, int32_t *out, int32_t cap, int32_t *n);
/* Options (ids of ll_option): LL_OPT_DECODE_GRAPH, LL_OPT_PREFILL_SPLITK,
 * LL_OPT_DECODE_SPLITK, LL_OPT_PREFILL_TILE; the others give LL_ERR_UNSUPPORTED. */
ll_status ll_mamba2_set_option(ll_mamba2 *m, int32_t option, int32_t value);
ll_status ll_mamba2_get_option(const ll_mamba2 *m, int32_t option, int32_t *value);
ll_status ll_mamba2_device_flags(ll_mamba2 *m, int32_t *flags);

/* Kernel classes of the Mamba2 forward pass (Sec. 3, Eq. 1). */
typedef enum {
  LL_M2K_META = 0,       /* prefill metadata */
  LL_M2K_EMBED = 1,      /* embedding gather */
  LL_M2K_RMSNORM = 2,    /* block RMSNorm kernel (decode batches <= 16 normalise in the GEMM) */
  LL_M2K_IN_PROJ = 3,    /* in_proj GEMM (decode: + the conv step and SiLU) */
  LL_M2K_CONV = 4,       /* causal depthwise conv + SiLU (prefill) */
  LL_M2K_SCAN_CHUNK = 5, /* prefill scan pass 1 */
  LL_M2K_SCAN_CARRY = 6, /* prefill scan pass 2 */
  LL_M2K_SCAN = 7,       /* scan with output (pass 3; the decode step) */
  LL_M2K_GNORM = 8,      /* gated RMSNorm kernel (decode batches <= 16: inside out_proj) */
  LL_M2K_OUT_PROJ = 9,   /* out_proj GEMM + residual add */
  LL_M2K_LM_HEAD = 10,   /* LM head + argmax partials */
  LL_M2K_ARGMAX = 11,    /* argmax reduction */
  LL_M2K_COUNT = 12
} ll_mamba2_kernel_class;

ll_status ll_mamba2_set_kernel_timing(ll_mamba2 *m, int32_t enable);
ll_status ll_mamba2_kernel_timing_read(ll_mamba2 *m, int32_t *counts, double *ms);
const char *ll_mamba2_kernel_class_name(int32_t cls);
void ll_mamba2_free(ll_mamba2 *m);

#ifdef __cplusplus
}
#endif
#endif /* LL_MAMBA2_H */
