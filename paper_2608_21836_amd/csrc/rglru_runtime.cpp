// C-ABI runtime of the Griffin recurrent-block (RG-LRU) model: config validation, workspace
// layout, weight repacking, prefill / decode dispatch with explicit conv and recurrent state,
// decode-step HIP graphs.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <vector>

#include "kernels.h"
#include "ll.h"
#include "ll_rglru.h"
#include "runtime_common.h"

using namespace ll;

namespace {

const char *const kRgClassNames[LL_RGK_COUNT] = {
    "prefill_meta", "embed",  "rmsnorm",        "in_proj",  "conv",     "gates",
    "scan_chunk",   "scan",   "out_proj_resid", "mlp_up",   "mlp_down", "lm_head_argmax",
    "argmax_reduce", "softcap"};

constexpr int kFusedNormMaxRows = 16;
constexpr float kRgGateC = 8.0f;  // the constant of the recurrent gate, log a = -c r softplus

struct RgLayout {
  size_t embed = 0, lm_head = 0, final_gain = 0;
  std::vector<size_t> gain_t, gain_c, w_in, b_y, b_x, conv_w, conv_b, w_gate, b_a, b_i, lam,
      w_out, b_out, w_up, b_g, b_u, w_down, b_down;
  size_t conv_state = 0, rec_state = 0;  // [L][B][K-1][W], [L][B][W]
  size_t x = 0, h = 0, gy = 0, raw = 0, xc = 0, abuf = 0, gbuf = 0, o = 0, act = 0, hf = 0;
  size_t hend = 0, aprod = 0, chunks = 0, seq_chunk0 = 0;
  size_t splitk = 0, splitk_bytes = 0;
  size_t pval = 0, pidx = 0, cu = 0, row_seq = 0, last_row = 0, err = 0;
  size_t total = 0;
  int bw = 0, max_rows = 0, max_chunks = 0, n_parts = 0;
};

ll_status validate(const ll_rg_config *c) {
  if (!c) return fail(LL_ERR_INVALID_ARGUMENT, "cfg is NULL");
  if (c->n_layers < 1 || c->d_model < 1 || c->lru_width < 1 || c->n_heads < 1 ||
      c->mlp_width < 1 || c->d_conv < 1 || c->vocab < 1)
    return fail(LL_ERR_INVALID_ARGUMENT, "model dimensions must be positive");
  if (c->max_batch < 1 || c->max_prefill_tokens < 1)
    return fail(LL_ERR_INVALID_ARGUMENT, "capacities must be positive");
  if (!(c->rms_eps >= 0.f) || !std::isfinite(c->rms_eps))
    return fail(LL_ERR_INVALID_ARGUMENT, "rms_eps must be finite and >= 0");
  if (!std::isfinite(c->embed_scale))
    return fail(LL_ERR_INVALID_ARGUMENT, "embed_scale must be finite");
  if (!(c->logit_cap > 0.f) || !std::isfinite(c->logit_cap))
    return fail(LL_ERR_INVALID_ARGUMENT, "logit_cap must be finite and > 0");
  if (c->dtype != LL_F32 && c->dtype != LL_BF16)
    return fail(LL_ERR_UNSUPPORTED, "dtype %d unknown", c->dtype);
  if (c->lru_width % c->n_heads || (c->lru_width / c->n_heads) % 64)
    return fail(LL_ERR_UNSUPPORTED, "lru_width %d / n_heads %d: blocks must be multiples of 64",
                c->lru_width, c->n_heads);
  if (c->d_conv > 4) return fail(LL_ERR_UNSUPPORTED, "d_conv %d > 4", c->d_conv);
  if (c->d_model % 128) return fail(LL_ERR_UNSUPPORTED, "d_model %d not a multiple of 128", c->d_model);
  if (c->mlp_width % 64) return fail(LL_ERR_UNSUPPORTED, "mlp_width %d not a multiple of 64", c->mlp_width);
  if (c->vocab % 32) return fail(LL_ERR_UNSUPPORTED, "vocab %d not a multiple of 32", c->vocab);
  if (c->max_batch > LL_MAX_BATCH)
    return fail(LL_ERR_UNSUPPORTED, "max_batch %d > %d", c->max_batch, LL_MAX_BATCH);
  return LL_OK;
}

RgLayout make_layout(const ll_rg_config &c) {
  RgLayout L;
  const size_t eb = elem_bytes(c.dtype);
  const size_t d = c.d_model, W = c.lru_width, F = c.mlp_width;
  L.bw = c.lru_width / c.n_heads;
  L.max_rows = std::max(c.max_prefill_tokens, c.max_batch);
  L.max_chunks = (c.max_prefill_tokens + 15) / 16 + c.max_batch;
  L.n_parts = c.vocab / 32;
  const size_t K1 = std::max(c.d_conv - 1, 1);
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align_up(off + std::max<size_t>(bytes, 1));
    return o;
  };
  L.embed = take((size_t)c.vocab * d * eb);
  L.lm_head = take((size_t)c.vocab * d * eb);
  L.final_gain = take(d * eb);
  for (int l = 0; l < c.n_layers; ++l) {
    L.gain_t.push_back(take(d * eb));
    L.gain_c.push_back(take(d * eb));
    L.w_in.push_back(take(2 * W * d * eb));
    L.b_y.push_back(take(W * 4));
    L.b_x.push_back(take(W * 4));
    L.conv_w.push_back(take(W * c.d_conv * 4));
    L.conv_b.push_back(take(W * 4));
    L.w_gate.push_back(take(2 * W * L.bw * eb));
    L.b_a.push_back(take(W * 4));
    L.b_i.push_back(take(W * 4));
    L.lam.push_back(take(W * 4));
    L.w_out.push_back(take(d * W * eb));
    L.b_out.push_back(take(d * 4));
    L.w_up.push_back(take(2 * F * d * eb));
    L.b_g.push_back(take(F * 4));
    L.b_u.push_back(take(F * 4));
    L.w_down.push_back(take(d * F * eb));
    L.b_down.push_back(take(d * 4));
  }
  L.conv_state = take((size_t)c.n_layers * c.max_batch * K1 * W * 4);
  L.rec_state = take((size_t)c.n_layers * c.max_batch * W * 4);
  const size_t R = L.max_rows;
  L.x = take(R * d * 4);
  L.h = take(R * d * eb);
  L.gy = take(R * W * eb);
  L.raw = take(R * W * 4);
  L.xc = take(R * W * eb);
  L.abuf = take(R * W * 4);
  L.gbuf = take(R * W * 4);
  L.o = take(R * W * eb);
  L.act = take(R * F * eb);
  L.hf = take((size_t)c.max_batch * d * eb);
  L.hend = take((size_t)L.max_chunks * W * 4);
  L.aprod = take((size_t)L.max_chunks * W * 4);
  L.chunks = take((size_t)L.max_chunks * 16);
  L.seq_chunk0 = take((c.max_batch + 1) * 4);
  {
    // split-K workspaces of the GEMMs that may split (not the grouped gate GEMM)
    const int shapes[4][2] = {{(int)(2 * W), (int)d}, {(int)d, (int)W}, {(int)(2 * F), (int)d},
                              {(int)d, (int)F}};
    for (const auto &nk : shapes) {
      L.splitk_bytes = std::max(L.splitk_bytes, splitk_plan(eb, c.max_batch, nk[0], nk[1]).ws_bytes);
      const int mmax = std::min(c.max_prefill_tokens, 64 * kPrefillSplitMinTiles);
      for (int mr = 64; mr < mmax + 64; mr += 64) {
        const int mm = std::min(mr, mmax);
        L.splitk_bytes = std::max(L.splitk_bytes, prefill_splitk_plan(eb, mm, nk[0], nk[1]).ws_bytes);
      }
    }
    L.splitk = take(L.splitk_bytes);
  }
  L.pval = take((size_t)c.max_batch * L.n_parts * 4);
  L.pidx = take((size_t)c.max_batch * L.n_parts * 4);
  L.cu = take((c.max_batch + 1) * 4);
  L.row_seq = take(R * 4);
  L.last_row = take(c.max_batch * 4);
  L.err = take(4);
  L.total = off;
  return L;
}

}  // namespace

struct ll_rg : ll::StateModel {
  ll_rg_config cfg;
  RgLayout L;
  ll_rg() : StateModel("ll_rg_reset", false) {}
  size_t K1() const { return (size_t)std::max(cfg.d_conv - 1, 1); }
  float *conv_state(int l) const {
    return at<float>(L.conv_state) + (size_t)l * cfg.max_batch * K1() * cfg.lru_width;
  }
  float *rec_state(int l) const {
    return at<float>(L.rec_state) + (size_t)l * cfg.max_batch * cfg.lru_width;
  }
};

namespace {

struct PrefillPlan {
  int n_chunks = 0;
  bool multi = false;
  bool fresh = false;
  int batch = 0;
};

ll_status enqueue_layers(ll_rg *m, int rows, const PrefillPlan *pp, hipStream_t s) {
  const ll_rg_config &c = m->cfg;
  const RgLayout &L = m->L;
  const bool decode = pp == nullptr;
  const int d = c.d_model, W = c.lru_width, F = c.mlp_width, dt = c.dtype;
  const size_t eb = elem_bytes(dt);
  const bool fuse_norm = decode && rows <= kFusedNormMaxRows &&
                         skinny_norm_lds(eb, rows, d) <= kSkinnyMaxNormLds;
  float *x = m->at<float>(L.x);
  const bool use_split = decode ? m->opt[LL_OPT_DECODE_SPLITK] : m->opt[LL_OPT_PREFILL_SPLITK];
  float *gemm_ws = use_split && L.splitk_bytes ? m->at<float>(L.splitk) : nullptr;
  const size_t gemm_ws_bytes = gemm_ws ? L.splitk_bytes : 0;
  auto gemm = [&](const void *a, int lda, const NormIn *nrm, const void *wt, int n, int k,
                  const EpiParams &ep) {
    return decode ? launch_gemm_skinny(dt, a, lda, nrm, wt, rows, n, k, ep, s, gemm_ws,
                                       gemm_ws_bytes, nullptr, nullptr,
                                       m->opt[LL_OPT_DECODE_SPLITK] == 2 ? 2 : 1)
                  : launch_gemm_tiled(dt, a, lda, wt, rows, n, k, ep, s, gemm_ws, gemm_ws_bytes,
                                      m->opt[LL_OPT_PREFILL_TILE]);
  };
  // RMSNorm of the residual rows: inside the next GEMM (small decode batches) or a kernel
  auto norm_in = [&](size_t gain, NormIn *nrm) -> ll_status {
    if (fuse_norm) {
      *nrm = NormIn{x, d, nullptr, m->at(gain), c.rms_eps};
      return LL_OK;
    }
    m->mark(LL_RGK_RMSNORM);
    LL_HIP(launch_rmsnorm(dt, x, d, nullptr, rows, d, m->at(gain), c.rms_eps, m->at(L.h), d, s));
    return LL_OK;
  };
  for (int l = 0; l < c.n_layers; ++l) {
    NormIn nrm;
    ll_status st = norm_in(L.gain_t[l], &nrm);
    if (st != LL_OK) return st;
    // linear_y | linear_x with the gelu branch and (decode) the conv step in the epilogue
    m->mark(LL_RGK_IN_PROJ);
    EpiParams ei;
    ei.kind = kEpiRgIn;
    ei.act = m->at(L.gy);
    ei.bias = m->at<float>(L.b_y[l]);
    ei.bias2 = m->at<float>(L.b_x[l]);
    ei.width = W;
    ei.conv_k = c.d_conv;
    if (decode) {
      ei.act2 = m->at(L.xc);
      ei.conv_state = m->conv_state(l);
      ei.conv_w = m->at<float>(L.conv_w[l]);
      ei.conv_b = m->at<float>(L.conv_b[l]);
    } else {
      ei.out_f32 = m->at<float>(L.raw);
      ei.ld_out = W;
    }
    LL_HIP(gemm(m->at(L.h), d, fuse_norm ? &nrm : nullptr, m->at(L.w_in[l]), 2 * W, d, ei));
    if (!decode) {
      m->mark(LL_RGK_CONV);
      LL_HIP(launch_mamba_conv(dt, m->at<float>(L.raw), W, m->at<int>(L.row_seq),
                               m->at<int>(L.cu), m->conv_state(l), pp->fresh,
                               m->at<float>(L.conv_w[l]), m->at<float>(L.conv_b[l]), rows, W,
                               c.d_conv, m->at(L.xc), s, 0));
    }
    // RG-LRU gates on the block-diagonal weights (decode: + the recurrence step)
    m->mark(LL_RGK_GATES);
    EpiParams eg;
    eg.kind = kEpiRglru;
    eg.rg_x = m->at(L.xc);
    eg.bias = m->at<float>(L.b_a[l]);
    eg.bias2 = m->at<float>(L.b_i[l]);
    eg.lam = m->at<float>(L.lam[l]);
    eg.width = W;
    eg.group_n = 2 * L.bw;
    eg.group_k = L.bw;
    if (decode) {
      eg.rg_state = m->rec_state(l);
      eg.rg_gy = m->at(L.gy);
      eg.act = m->at(L.o);
    } else {
      eg.out_f32 = m->at<float>(L.abuf);
      eg.out2 = m->at<float>(L.gbuf);
      eg.row_seq = m->at<int>(L.row_seq);
      eg.cu = m->at<int>(L.cu);
      eg.rg_fresh = pp->fresh;
    }
    LL_HIP(gemm(m->at(L.xc), W, nullptr, m->at(L.w_gate[l]), 2 * W, L.bw, eg));
    if (!decode) {
      RgScanArgs a;
      a.a = m->at<float>(L.abuf);
      a.g = m->at<float>(L.gbuf);
      a.gy = m->at(L.gy);
      a.out = m->at(L.o);
      a.state = m->rec_state(l);
      a.hend = m->at<float>(L.hend);
      a.aprod = m->at<float>(L.aprod);
      a.chunks = m->at<int4>(L.chunks);
      a.seq_chunk0 = m->at<int>(L.seq_chunk0);
      a.cu = m->at<int>(L.cu);
      a.conv = m->conv_state(l);
      a.raw = m->at<float>(L.raw);
      a.ld_raw = W;
      a.W = W;
      a.K = c.d_conv;
      a.fresh = pp->fresh;
      if (pp->multi) {
        m->mark(LL_RGK_SCAN_CHUNK);
        LL_HIP(launch_rg_scan_chunks(a, pp->n_chunks, s));
      }
      m->mark(LL_RGK_SCAN);
      LL_HIP(launch_rg_scan_out(dt, a, pp->n_chunks, s));
    }
    m->mark(LL_RGK_OUT_PROJ);
    EpiParams eo;
    eo.kind = kEpiBiasResid;
    eo.out_f32 = x;
    eo.ld_out = d;
    eo.bias = m->at<float>(L.b_out[l]);
    LL_HIP(gemm(m->at(L.o), W, nullptr, m->at(L.w_out[l]), d, W, eo));
    // MLP: GeGLU with biases
    if ((st = norm_in(L.gain_c[l], &nrm)) != LL_OK) return st;
    m->mark(LL_RGK_MLP_UP);
    EpiParams eu;
    eu.kind = kEpiGeglu;
    eu.act = m->at(L.act);
    eu.ld_act = F;
    eu.bias = m->at<float>(L.b_g[l]);
    eu.bias2 = m->at<float>(L.b_u[l]);
    LL_HIP(gemm(m->at(L.h), d, fuse_norm ? &nrm : nullptr, m->at(L.w_up[l]), 2 * F, d, eu));
    m->mark(LL_RGK_MLP_DOWN);
    EpiParams ed;
    ed.kind = kEpiBiasResid;
    ed.out_f32 = x;
    ed.ld_out = d;
    ed.bias = m->at<float>(L.b_down[l]);
    LL_HIP(gemm(m->at(L.act), F, nullptr, m->at(L.w_down[l]), d, F, ed));
  }
  return LL_OK;
}

ll_status enqueue_head(ll_rg *m, int batch, const int *rowmap, int *next, float *logits,
                       hipStream_t s) {
  const ll_rg_config &c = m->cfg;
  const RgLayout &L = m->L;
  EpiParams ep;
  ep.kind = kEpiArgmax;
  ep.out_f32 = logits;
  ep.ld_out = c.vocab;
  ep.part_val = m->at<float>(L.pval);
  ep.part_idx = m->at<int>(L.pidx);
  ep.n_parts = L.n_parts;
  NormIn nrm{m->at<float>(L.x), c.d_model, rowmap, m->at(L.final_gain), c.rms_eps};
  const bool fuse_norm = batch <= kFusedNormMaxRows &&
                         skinny_norm_lds(elem_bytes(c.dtype), batch, c.d_model) <= kSkinnyMaxNormLds;
  if (!fuse_norm) {
    m->mark(LL_RGK_RMSNORM);
    LL_HIP(launch_rmsnorm(c.dtype, m->at<float>(L.x), c.d_model, rowmap, batch, c.d_model,
                          m->at(L.final_gain), c.rms_eps, m->at(L.hf), c.d_model, s));
  }
  // the argmax of the capped logits is that of the raw ones (cap * tanh(l / cap) increases)
  m->mark(LL_RGK_LM_HEAD);
  LL_HIP(launch_gemm_skinny(c.dtype, m->at(L.hf), c.d_model, fuse_norm ? &nrm : nullptr,
                            m->at(L.lm_head), batch, c.vocab, c.d_model, ep, s));
  m->mark(LL_RGK_ARGMAX);
  LL_HIP(launch_argmax_reduce(ep.part_val, ep.part_idx, batch, ep.n_parts, next, nullptr, s));
  if (logits) {
    m->mark(LL_RGK_SOFTCAP);
    LL_HIP(launch_softcap(logits, (long)batch * c.vocab, c.logit_cap, s));
  }
  return LL_OK;
}

ll_status enqueue_decode(ll_rg *m, const int32_t *in, int32_t *out, float *logits,
                         hipStream_t s) {
  const ll_rg_config &c = m->cfg;
  m->mark(LL_RGK_EMBED);
  LL_HIP(launch_embed(c.dtype, in, m->batch, m->at(m->L.embed), c.vocab, c.d_model,
                      m->at<float>(m->L.x), m->at<int>(m->L.err), s, c.embed_scale));
  ll_status st = enqueue_layers(m, m->batch, nullptr, s);
  if (st != LL_OK) return st;
  return enqueue_head(m, m->batch, nullptr, out, logits, s);
}

}  // namespace

extern "C" {

ll_status ll_rg_workspace_size(const ll_rg_config *cfg, size_t *bytes) {
  g_err.clear();
  if (!bytes) return fail(LL_ERR_INVALID_ARGUMENT, "bytes is NULL");
  ll_status st = validate(cfg);
  if (st != LL_OK) return st;
  *bytes = make_layout(*cfg).total;
  return LL_OK;
}

ll_status ll_rg_load(const ll_rg_config *cfg, const ll_rg_weights *w, void *workspace,
                     size_t workspace_bytes, void *hip_stream, ll_rg **out) {
  g_err.clear();
  if (!out) return fail(LL_ERR_INVALID_ARGUMENT, "out is NULL");
  *out = nullptr;
  ll_status st = validate(cfg);
  if (st != LL_OK) return st;
  if (!w) return fail(LL_ERR_INVALID_ARGUMENT, "weights is NULL");
  if (!w->embed || !w->final_norm) return fail(LL_ERR_INVALID_ARGUMENT, "embed and final_norm must be set");
  const void *const *arrays[] = {
      w->norm_t, w->linear_y, (const void *const *)w->linear_y_b, w->linear_x,
      (const void *const *)w->linear_x_b, (const void *const *)w->conv_w,
      (const void *const *)w->conv_b, w->gate_a, (const void *const *)w->gate_a_b, w->gate_x,
      (const void *const *)w->gate_x_b, (const void *const *)w->lambda, w->linear_out,
      (const void *const *)w->linear_out_b, w->norm_c, w->mlp_gate,
      (const void *const *)w->mlp_gate_b, w->mlp_up, (const void *const *)w->mlp_up_b,
      w->mlp_down, (const void *const *)w->mlp_down_b};
  for (auto a : arrays) {
    if (!a) return fail(LL_ERR_INVALID_ARGUMENT, "a per-layer weight array is NULL");
    for (int l = 0; l < cfg->n_layers; ++l)
      if (!a[l]) return fail(LL_ERR_INVALID_ARGUMENT, "layer %d weight pointer is NULL", l);
  }
  if ((st = check_ws(workspace)) != LL_OK) return st;
  const RgLayout L = make_layout(*cfg);
  if (workspace_bytes < L.total)
    return fail(LL_ERR_WORKSPACE, "workspace has %zu bytes, needs %zu", workspace_bytes, L.total);

  ll_rg *m = new ll_rg();
  m->cfg = *cfg;
  m->L = L;
  m->ws = reinterpret_cast<char *>(workspace);
  m->stream = reinterpret_cast<hipStream_t>(hip_stream);
  const ll_rg_config &c = *cfg;
  const size_t eb = elem_bytes(c.dtype);
  const int d = c.d_model, W = c.lru_width, F = c.mlp_width, H = c.n_heads, bw = L.bw;
  hipStream_t s = m->stream;
  auto bail = [&](ll_status e) {
    delete m;
    return e;
  };
#define LOAD_HIP(expr)                                                                    \
  do {                                                                                    \
    hipError_t e_ = (expr);                                                               \
    if (e_ != hipSuccess)                                                                 \
      return bail(fail(LL_ERR_HIP, "%s failed: %s", #expr, hipGetErrorString(e_)));       \
  } while (0)
  auto copy = [&](size_t dst, const void *src, size_t bytes) {
    return hipMemcpyAsync(m->at(dst), src, bytes, hipMemcpyDeviceToDevice, s);
  };
  LOAD_HIP(copy(L.embed, w->embed, (size_t)c.vocab * d * eb));
  RepackSrc lm{{w->embed, nullptr, nullptr}, {c.vocab, 0, 0}};
  LOAD_HIP(launch_repack(c.dtype, lm, c.vocab, d, kPermNone, 64, 64, m->at(L.lm_head), s));
  LOAD_HIP(launch_rg_prep(c.dtype, w->final_norm, w->final_norm, d, nullptr, 0, kRgGateC,
                          m->at(L.final_gain), m->at(L.final_gain), nullptr, s));
  for (int l = 0; l < c.n_layers; ++l) {
    LOAD_HIP(launch_rg_prep(c.dtype, w->norm_t[l], w->norm_c[l], d, w->lambda[l], W, kRgGateC,
                            m->at(L.gain_t[l]), m->at(L.gain_c[l]), m->at<float>(L.lam[l]), s));
    RepackSrc in{{w->linear_y[l], w->linear_x[l], nullptr}, {W, W, 0}};
    LOAD_HIP(launch_repack(c.dtype, in, 2 * W, d, kPermNone, 64, 64, m->at(L.w_in[l]), s));
    // gate blocks, head by head: recurrence-gate and input-gate rows interleaved per 16
    for (int k = 0; k < H; ++k) {
      const size_t blk = (size_t)k * bw * bw * eb;
      RepackSrc g{{reinterpret_cast<const char *>(w->gate_a[l]) + blk,
                   reinterpret_cast<const char *>(w->gate_x[l]) + blk, nullptr},
                  {bw, bw, 0}};
      LOAD_HIP(launch_repack(c.dtype, g, 2 * bw, bw, kPermGlu, 64, bw,
                             m->at<char>(L.w_gate[l]) + 2 * blk, s));
    }
    RepackSrc op{{w->linear_out[l], nullptr, nullptr}, {d, 0, 0}};
    LOAD_HIP(launch_repack(c.dtype, op, d, W, kPermNone, 64, 64, m->at(L.w_out[l]), s));
    RepackSrc up{{w->mlp_gate[l], w->mlp_up[l], nullptr}, {F, F, 0}};
    LOAD_HIP(launch_repack(c.dtype, up, 2 * F, d, kPermGlu, 64, F, m->at(L.w_up[l]), s));
    RepackSrc dn{{w->mlp_down[l], nullptr, nullptr}, {d, 0, 0}};
    LOAD_HIP(launch_repack(c.dtype, dn, d, F, kPermNone, 64, 64, m->at(L.w_down[l]), s));
    LOAD_HIP(copy(L.b_y[l], w->linear_y_b[l], (size_t)W * 4));
    LOAD_HIP(copy(L.b_x[l], w->linear_x_b[l], (size_t)W * 4));
    LOAD_HIP(copy(L.conv_w[l], w->conv_w[l], (size_t)W * c.d_conv * 4));
    LOAD_HIP(copy(L.conv_b[l], w->conv_b[l], (size_t)W * 4));
    LOAD_HIP(copy(L.b_a[l], w->gate_a_b[l], (size_t)W * 4));
    LOAD_HIP(copy(L.b_i[l], w->gate_x_b[l], (size_t)W * 4));
    LOAD_HIP(copy(L.b_out[l], w->linear_out_b[l], (size_t)d * 4));
    LOAD_HIP(copy(L.b_g[l], w->mlp_gate_b[l], (size_t)F * 4));
    LOAD_HIP(copy(L.b_u[l], w->mlp_up_b[l], (size_t)F * 4));
    LOAD_HIP(copy(L.b_down[l], w->mlp_down_b[l], (size_t)d * 4));
  }
  LOAD_HIP(hipMemsetAsync(m->at(L.err), 0, 4, s));
#undef LOAD_HIP
  *out = m;
  return LL_OK;
}

ll_status ll_rg_prefill(ll_rg *m, int32_t batch, const int32_t *seq_lens_host,
                        const int32_t *tokens_dev, int32_t *next_tokens_dev, float *logits_dev) {
  g_err.clear();
  if (!m) return fail(LL_ERR_INVALID_ARGUMENT, "model is NULL");
  if (!seq_lens_host || !tokens_dev || !next_tokens_dev)
    return fail(LL_ERR_INVALID_ARGUMENT, "seq_lens_host, tokens_dev and next_tokens_dev must be set");
  const ll_rg_config &c = m->cfg;
  long total = 0;
  ll_status vst = m->check_prefill(batch, seq_lens_host, c.max_batch, c.max_prefill_tokens, &total);
  if (vst != LL_OK) return vst;
  const bool cont = m->batch != 0;
  int max_len = 0;
  MambaMeta mm;
  mm.batch = batch;
  for (int b = 0; b < batch; ++b) {
    max_len = std::max(max_len, (int)seq_lens_host[b]);
    mm.lens[b] = seq_lens_host[b];
  }
  const int T = (int)total;
  const int clen = rg_chunk_len(max_len);
  PrefillPlan pp;
  pp.fresh = !cont;
  pp.batch = batch;
  for (int b = 0; b < batch; ++b) {
    const int n = (mm.lens[b] + clen - 1) / clen;
    pp.n_chunks += n;
    pp.multi = pp.multi || n > 1;
  }
  if (pp.n_chunks > m->L.max_chunks)
    return fail(LL_ERR_CAPACITY, "%d scan chunks > %d", pp.n_chunks, m->L.max_chunks);
  hipStream_t s = m->stream;
  const RgLayout &L = m->L;
  TimerScope scope(m->timer, 0);
  m->mark(LL_RGK_META);
  LL_HIP(launch_mamba_meta(mm, T, clen, m->at<int>(L.cu), m->at<int>(L.row_seq),
                           m->at<int>(L.last_row), m->at<int4>(L.chunks),
                           m->at<int>(L.seq_chunk0), s));
  m->mark(LL_RGK_EMBED);
  LL_HIP(launch_embed(c.dtype, tokens_dev, T, m->at(L.embed), c.vocab, c.d_model,
                      m->at<float>(L.x), m->at<int>(L.err), s, c.embed_scale));
  ll_status st = enqueue_layers(m, T, &pp, s);
  if (st != LL_OK) return st;
  st = enqueue_head(m, batch, m->at<int>(L.last_row), next_tokens_dev, logits_dev, s);
  if (st != LL_OK) return st;
  m->commit_prefill(batch, seq_lens_host);
  return LL_OK;
}

ll_status ll_rg_decode_step(ll_rg *m, const int32_t *in_tokens_dev, int32_t *next_tokens_dev,
                            float *logits_dev) {
  g_err.clear();
  if (!m) return fail(LL_ERR_INVALID_ARGUMENT, "model is NULL");
  if (!in_tokens_dev || !next_tokens_dev)
    return fail(LL_ERR_INVALID_ARGUMENT, "in_tokens_dev and next_tokens_dev must be set");
  return m->decode(in_tokens_dev, next_tokens_dev, logits_dev, [&](hipStream_t s) {
    return enqueue_decode(m, in_tokens_dev, next_tokens_dev, logits_dev, s);
  });
}

ll_status ll_rg_reset(ll_rg *m) {
  g_err.clear();
  if (!m) return fail(LL_ERR_INVALID_ARGUMENT, "model is NULL");
  return m->reset();
}

ll_status ll_rg_seq_lengths(const ll_rg *m, int32_t *out, int32_t cap, int32_t *n) {
  g_err.clear();
  if (!m) return fail(LL_ERR_INVALID_ARGUMENT, "model is NULL");
  return m->seq_lengths(out, cap, n);
}

ll_status ll_rg_set_option(ll_rg *m, int32_t option, int32_t value) {
  g_err.clear();
  if (!m) return fail(LL_ERR_INVALID_ARGUMENT, "model is NULL");
  return m->set_option(option, value);
}

ll_status ll_rg_get_option(const ll_rg *m, int32_t option, int32_t *value) {
  g_err.clear();
  if (!m) return fail(LL_ERR_INVALID_ARGUMENT, "model is NULL");
  return m->get_option(option, value);
}

ll_status ll_rg_device_flags(ll_rg *m, int32_t *flags) {
  g_err.clear();
  if (!m) return fail(LL_ERR_INVALID_ARGUMENT, "model is NULL");
  return m->device_flags(m->L.err, flags);
}

ll_status ll_rg_set_kernel_timing(ll_rg *m, int32_t enable) {
  g_err.clear();
  if (!m) return fail(LL_ERR_INVALID_ARGUMENT, "model is NULL");
  return m->set_kernel_timing(enable);
}

ll_status ll_rg_kernel_timing_read(ll_rg *m, int32_t *counts, double *ms) {
  g_err.clear();
  if (!m) return fail(LL_ERR_INVALID_ARGUMENT, "model is NULL");
  return m->kernel_timing_read(LL_RGK_COUNT, counts, ms);
}

const char *ll_rg_kernel_class_name(int32_t cls) {
  return (cls >= 0 && cls < LL_RGK_COUNT) ? kRgClassNames[cls] : "";
}

void ll_rg_free(ll_rg *m) { delete m; }

}  // extern "C"
