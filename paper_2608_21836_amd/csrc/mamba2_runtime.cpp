// C-ABI runtime of the Mamba2 model: config validation, workspace layout, weight repacking,
// prefill / decode dispatch with explicit conv and SSM state, decode-step HIP graphs.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <vector>

#include "kernels.h"
#include "ll.h"
#include "ll_mamba2.h"
#include "runtime_common.h"

using namespace ll;

namespace {

const char *const kM2ClassNames[LL_M2K_COUNT] = {
    "prefill_meta", "embed",      "rmsnorm", "in_proj",    "conv_silu",      "scan_chunk",
    "scan_carry",   "scan",       "gated_rmsnorm", "out_proj_resid", "lm_head_argmax",
    "argmax_reduce"};

constexpr int kFusedNormMaxRows = 16;

struct M2Layout {
  size_t embed = 0, lm_head = 0, final_norm = 0;
  std::vector<size_t> norm, w_in, conv_w, conv_b, dt_b, A2, D, gnorm, w_out;
  size_t conv_state = 0, ssm_state = 0;  // [L][B][K-1][CD], [L][B][H][P][N]
  size_t x = 0, h = 0, zxd = 0, xbc = 0, g = 0, hn = 0, hf = 0;
  size_t hloc = 0, dtsum = 0, chunks = 0, seq_chunk0 = 0;
  size_t splitk = 0, splitk_bytes = 0;
  size_t pval = 0, pidx = 0, cu = 0, row_seq = 0, last_row = 0, err = 0;
  size_t total = 0;
  int H = 0, CD = 0, NZ = 0, max_rows = 0, max_chunks = 0, n_parts = 0;
};

ll_status validate(const ll_mamba2_config *c) {
  if (!c) return fail(LL_ERR_INVALID_ARGUMENT, "cfg is NULL");
  if (c->n_layers < 1 || c->d_model < 1 || c->d_inner < 1 || c->d_state < 1 || c->head_dim < 1 ||
      c->n_groups < 1 || c->d_conv < 1 || c->vocab < 1)
    return fail(LL_ERR_INVALID_ARGUMENT, "model dimensions must be positive");
  if (c->max_batch < 1 || c->max_prefill_tokens < 1)
    return fail(LL_ERR_INVALID_ARGUMENT, "capacities must be positive");
  if (!(c->rms_eps >= 0.f) || !std::isfinite(c->rms_eps))
    return fail(LL_ERR_INVALID_ARGUMENT, "rms_eps must be finite and >= 0");
  if (c->dtype != LL_F32 && c->dtype != LL_BF16)
    return fail(LL_ERR_UNSUPPORTED, "dtype %d unknown", c->dtype);
  const int N = c->d_state;
  if (N != 32 && N != 64 && N != 128 && N != 256)
    return fail(LL_ERR_UNSUPPORTED, "d_state %d not in {32, 64, 128, 256}", N);
  if (c->head_dim % kM2Rows || c->d_inner % c->head_dim)
    return fail(LL_ERR_UNSUPPORTED, "head_dim %d: a multiple of 16 dividing d_inner", c->head_dim);
  if ((c->d_inner / c->head_dim) % c->n_groups)
    return fail(LL_ERR_UNSUPPORTED, "n_groups %d does not divide the head count", c->n_groups);
  if (c->d_conv > 4) return fail(LL_ERR_UNSUPPORTED, "d_conv %d > 4", c->d_conv);
  if (c->d_model % 128) return fail(LL_ERR_UNSUPPORTED, "d_model %d not a multiple of 128", c->d_model);
  if (c->d_inner % 64) return fail(LL_ERR_UNSUPPORTED, "d_inner %d not a multiple of 64", c->d_inner);
  if (c->vocab % 32) return fail(LL_ERR_UNSUPPORTED, "vocab %d not a multiple of 32", c->vocab);
  if (c->max_batch > LL_MAX_BATCH)
    return fail(LL_ERR_UNSUPPORTED, "max_batch %d > %d", c->max_batch, LL_MAX_BATCH);
  return LL_OK;
}

// 16-bit models run the prefill scan in its matrix form on MFMA (fp16 operands); fp32 models
// keep the fp32 step recurrence.
bool use_ssd(const ll_mamba2_config &c) {
  return c.dtype != LL_F32 && mamba2_ssd_ok(c.head_dim, c.d_state);
}

M2Layout make_layout(const ll_mamba2_config &c) {
  M2Layout L;
  const size_t eb = elem_bytes(c.dtype);
  const size_t d = c.d_model, di = c.d_inner, N = c.d_state, P = c.head_dim;
  L.H = c.d_inner / c.head_dim;
  L.CD = c.d_inner + 2 * c.n_groups * c.d_state;
  L.NZ = (c.d_inner + L.CD + L.H + 127) / 128 * 128;  // in_proj rows padded to 128 columns
  L.max_rows = std::max(c.max_prefill_tokens, c.max_batch);
  L.max_chunks = mamba2_max_chunks(c.max_prefill_tokens, c.max_batch, L.H, c.head_dim);
  if (use_ssd(c))
    L.max_chunks = std::max(L.max_chunks, (c.max_prefill_tokens + kM2SsdChunk - 1) / kM2SsdChunk +
                                              c.max_batch);
  L.n_parts = c.vocab / 32;
  const size_t K1 = std::max(c.d_conv - 1, 1), H = L.H, CD = L.CD, NZ = L.NZ;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align_up(off + std::max<size_t>(bytes, 1));
    return o;
  };
  L.embed = take((size_t)c.vocab * d * eb);
  L.lm_head = take((size_t)c.vocab * d * eb);
  L.final_norm = take(d * eb);
  for (int l = 0; l < c.n_layers; ++l) {
    L.norm.push_back(take(d * eb));
    L.w_in.push_back(take(NZ * d * eb));
    L.conv_w.push_back(take(CD * c.d_conv * 4));
    L.conv_b.push_back(take(CD * 4));
    L.dt_b.push_back(take(H * 4));
    L.A2.push_back(take(H * 4));
    L.D.push_back(take(H * 4));
    L.gnorm.push_back(take(di * eb));
    L.w_out.push_back(take(d * di * eb));
  }
  L.conv_state = take((size_t)c.n_layers * c.max_batch * K1 * CD * 4);
  L.ssm_state = take((size_t)c.n_layers * c.max_batch * H * P * N * 4);
  const size_t R = L.max_rows;
  L.x = take(R * d * 4);
  L.h = take(R * d * eb);
  L.zxd = take(R * NZ * 4);
  L.xbc = take(R * CD * 4);
  L.g = take(R * di * 4);
  L.hn = take(R * di * eb);
  L.hf = take((size_t)c.max_batch * d * eb);
  L.hloc = take((size_t)L.max_chunks * H * P * N * 4);
  L.dtsum = take((size_t)L.max_chunks * H * 4);
  L.chunks = take((size_t)L.max_chunks * 16);
  L.seq_chunk0 = take((c.max_batch + 1) * 4);
  {
    const int shapes[2][2] = {{(int)NZ, (int)d}, {(int)d, (int)di}};
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

struct ll_mamba2 : ll::StateModel {
  ll_mamba2_config cfg;
  M2Layout L;
  ll_mamba2() : StateModel("ll_mamba2_reset", false) {}
  size_t K1() const { return (size_t)std::max(cfg.d_conv - 1, 1); }
  float *conv_state(int l) const {
    return at<float>(L.conv_state) + (size_t)l * cfg.max_batch * K1() * L.CD;
  }
  float *ssm_state(int l) const {
    return at<float>(L.ssm_state) +
           (size_t)l * cfg.max_batch * L.H * cfg.head_dim * cfg.d_state;
  }
};

namespace {

struct PrefillPlan {
  int n_chunks = 0;
  bool multi = false;
  bool fresh = false;
  int batch = 0;
};

M2ScanArgs scan_args(const ll_mamba2 *m, int l) {
  const ll_mamba2_config &c = m->cfg;
  const M2Layout &L = m->L;
  M2ScanArgs a;
  a.zxd = m->at<float>(L.zxd);
  a.ldz = L.NZ;
  a.dt_col = c.d_inner + L.CD;
  a.xbc = m->at<float>(L.xbc);
  a.dt_b = m->at<float>(L.dt_b[l]);
  a.A2 = m->at<float>(L.A2[l]);
  a.D = m->at<float>(L.D[l]);
  a.ssm = m->ssm_state(l);
  a.g = m->at<float>(L.g);
  a.hloc = m->at<float>(L.hloc);
  a.dtsum = m->at<float>(L.dtsum);
  a.conv = m->conv_state(l);
  a.conv_col = c.d_inner;
  a.conv_n = L.CD;
  a.K = c.d_conv;
  a.di = c.d_inner;
  a.H = L.H;
  a.P = c.head_dim;
  a.N = c.d_state;
  a.G = c.n_groups;
  return a;
}

ll_status enqueue_layers(ll_mamba2 *m, int rows, const PrefillPlan *pp, hipStream_t s,
                         bool *hf_ready) {
  *hf_ready = false;
  const ll_mamba2_config &c = m->cfg;
  const M2Layout &L = m->L;
  const bool decode = pp == nullptr;
  const int d = c.d_model, di = c.d_inner, dt = c.dtype;
  const size_t eb = elem_bytes(dt);
  const bool fuse_norm = decode && rows <= kFusedNormMaxRows &&
                         skinny_norm_lds(eb, rows, d) <= kSkinnyMaxNormLds;
  const bool fuse_gnorm = decode && rows <= kFusedNormMaxRows &&
                          skinny_norm_lds(eb, rows, di) <= kSkinnyMaxNormLds;
  float *x = m->at<float>(L.x);
  const bool use_split = decode ? m->opt[LL_OPT_DECODE_SPLITK] : m->opt[LL_OPT_PREFILL_SPLITK];
  float *gemm_ws = use_split && L.splitk_bytes ? m->at<float>(L.splitk) : nullptr;
  const size_t gemm_ws_bytes = gemm_ws ? L.splitk_bytes : 0;
  auto gemm = [&](const void *a, int lda, const NormIn *nrm, const void *wt, int n, int k,
                  const EpiParams &ep, const PostNorm *post = nullptr, bool *post_done = nullptr) {
    return decode ? launch_gemm_skinny(dt, a, lda, nrm, wt, rows, n, k, ep, s, gemm_ws,
                                       gemm_ws_bytes, post, post_done,
                                       m->opt[LL_OPT_DECODE_SPLITK] == 2 ? 2 : 1)
                  : launch_gemm_tiled(dt, a, lda, wt, rows, n, k, ep, s, gemm_ws, gemm_ws_bytes,
                                      m->opt[LL_OPT_PREFILL_TILE]);
  };
  bool h_ready = false;
  for (int l = 0; l < c.n_layers; ++l) {
    NormIn nrm;
    if (fuse_norm) {
      nrm = NormIn{x, d, nullptr, m->at(L.norm[l]), c.rms_eps};
    } else if (!h_ready) {
      m->mark(LL_M2K_RMSNORM);
      LL_HIP(launch_rmsnorm(dt, x, d, nullptr, rows, d, m->at(L.norm[l]), c.rms_eps, m->at(L.h),
                            d, s));
    }
    h_ready = false;
    M2ScanArgs a = scan_args(m, l);
    m->mark(LL_M2K_IN_PROJ);
    if (decode) {
      // the conv step in the in_proj epilogue; z and dt stay in zxd
      EpiParams ep;
      ep.kind = kEpiConvF32;
      ep.act = m->at(L.xbc);
      ep.out_f32 = m->at<float>(L.zxd);
      ep.ld_out = L.NZ;
      ep.conv_state = m->conv_state(l);
      ep.conv_w = m->at<float>(L.conv_w[l]);
      ep.conv_b = m->at<float>(L.conv_b[l]);
      ep.conv_k = c.d_conv;
      ep.conv_col0 = di;
      ep.conv_n = L.CD;
      LL_HIP(gemm(m->at(L.h), d, fuse_norm ? &nrm : nullptr, m->at(L.w_in[l]), L.NZ, d, ep));
      a.carry = 1;
      m->mark(LL_M2K_SCAN);
      LL_HIP(launch_m2_scan_out(a, rows, s));
    } else {
      EpiParams ep;
      ep.kind = kEpiStore;
      ep.out_f32 = m->at<float>(L.zxd);
      ep.ld_out = L.NZ;
      LL_HIP(gemm(m->at(L.h), d, nullptr, m->at(L.w_in[l]), L.NZ, d, ep));
      m->mark(LL_M2K_CONV);
      LL_HIP(launch_mamba_conv(kF32, m->at<float>(L.zxd) + di, L.NZ, m->at<int>(L.row_seq),
                               m->at<int>(L.cu), m->conv_state(l), pp->fresh,
                               m->at<float>(L.conv_w[l]), m->at<float>(L.conv_b[l]), rows, L.CD,
                               c.d_conv, m->at(L.xbc), s));
      a.chunks = m->at<int4>(L.chunks);
      a.seq_chunk0 = m->at<int>(L.seq_chunk0);
      a.cu = m->at<int>(L.cu);
      a.fresh = pp->fresh;
      a.update_conv = 1;
      a.mfma = use_ssd(c);
      if (pp->multi) {
        m->mark(LL_M2K_SCAN_CHUNK);
        LL_HIP(launch_m2_scan_chunks(a, pp->n_chunks, s));
        m->mark(LL_M2K_SCAN_CARRY);
        LL_HIP(launch_m2_scan_carry(a, pp->batch, s));
        a.carry = 2;
      } else {
        a.carry = pp->fresh ? 0 : 1;
      }
      m->mark(LL_M2K_SCAN);
      LL_HIP(launch_m2_scan_out(a, pp->n_chunks, s));
    }
    // gated RMSNorm of g, then out_proj with the residual add
    NormIn gn{m->at<float>(L.g), di, nullptr, m->at(L.gnorm[l]), c.rms_eps};
    if (!fuse_gnorm) {
      m->mark(LL_M2K_GNORM);
      LL_HIP(launch_rmsnorm(dt, m->at<float>(L.g), di, nullptr, rows, di, m->at(L.gnorm[l]),
                            c.rms_eps, m->at(L.hn), di, s));
    }
    m->mark(LL_M2K_OUT_PROJ);
    const bool last = l + 1 == c.n_layers;
    PostNorm pn;
    pn.gain = m->at(last ? L.final_norm : L.norm[l + 1]);
    pn.eps = c.rms_eps;
    pn.out = m->at(last ? L.hf : L.h);
    pn.ld_out = d;
    bool done = false;
    EpiParams er;
    er.kind = kEpiResid;
    er.out_f32 = x;
    er.ld_out = d;
    LL_HIP(gemm(m->at(L.hn), di, fuse_gnorm ? &gn : nullptr, m->at(L.w_out[l]), d, di, er,
                (decode && !fuse_norm && !fuse_gnorm) ? &pn : nullptr, &done));
    if (last) *hf_ready = done;
    else h_ready = done;
  }
  return LL_OK;
}

ll_status enqueue_head(ll_mamba2 *m, int batch, const int *rowmap, int *next, float *logits,
                       hipStream_t s, bool hf_ready) {
  const ll_mamba2_config &c = m->cfg;
  const M2Layout &L = m->L;
  EpiParams ep;
  ep.kind = kEpiArgmax;
  ep.out_f32 = logits;
  ep.ld_out = c.vocab;
  ep.part_val = m->at<float>(L.pval);
  ep.part_idx = m->at<int>(L.pidx);
  ep.n_parts = L.n_parts;
  NormIn nrm{m->at<float>(L.x), c.d_model, rowmap, m->at(L.final_norm), c.rms_eps};
  const bool fuse_norm = batch <= kFusedNormMaxRows &&
                         skinny_norm_lds(elem_bytes(c.dtype), batch, c.d_model) <= kSkinnyMaxNormLds;
  if (!fuse_norm && !hf_ready) {
    m->mark(LL_M2K_RMSNORM);
    LL_HIP(launch_rmsnorm(c.dtype, m->at<float>(L.x), c.d_model, rowmap, batch, c.d_model,
                          m->at(L.final_norm), c.rms_eps, m->at(L.hf), c.d_model, s));
  }
  m->mark(LL_M2K_LM_HEAD);
  LL_HIP(launch_gemm_skinny(c.dtype, m->at(L.hf), c.d_model, fuse_norm ? &nrm : nullptr,
                            m->at(L.lm_head), batch, c.vocab, c.d_model, ep, s));
  m->mark(LL_M2K_ARGMAX);
  LL_HIP(launch_argmax_reduce(ep.part_val, ep.part_idx, batch, ep.n_parts, next, nullptr, s));
  return LL_OK;
}

ll_status enqueue_decode(ll_mamba2 *m, const int32_t *in, int32_t *out, float *logits,
                         hipStream_t s) {
  const ll_mamba2_config &c = m->cfg;
  m->mark(LL_M2K_EMBED);
  LL_HIP(launch_embed(c.dtype, in, m->batch, m->at(m->L.embed), c.vocab, c.d_model,
                      m->at<float>(m->L.x), m->at<int>(m->L.err), s));
  bool hf_ready = false;
  ll_status st = enqueue_layers(m, m->batch, nullptr, s, &hf_ready);
  if (st != LL_OK) return st;
  return enqueue_head(m, m->batch, nullptr, out, logits, s, hf_ready);
}

}  // namespace

extern "C" {

ll_status ll_mamba2_workspace_size(const ll_mamba2_config *cfg, size_t *bytes) {
  g_err.clear();
  if (!bytes) return fail(LL_ERR_INVALID_ARGUMENT, "bytes is NULL");
  ll_status st = validate(cfg);
  if (st != LL_OK) return st;
  *bytes = make_layout(*cfg).total;
  return LL_OK;
}

ll_status ll_mamba2_load(const ll_mamba2_config *cfg, const ll_mamba2_weights *w, void *workspace,
                         size_t workspace_bytes, void *hip_stream, ll_mamba2 **out) {
  g_err.clear();
  if (!out) return fail(LL_ERR_INVALID_ARGUMENT, "out is NULL");
  *out = nullptr;
  ll_status st = validate(cfg);
  if (st != LL_OK) return st;
  if (!w) return fail(LL_ERR_INVALID_ARGUMENT, "weights is NULL");
  if (!w->embed || !w->final_norm) return fail(LL_ERR_INVALID_ARGUMENT, "embed and final_norm must be set");
  const void *const *arrays[] = {w->norm, w->in_proj, (const void *const *)w->conv_w,
                                 (const void *const *)w->conv_b, (const void *const *)w->dt_b,
                                 (const void *const *)w->A_log, (const void *const *)w->D,
                                 w->gnorm, w->out_proj};
  for (auto a : arrays) {
    if (!a) return fail(LL_ERR_INVALID_ARGUMENT, "a per-layer weight array is NULL");
    for (int l = 0; l < cfg->n_layers; ++l)
      if (!a[l]) return fail(LL_ERR_INVALID_ARGUMENT, "layer %d weight pointer is NULL", l);
  }
  if ((st = check_ws(workspace)) != LL_OK) return st;
  const M2Layout L = make_layout(*cfg);
  if (workspace_bytes < L.total)
    return fail(LL_ERR_WORKSPACE, "workspace has %zu bytes, needs %zu", workspace_bytes, L.total);

  ll_mamba2 *m = new ll_mamba2();
  m->cfg = *cfg;
  m->L = L;
  m->ws = reinterpret_cast<char *>(workspace);
  m->stream = reinterpret_cast<hipStream_t>(hip_stream);
  const ll_mamba2_config &c = *cfg;
  const size_t eb = elem_bytes(c.dtype);
  const int d = c.d_model, di = c.d_inner;
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
  LOAD_HIP(copy(L.final_norm, w->final_norm, d * eb));
  RepackSrc lm{{w->embed, nullptr, nullptr}, {c.vocab, 0, 0}};
  LOAD_HIP(launch_repack(c.dtype, lm, c.vocab, d, kPermNone, 64, 64, m->at(L.lm_head), s));
  const int in_rows = di + L.CD + L.H;
  for (int l = 0; l < c.n_layers; ++l) {
    LOAD_HIP(copy(L.norm[l], w->norm[l], d * eb));
    // in_proj rows zero-padded to a multiple of 128 output columns
    RepackSrc in{{w->in_proj[l], nullptr, nullptr}, {in_rows, 0, 0}};
    LOAD_HIP(launch_repack(c.dtype, in, L.NZ, d, kPermNone, 64, 64, m->at(L.w_in[l]), s));
    RepackSrc op{{w->out_proj[l], nullptr, nullptr}, {d, 0, 0}};
    LOAD_HIP(launch_repack(c.dtype, op, d, di, kPermNone, 64, 64, m->at(L.w_out[l]), s));
    LOAD_HIP(copy(L.conv_w[l], w->conv_w[l], (size_t)L.CD * c.d_conv * 4));
    LOAD_HIP(copy(L.conv_b[l], w->conv_b[l], (size_t)L.CD * 4));
    LOAD_HIP(copy(L.dt_b[l], w->dt_b[l], (size_t)L.H * 4));
    LOAD_HIP(copy(L.D[l], w->D[l], (size_t)L.H * 4));
    LOAD_HIP(copy(L.gnorm[l], w->gnorm[l], (size_t)di * eb));
    // A * log2(e) = -exp(A_log) * log2(e)
    LOAD_HIP(launch_transpose_f32(w->A_log[l], L.H, 1, 1, m->at<float>(L.A2[l]), 1,
                                  1.4426950408889634f, s));
  }
  LOAD_HIP(hipMemsetAsync(m->at(L.err), 0, 4, s));
#undef LOAD_HIP
  *out = m;
  return LL_OK;
}

ll_status ll_mamba2_prefill(ll_mamba2 *m, int32_t batch, const int32_t *seq_lens_host,
                            const int32_t *tokens_dev, int32_t *next_tokens_dev,
                            float *logits_dev) {
  g_err.clear();
  if (!m) return fail(LL_ERR_INVALID_ARGUMENT, "model is NULL");
  if (!seq_lens_host || !tokens_dev || !next_tokens_dev)
    return fail(LL_ERR_INVALID_ARGUMENT, "seq_lens_host, tokens_dev and next_tokens_dev must be set");
  const ll_mamba2_config &c = m->cfg;
  long total = 0;
  ll_status vst = m->check_prefill(batch, seq_lens_host, c.max_batch, c.max_prefill_tokens, &total);
  if (vst != LL_OK) return vst;
  const bool cont = m->batch != 0;
  MambaMeta mm;
  mm.batch = batch;
  for (int b = 0; b < batch; ++b) {
    mm.lens[b] = seq_lens_host[b];
  }
  const int T = (int)total;
  const int clen = use_ssd(c) ? kM2SsdChunk : mamba2_chunk_len(T, m->L.H, c.head_dim);
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
  const M2Layout &L = m->L;
  TimerScope scope(m->timer, 0);
  m->mark(LL_M2K_META);
  LL_HIP(launch_mamba_meta(mm, T, clen, m->at<int>(L.cu), m->at<int>(L.row_seq),
                           m->at<int>(L.last_row), m->at<int4>(L.chunks),
                           m->at<int>(L.seq_chunk0), s));
  m->mark(LL_M2K_EMBED);
  LL_HIP(launch_embed(c.dtype, tokens_dev, T, m->at(L.embed), c.vocab, c.d_model,
                      m->at<float>(L.x), m->at<int>(L.err), s));
  bool hf_ready = false;
  ll_status st = enqueue_layers(m, T, &pp, s, &hf_ready);
  if (st != LL_OK) return st;
  st = enqueue_head(m, batch, m->at<int>(L.last_row), next_tokens_dev, logits_dev, s, false);
  if (st != LL_OK) return st;
  m->commit_prefill(batch, seq_lens_host);
  return LL_OK;
}

ll_status ll_mamba2_decode_step(ll_mamba2 *m, const int32_t *in_tokens_dev,
                                int32_t *next_tokens_dev, float *logits_dev) {
  g_err.clear();
  if (!m) return fail(LL_ERR_INVALID_ARGUMENT, "model is NULL");
  if (!in_tokens_dev || !next_tokens_dev)
    return fail(LL_ERR_INVALID_ARGUMENT, "in_tokens_dev and next_tokens_dev must be set");
  return m->decode(in_tokens_dev, next_tokens_dev, logits_dev, [&](hipStream_t s) {
    return enqueue_decode(m, in_tokens_dev, next_tokens_dev, logits_dev, s);
  });
}

ll_status ll_mamba2_reset(ll_mamba2 *m) {
  g_err.clear();
  if (!m) return fail(LL_ERR_INVALID_ARGUMENT, "model is NULL");
  return m->reset();
}

ll_status ll_mamba2_seq_lengths(const ll_mamba2 *m, int32_t *out, int32_t cap, int32_t *n) {
  g_err.clear();
  if (!m) return fail(LL_ERR_INVALID_ARGUMENT, "model is NULL");
  return m->seq_lengths(out, cap, n);
}

ll_status ll_mamba2_set_option(ll_mamba2 *m, int32_t option, int32_t value) {
  g_err.clear();
  if (!m) return fail(LL_ERR_INVALID_ARGUMENT, "model is NULL");
  return m->set_option(option, value);
}

ll_status ll_mamba2_get_option(const ll_mamba2 *m, int32_t option, int32_t *value) {
  g_err.clear();
  if (!m) return fail(LL_ERR_INVALID_ARGUMENT, "model is NULL");
  return m->get_option(option, value);
}

ll_status ll_mamba2_device_flags(ll_mamba2 *m, int32_t *flags) {
  g_err.clear();
  if (!m) return fail(LL_ERR_INVALID_ARGUMENT, "model is NULL");
  return m->device_flags(m->L.err, flags);
}

ll_status ll_mamba2_set_kernel_timing(ll_mamba2 *m, int32_t enable) {
  g_err.clear();
  if (!m) return fail(LL_ERR_INVALID_ARGUMENT, "model is NULL");
  return m->set_kernel_timing(enable);
}

ll_status ll_mamba2_kernel_timing_read(ll_mamba2 *m, int32_t *counts, double *ms) {
  g_err.clear();
  if (!m) return fail(LL_ERR_INVALID_ARGUMENT, "model is NULL");
  return m->kernel_timing_read(LL_M2K_COUNT, counts, ms);
}

const char *ll_mamba2_kernel_class_name(int32_t cls) {
  return (cls >= 0 && cls < LL_M2K_COUNT) ? kM2ClassNames[cls] : "";
}

void ll_mamba2_free(ll_mamba2 *m) { delete m; }

}  // extern "C"
