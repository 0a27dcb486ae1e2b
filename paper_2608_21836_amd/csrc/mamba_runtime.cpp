// C-ABI runtime of the selective state-space (Mamba) model: config validation, workspace
// layout, weight repacking, the prefill / decode phase dispatch with explicit conv and SSM
// state, and decode-step HIP graphs.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <vector>

#include "kernels.h"
#include "ll.h"
#include "ll_mamba.h"
#include "runtime_common.h"

using namespace ll;

namespace {

const char *const kMambaClassNames[LL_MK_COUNT] = {
    "prefill_meta", "embed",      "rmsnorm", "in_proj",  "conv_silu",      "x_proj",
    "scan_chunk",   "scan_carry", "scan",    "out_proj_resid", "lm_head_argmax", "argmax_reduce"};

constexpr int kDState = 16;
constexpr int kFusedNormMaxRows = 16;

struct MLayout {
  size_t embed = 0, lm_head = 0, final_norm = 0;
  std::vector<size_t> norm, w_in, w_x, w_out, conv_w, conv_b, dtwT, dt_b, A2, D;
  size_t conv_state = 0, ssm_state = 0;  // [L][max_batch][K-1][di], [L][max_batch][di][N]
  size_t x = 0, h = 0, xz = 0, u = 0, xdbl = 0, y = 0, hf = 0;
  size_t hloc = 0, dtsum = 0, chunks = 0, seq_chunk0 = 0;
  size_t splitk = 0, splitk_bytes = 0;
  size_t pval = 0, pidx = 0, cu = 0, row_seq = 0, last_row = 0, err = 0;
  size_t total = 0;
  int NX = 0, max_rows = 0, max_chunks = 0, n_parts = 0;
};

ll_status validate(const ll_mamba_config *c) {
  if (!c) return fail(LL_ERR_INVALID_ARGUMENT, "cfg is NULL");
  if (c->n_layers < 1 || c->d_model < 1 || c->d_inner < 1 || c->d_state < 1 || c->d_conv < 1 ||
      c->dt_rank < 1 || c->vocab < 1)
    return fail(LL_ERR_INVALID_ARGUMENT, "model dimensions must be positive");
  if (c->max_batch < 1 || c->max_prefill_tokens < 1)
    return fail(LL_ERR_INVALID_ARGUMENT, "capacities must be positive");
  if (!(c->rms_eps >= 0.f) || !std::isfinite(c->rms_eps))
    return fail(LL_ERR_INVALID_ARGUMENT, "rms_eps must be finite and >= 0");
  if (c->dtype != LL_F32 && c->dtype != LL_BF16)
    return fail(LL_ERR_UNSUPPORTED, "dtype %d unknown", c->dtype);
  if (c->d_state != kDState) return fail(LL_ERR_UNSUPPORTED, "d_state %d != 16", c->d_state);
  if (c->d_conv > 4) return fail(LL_ERR_UNSUPPORTED, "d_conv %d > 4", c->d_conv);
  if (c->dt_rank > 160) return fail(LL_ERR_UNSUPPORTED, "dt_rank %d > 160", c->dt_rank);
  if (c->d_model % 128) return fail(LL_ERR_UNSUPPORTED, "d_model %d not a multiple of 128", c->d_model);
  if (c->d_inner % 64) return fail(LL_ERR_UNSUPPORTED, "d_inner %d not a multiple of 64", c->d_inner);
  if (c->vocab % 32) return fail(LL_ERR_UNSUPPORTED, "vocab %d not a multiple of 32", c->vocab);
  if (c->max_batch > LL_MAX_BATCH)
    return fail(LL_ERR_UNSUPPORTED, "max_batch %d > %d", c->max_batch, LL_MAX_BATCH);
  return LL_OK;
}

MLayout make_layout(const ll_mamba_config &c) {
  MLayout L;
  const size_t eb = elem_bytes(c.dtype);
  const size_t d = c.d_model, di = c.d_inner, N = c.d_state, K1 = c.d_conv - 1;
  L.NX = (c.dt_rank + 2 * c.d_state + 127) / 128 * 128;
  L.max_rows = std::max(c.max_prefill_tokens, c.max_batch);
  L.max_chunks = mamba_max_chunks(c.max_prefill_tokens, c.max_batch, c.d_inner);
  L.n_parts = c.vocab / 32;
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
    L.w_in.push_back(take(2 * di * d * eb));
    L.w_x.push_back(take((size_t)L.NX * di * eb));
    L.w_out.push_back(take(d * di * eb));
    L.conv_w.push_back(take(di * c.d_conv * 4));
    L.conv_b.push_back(take(di * 4));
    L.dtwT.push_back(take((size_t)((c.dt_rank + 15) / 16 * 16) * di * 4));  // rows padded to 16
    L.dt_b.push_back(take(di * 4));
    L.A2.push_back(take(N * di * 4));
    L.D.push_back(take(di * 4));
  }
  L.conv_state = take((size_t)c.n_layers * c.max_batch * std::max<size_t>(K1, 1) * di * 4);
  L.ssm_state = take((size_t)c.n_layers * c.max_batch * N * di * 4);
  const size_t R = L.max_rows;
  L.x = take(R * d * 4);
  L.h = take(R * d * eb);
  L.xz = take(R * 2 * di * 4);
  L.u = take(R * di * eb);
  L.xdbl = take(R * L.NX * 4);
  L.y = take(R * di * eb);
  L.hf = take((size_t)c.max_batch * d * eb);
  L.hloc = take((size_t)L.max_chunks * N * di * 4);
  L.dtsum = take((size_t)L.max_chunks * di * 4);
  L.chunks = take((size_t)L.max_chunks * 16);
  L.seq_chunk0 = take((c.max_batch + 1) * 4);
  {
    const int shapes[3][2] = {{2 * (int)di, (int)d}, {L.NX, (int)di}, {(int)d, (int)di}};
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

struct ll_mamba : ll::StateModel {
  ll_mamba_config cfg;
  MLayout L;
  ll_mamba() : StateModel("ll_mamba_reset", true) {}
  size_t K1() const { return (size_t)std::max(cfg.d_conv - 1, 1); }
  float *conv_state(int l) const {
    return at<float>(L.conv_state) + (size_t)l * cfg.max_batch * K1() * cfg.d_inner;
  }
  float *ssm_state(int l) const {
    return at<float>(L.ssm_state) + (size_t)l * cfg.max_batch * cfg.d_state * cfg.d_inner;
  }
};

namespace {

EpiParams store_epi(float *out, int ld) {
  EpiParams ep;
  ep.kind = kEpiStore;
  ep.out_f32 = out;
  ep.ld_out = ld;
  return ep;
}

EpiParams resid_epi(float *out, int ld) {
  EpiParams ep;
  ep.kind = kEpiResid;
  ep.out_f32 = out;
  ep.ld_out = ld;
  return ep;
}

ScanArgs scan_args(const ll_mamba *m, int l) {
  const ll_mamba_config &c = m->cfg;
  const MLayout &L = m->L;
  ScanArgs a;
  a.xdbl = m->at<float>(L.xdbl);
  a.ldx = L.NX;
  a.u = m->at(L.u);
  a.xz = m->at<float>(L.xz);
  a.ldxz = 2 * c.d_inner;
  a.dtwT = m->at<float>(L.dtwT[l]);
  a.dt_b = m->at<float>(L.dt_b[l]);
  a.A2 = m->at<float>(L.A2[l]);
  a.D = m->at<float>(L.D[l]);
  a.ssm = m->ssm_state(l);
  a.conv = m->conv_state(l);
  a.y = m->at(L.y);
  a.hloc = m->at<float>(L.hloc);
  a.dtsum = m->at<float>(L.dtsum);
  a.di = c.d_inner;
  a.R = c.dt_rank;
  a.N = c.d_state;
  a.K = c.d_conv;
  return a;
}

// The fused decode step takes up to kSsmDecodeMaxRows sequences and x_proj widths up to
// kSsmDecodeMaxX.
bool ssm_decode_fits(const ll_mamba_config &c, int rows) {
  return rows <= kSsmDecodeMaxRows && c.dt_rank + 2 * c.d_state <= kSsmDecodeMaxX;
}

// Per-call prefill description (null for decode).
struct PrefillPlan {
  int n_chunks = 0;
  bool multi = false;  // some sequence spans more than one chunk
  bool fresh = false;  // sequences start from zero state
  int batch = 0;
};

// The mixer layers for `rows` rows: decode (one row per sequence) or a prefill.
ll_status enqueue_layers(ll_mamba *m, int rows, const PrefillPlan *pp, hipStream_t s,
                         bool *hf_ready) {
  *hf_ready = false;
  const ll_mamba_config &c = m->cfg;
  const MLayout &L = m->L;
  const bool decode = pp == nullptr;
  const int d = c.d_model, di = c.d_inner, dt = c.dtype;
  const bool fuse_norm = decode && rows <= kFusedNormMaxRows &&
                         skinny_norm_lds(elem_bytes(dt), rows, d) <= kSkinnyMaxNormLds;
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
  const bool fused = decode && m->opt[LL_OPT_DECODE_FUSED] && ssm_decode_fits(c, rows);
  const bool fused_out = fused && m->opt[LL_OPT_DECODE_FUSED] == 2;
  bool h_ready = false;
  for (int l = 0; l < c.n_layers; ++l) {
    NormIn nrm;
    if (fuse_norm) {
      nrm = NormIn{x, d, nullptr, m->at(L.norm[l]), c.rms_eps};
    } else if (!h_ready) {
      m->mark(LL_MK_RMSNORM);
      LL_HIP(launch_rmsnorm(dt, x, d, nullptr, rows, d, m->at(L.norm[l]), c.rms_eps, m->at(L.h),
                            d, s));
    }
    h_ready = false;
    m->mark(LL_MK_IN_PROJ);
    if (fused) {
      // conv step in the in_proj epilogue, then x_proj + dt + scan step + gate in one kernel
      EpiParams ep;
      ep.kind = kEpiConv;
      ep.act = m->at(L.u);
      ep.out_f32 = m->at<float>(L.xz);  // z at columns [di, 2 di)
      ep.ld_out = 2 * di;
      ep.conv_state = m->conv_state(l);
      ep.conv_w = m->at<float>(L.conv_w[l]);
      ep.conv_b = m->at<float>(L.conv_b[l]);
      ep.conv_k = c.d_conv;
      ep.conv_col0 = 0;
      ep.conv_n = di;
      LL_HIP(gemm(m->at(L.h), d, fuse_norm ? &nrm : nullptr, m->at(L.w_in[l]), 2 * di, d, ep));
      SsmDecodeArgs sa;
      sa.u = m->at(L.u);
      sa.z = m->at<float>(L.xz) + di;
      sa.ldz = 2 * di;
      sa.wx = m->at(L.w_x[l]);
      sa.dtwT = m->at<float>(L.dtwT[l]);
      sa.dt_b = m->at<float>(L.dt_b[l]);
      sa.A2 = m->at<float>(L.A2[l]);
      sa.D = m->at<float>(L.D[l]);
      sa.ssm = m->ssm_state(l);
      sa.rows = rows;
      sa.di = di;
      sa.R = c.dt_rank;
      sa.N = c.d_state;
      if (fused_out) {  // out_proj and the residual add inside the step
        sa.wout = m->at(L.w_out[l]);
        sa.x = x;
        sa.ldx = d;
        sa.d = d;
      } else {
        sa.y = m->at(L.y);
      }
      m->mark(LL_MK_SCAN);
      LL_HIP(launch_ssm_decode(dt, sa, s));
    } else {
      LL_HIP(gemm(m->at(L.h), d, fuse_norm ? &nrm : nullptr, m->at(L.w_in[l]), 2 * di, d,
                  store_epi(m->at<float>(L.xz), 2 * di)));
      m->mark(LL_MK_CONV);
      LL_HIP(launch_mamba_conv(dt, m->at<float>(L.xz), 2 * di,
                               decode ? nullptr : m->at<int>(L.row_seq),
                               decode ? nullptr : m->at<int>(L.cu), m->conv_state(l),
                               decode ? 0 : pp->fresh, m->at<float>(L.conv_w[l]),
                               m->at<float>(L.conv_b[l]), rows, di, c.d_conv, m->at(L.u), s));
      m->mark(LL_MK_X_PROJ);
      LL_HIP(gemm(m->at(L.u), di, nullptr, m->at(L.w_x[l]), L.NX, di,
                  store_epi(m->at<float>(L.xdbl), L.NX)));
      ScanArgs a = scan_args(m, l);
      if (decode) {
        a.carry = 1;
        m->mark(LL_MK_SCAN);
        LL_HIP(launch_scan_out(dt, a, rows, s));
      } else {
        a.chunks = m->at<int4>(L.chunks);
        a.seq_chunk0 = m->at<int>(L.seq_chunk0);
        a.cu = m->at<int>(L.cu);
        a.fresh = pp->fresh;
        if (pp->multi) {
          m->mark(LL_MK_SCAN_CHUNK);
          LL_HIP(launch_scan_chunks(dt, a, pp->n_chunks, s));
          m->mark(LL_MK_SCAN_CARRY);
          LL_HIP(launch_scan_carry(a, pp->batch, s));
          a.carry = 2;
        } else {
          a.carry = pp->fresh ? 0 : 1;
        }
        m->mark(LL_MK_SCAN);
        LL_HIP(launch_scan_out(dt, a, pp->n_chunks, s));
      }
    }
    if (fused_out) continue;  // out_proj ran inside the fused step
    m->mark(LL_MK_OUT_PROJ);
    const bool last = l + 1 == c.n_layers;
    PostNorm pn;
    pn.gain = m->at(last ? L.final_norm : L.norm[l + 1]);
    pn.eps = c.rms_eps;
    pn.out = m->at(last ? L.hf : L.h);
    pn.ld_out = d;
    bool done = false;
    LL_HIP(gemm(m->at(L.y), di, nullptr, m->at(L.w_out[l]), d, di, resid_epi(x, d),
                (decode && !fuse_norm) ? &pn : nullptr, &done));
    if (last) *hf_ready = done;
    else h_ready = done;
  }
  return LL_OK;
}

// Final RMSNorm of one row per sequence, the tied LM head with argmax partials, the reduction.
ll_status enqueue_head(ll_mamba *m, int batch, const int *rowmap, int *next, float *logits,
                       hipStream_t s, bool hf_ready) {
  const ll_mamba_config &c = m->cfg;
  const MLayout &L = m->L;
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
    m->mark(LL_MK_RMSNORM);
    LL_HIP(launch_rmsnorm(c.dtype, m->at<float>(L.x), c.d_model, rowmap, batch, c.d_model,
                          m->at(L.final_norm), c.rms_eps, m->at(L.hf), c.d_model, s));
  }
  m->mark(LL_MK_LM_HEAD);
  LL_HIP(launch_gemm_skinny(c.dtype, m->at(L.hf), c.d_model, fuse_norm ? &nrm : nullptr,
                            m->at(L.lm_head), batch, c.vocab, c.d_model, ep, s));
  m->mark(LL_MK_ARGMAX);
  LL_HIP(launch_argmax_reduce(ep.part_val, ep.part_idx, batch, ep.n_parts, next, nullptr, s));
  return LL_OK;
}

ll_status enqueue_decode(ll_mamba *m, const int32_t *in, int32_t *out, float *logits,
                         hipStream_t s) {
  const ll_mamba_config &c = m->cfg;
  m->mark(LL_MK_EMBED);
  LL_HIP(launch_embed(c.dtype, in, m->batch, m->at(m->L.embed), c.vocab, c.d_model,
                      m->at<float>(m->L.x), m->at<int>(m->L.err), s));
  bool hf_ready = false;
  ll_status st = enqueue_layers(m, m->batch, nullptr, s, &hf_ready);
  if (st != LL_OK) return st;
  return enqueue_head(m, m->batch, nullptr, out, logits, s, hf_ready);
}

}  // namespace

extern "C" {

ll_status ll_mamba_workspace_size(const ll_mamba_config *cfg, size_t *bytes) {
  g_err.clear();
  if (!bytes) return fail(LL_ERR_INVALID_ARGUMENT, "bytes is NULL");
  ll_status st = validate(cfg);
  if (st != LL_OK) return st;
  *bytes = make_layout(*cfg).total;
  return LL_OK;
}

ll_status ll_mamba_load(const ll_mamba_config *cfg, const ll_mamba_weights *w, void *workspace,
                        size_t workspace_bytes, void *hip_stream, ll_mamba **out) {
  g_err.clear();
  if (!out) return fail(LL_ERR_INVALID_ARGUMENT, "out is NULL");
  *out = nullptr;
  ll_status st = validate(cfg);
  if (st != LL_OK) return st;
  if (!w) return fail(LL_ERR_INVALID_ARGUMENT, "weights is NULL");
  if (!w->embed || !w->final_norm) return fail(LL_ERR_INVALID_ARGUMENT, "embed and final_norm must be set");
  const void *const *arrays[] = {w->norm, w->in_proj, (const void *const *)w->conv_w,
                                 (const void *const *)w->conv_b, w->x_proj,
                                 (const void *const *)w->dt_w, (const void *const *)w->dt_b,
                                 (const void *const *)w->A_log, (const void *const *)w->D,
                                 w->out_proj};
  for (auto a : arrays) {
    if (!a) return fail(LL_ERR_INVALID_ARGUMENT, "a per-layer weight array is NULL");
    for (int l = 0; l < cfg->n_layers; ++l)
      if (!a[l]) return fail(LL_ERR_INVALID_ARGUMENT, "layer %d weight pointer is NULL", l);
  }
  if ((st = check_ws(workspace)) != LL_OK) return st;
  const MLayout L = make_layout(*cfg);
  if (workspace_bytes < L.total)
    return fail(LL_ERR_WORKSPACE, "workspace has %zu bytes, needs %zu", workspace_bytes, L.total);

  ll_mamba *m = new ll_mamba();
  m->cfg = *cfg;
  m->L = L;
  m->ws = reinterpret_cast<char *>(workspace);
  m->stream = reinterpret_cast<hipStream_t>(hip_stream);
  const ll_mamba_config &c = *cfg;
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
  for (int l = 0; l < c.n_layers; ++l) {
    LOAD_HIP(copy(L.norm[l], w->norm[l], d * eb));
    RepackSrc in{{w->in_proj[l], nullptr, nullptr}, {2 * di, 0, 0}};
    LOAD_HIP(launch_repack(c.dtype, in, 2 * di, d, kPermNone, 64, 64, m->at(L.w_in[l]), s));
    // x_proj rows padded with zeros to a multiple of 128 output columns
    RepackSrc xp{{w->x_proj[l], nullptr, nullptr}, {c.dt_rank + 2 * c.d_state, 0, 0}};
    LOAD_HIP(launch_repack(c.dtype, xp, L.NX, di, kPermNone, 64, 64, m->at(L.w_x[l]), s));
    RepackSrc op{{w->out_proj[l], nullptr, nullptr}, {d, 0, 0}};
    LOAD_HIP(launch_repack(c.dtype, op, d, di, kPermNone, 64, 64, m->at(L.w_out[l]), s));
    LOAD_HIP(copy(L.conv_w[l], w->conv_w[l], (size_t)di * c.d_conv * 4));
    LOAD_HIP(copy(L.conv_b[l], w->conv_b[l], (size_t)di * 4));
    LOAD_HIP(copy(L.dt_b[l], w->dt_b[l], (size_t)di * 4));
    LOAD_HIP(copy(L.D[l], w->D[l], (size_t)di * 4));
    LOAD_HIP(launch_transpose_f32(w->dt_w[l], di, c.dt_rank, (c.dt_rank + 15) / 16 * 16,
                                  m->at<float>(L.dtwT[l]), 0, 1.f, s));
    // A * log2(e) = -exp(A_log) * log2(e), state-major
    LOAD_HIP(launch_transpose_f32(w->A_log[l], di, c.d_state, c.d_state, m->at<float>(L.A2[l]),
                                  1, 1.4426950408889634f, s));
  }
  LOAD_HIP(hipMemsetAsync(m->at(L.err), 0, 4, s));
#undef LOAD_HIP
  *out = m;
  return LL_OK;
}

ll_status ll_mamba_prefill(ll_mamba *m, int32_t batch, const int32_t *seq_lens_host,
                           const int32_t *tokens_dev, int32_t *next_tokens_dev,
                           float *logits_dev) {
  g_err.clear();
  if (!m) return fail(LL_ERR_INVALID_ARGUMENT, "model is NULL");
  if (!seq_lens_host || !tokens_dev || !next_tokens_dev)
    return fail(LL_ERR_INVALID_ARGUMENT, "seq_lens_host, tokens_dev and next_tokens_dev must be set");
  const ll_mamba_config &c = m->cfg;
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
  const int clen = mamba_chunk_len(T, c.d_inner);
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
  const MLayout &L = m->L;
  TimerScope scope(m->timer, 0);
  m->mark(LL_MK_META);
  LL_HIP(launch_mamba_meta(mm, T, clen, m->at<int>(L.cu), m->at<int>(L.row_seq),
                           m->at<int>(L.last_row), m->at<int4>(L.chunks),
                           m->at<int>(L.seq_chunk0), s));
  m->mark(LL_MK_EMBED);
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

ll_status ll_mamba_decode_step(ll_mamba *m, const int32_t *in_tokens_dev, int32_t *next_tokens_dev,
                               float *logits_dev) {
  g_err.clear();
  if (!m) return fail(LL_ERR_INVALID_ARGUMENT, "model is NULL");
  if (!in_tokens_dev || !next_tokens_dev)
    return fail(LL_ERR_INVALID_ARGUMENT, "in_tokens_dev and next_tokens_dev must be set");
  return m->decode(in_tokens_dev, next_tokens_dev, logits_dev, [&](hipStream_t s) {
    return enqueue_decode(m, in_tokens_dev, next_tokens_dev, logits_dev, s);
  });
}

ll_status ll_mamba_reset(ll_mamba *m) {
  g_err.clear();
  if (!m) return fail(LL_ERR_INVALID_ARGUMENT, "model is NULL");
  return m->reset();
}

ll_status ll_mamba_seq_lengths(const ll_mamba *m, int32_t *out, int32_t cap, int32_t *n) {
  g_err.clear();
  if (!m) return fail(LL_ERR_INVALID_ARGUMENT, "model is NULL");
  return m->seq_lengths(out, cap, n);
}

ll_status ll_mamba_set_option(ll_mamba *m, int32_t option, int32_t value) {
  g_err.clear();
  if (!m) return fail(LL_ERR_INVALID_ARGUMENT, "model is NULL");
  return m->set_option(option, value);
}

ll_status ll_mamba_get_option(const ll_mamba *m, int32_t option, int32_t *value) {
  g_err.clear();
  if (!m) return fail(LL_ERR_INVALID_ARGUMENT, "model is NULL");
  return m->get_option(option, value);
}

ll_status ll_mamba_device_flags(ll_mamba *m, int32_t *flags) {
  g_err.clear();
  if (!m) return fail(LL_ERR_INVALID_ARGUMENT, "model is NULL");
  return m->device_flags(m->L.err, flags);
}

ll_status ll_mamba_set_kernel_timing(ll_mamba *m, int32_t enable) {
  g_err.clear();
  if (!m) return fail(LL_ERR_INVALID_ARGUMENT, "model is NULL");
  return m->set_kernel_timing(enable);
}

ll_status ll_mamba_kernel_timing_read(ll_mamba *m, int32_t *counts, double *ms) {
  g_err.clear();
  if (!m) return fail(LL_ERR_INVALID_ARGUMENT, "model is NULL");
  return m->kernel_timing_read(LL_MK_COUNT, counts, ms);
}

const char *ll_mamba_kernel_class_name(int32_t cls) {
  return (cls >= 0 && cls < LL_MK_COUNT) ? kMambaClassNames[cls] : "";
}

void ll_mamba_free(ll_mamba *m) { delete m; }

}  // extern "C"
