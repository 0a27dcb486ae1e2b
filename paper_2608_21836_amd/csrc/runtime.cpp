// C-ABI runtime: config validation, workspace layout, weight repacking, phase dispatch
// (prefill vs decode, Sec. 2.1 and Sec. 3.1 of the paper), decode-step HIP graphs and the
// per-kernel entry points of ll_ops.h.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "kernels.h"
#include "ll.h"
#include "ll_ops.h"
#include "runtime_common.h"

namespace ll {
thread_local LaunchTimer *g_launch_timer = nullptr;
thread_local std::string g_err;
}

using namespace ll;

namespace {

const char *const kClassNames[LL_K_COUNT] = {
    "prefill_meta", "embed",          "rmsnorm",       "qkv_rope_append",
    "attention",    "attn_combine",   "o_proj_resid",  "gate_up_swiglu",
    "down_resid",   "lm_head_argmax", "argmax_reduce"};

struct Layout {
  size_t embed = 0, final_norm = 0, lm_head = 0;
  std::vector<size_t> wqkv, wo, wgu, wd, attn_norm, mlp_norm;
  size_t kcache = 0, vcache = 0, rcos = 0, rsin = 0;
  size_t x = 0, h = 0, q = 0, o = 0, act = 0, hf = 0;
  size_t part_o = 0, part_ml = 0, pval = 0, pidx = 0;
  size_t splitk = 0, splitk_bytes = 0;  // fp32 split-K partials of the decode GEMMs
  size_t kstart = 0;                     // cached keys before each sequence's prefill chunk
  size_t cu = 0, row_seq = 0, row_pos = 0, last_row = 0, lens = 0, qtiles = 0, sched = 0, err = 0;
  size_t total = 0;
  size_t kv_layer_elems = 0;
  size_t kv_table = 0;                   // paged cache: int32 [max_batch][kv_max_pages]
  int kv_max_pages = 0, kv_pages = 0;
  AttnDecodePlan attn;
  int n_parts = 0, max_rows = 0, n_qkv = 0;
  struct Region {
    std::string name;
    size_t off, bytes;
  };
  std::vector<Region> regions;  // every region of the workspace, in address order
};

ll_status validate_config(const ll_config *c) {
  if (!c) return fail(LL_ERR_INVALID_ARGUMENT, "cfg is NULL");
  if (c->n_layers < 1 || c->d_model < 1 || c->n_heads < 1 || c->n_kv_heads < 1 ||
      c->head_dim < 1 || c->ffn_dim < 1 || c->vocab < 1)
    return fail(LL_ERR_INVALID_ARGUMENT, "model dimensions must be positive");
  if (c->max_batch < 1 || c->max_prefill_tokens < 1 || c->max_ctx < 1)
    return fail(LL_ERR_INVALID_ARGUMENT, "capacities must be positive");
  if (!(c->rms_eps >= 0.f) || !std::isfinite(c->rms_eps))
    return fail(LL_ERR_INVALID_ARGUMENT, "rms_eps must be finite and >= 0");
  if (!(c->rope_theta > 0.0) || !std::isfinite(c->rope_theta))
    return fail(LL_ERR_INVALID_ARGUMENT, "rope_theta must be finite and > 0");
  if (c->dtype != LL_F32 && c->dtype != LL_BF16)
    return fail(LL_ERR_UNSUPPORTED, "dtype %d unknown", c->dtype);
  if (c->head_dim != 64 && c->head_dim != 128)
    return fail(LL_ERR_UNSUPPORTED, "head_dim %d not in {64, 128}", c->head_dim);
  if (c->n_heads % c->n_kv_heads)
    return fail(LL_ERR_UNSUPPORTED, "n_heads %d not a multiple of n_kv_heads %d", c->n_heads,
                c->n_kv_heads);
  const int g = c->n_heads / c->n_kv_heads;
  if (g != 1 && g != 2 && g != 4 && g != 8)
    return fail(LL_ERR_UNSUPPORTED, "head group %d not in {1, 2, 4, 8}", g);
  if (c->d_model % 128)
    return fail(LL_ERR_UNSUPPORTED, "d_model %d not a multiple of 128", c->d_model);
  if (((c->n_heads + 2 * c->n_kv_heads) * c->head_dim) % 128)
    return fail(LL_ERR_UNSUPPORTED, "(n_heads + 2 n_kv_heads) * head_dim not a multiple of 128");
  if (c->ffn_dim % 64)
    return fail(LL_ERR_UNSUPPORTED, "ffn_dim %d not a multiple of 64", c->ffn_dim);
  if (c->vocab % 32) return fail(LL_ERR_UNSUPPORTED, "vocab %d not a multiple of 32", c->vocab);
  if (c->max_batch > LL_MAX_BATCH)
    return fail(LL_ERR_UNSUPPORTED, "max_batch %d > %d", c->max_batch, LL_MAX_BATCH);
  if (c->max_ctx > attn_decode_max_ctx())
    return fail(LL_ERR_UNSUPPORTED, "max_ctx %d > %d", c->max_ctx, attn_decode_max_ctx());
  if (c->kv_page < 0 || c->kv_pages < 0)
    return fail(LL_ERR_INVALID_ARGUMENT, "kv_page and kv_pages must be >= 0");
  if (c->kv_page == 0 && c->kv_pages != 0)
    return fail(LL_ERR_INVALID_ARGUMENT, "kv_pages %d without kv_page", c->kv_pages);
  if (c->kv_page % 256)
    return fail(LL_ERR_UNSUPPORTED, "kv_page %d not a multiple of 256", c->kv_page);
  if (c->f16_compute != 0 && c->f16_compute != 1)
    return fail(LL_ERR_INVALID_ARGUMENT, "f16_compute %d not 0 or 1", c->f16_compute);
  if (c->f16_compute && c->dtype != LL_BF16)
    return fail(LL_ERR_INVALID_ARGUMENT, "f16_compute needs bf16 weights");
  return LL_OK;
}

Layout make_layout(const ll_config &c) {
  Layout L;
  const size_t eb = elem_bytes(c.dtype);
  const size_t d = c.d_model, qd = (size_t)c.n_heads * c.head_dim;
  L.n_qkv = (c.n_heads + 2 * c.n_kv_heads) * c.head_dim;
  L.max_rows = std::max(c.max_prefill_tokens, c.max_batch);
  L.attn = attn_decode_plan(c.head_dim, (int)eb, c.max_batch, c.n_kv_heads, c.max_ctx);
  L.n_parts = c.vocab / 32;
  size_t off = 0;
  // Every region is followed by a guard gap of kGuardBytes that no kernel writes, so that a
  // write past the end of a region is detectable (ll_workspace_regions lists the regions).
  auto take = [&](std::string name, size_t bytes) {
    const size_t o = off;
    L.regions.push_back({std::move(name), o, bytes});
    off = align_up(off + bytes) + kGuardBytes;
    return o;
  };
  L.embed = take("embed", (size_t)c.vocab * d * eb);
  for (int l = 0; l < c.n_layers; ++l) {
    L.wqkv.push_back(take("layers." + std::to_string(l) + ".wqkv", (size_t)L.n_qkv * d * eb));
    L.wo.push_back(take("layers." + std::to_string(l) + ".wo", d * qd * eb));
    L.wgu.push_back(take("layers." + std::to_string(l) + ".wgu", 2 * (size_t)c.ffn_dim * d * eb));
    L.wd.push_back(take("layers." + std::to_string(l) + ".wd", d * c.ffn_dim * eb));
    L.attn_norm.push_back(take("layers." + std::to_string(l) + ".attn_norm", d * eb));
    L.mlp_norm.push_back(take("layers." + std::to_string(l) + ".mlp_norm", d * eb));
  }
  L.final_norm = take("final_norm", d * eb);
  L.lm_head = take("lm_head", (size_t)c.vocab * d * eb);
  if (c.kv_page > 0) {
    L.kv_max_pages = (c.max_ctx + c.kv_page - 1) / c.kv_page;
    L.kv_pages = c.kv_pages > 0 ? c.kv_pages : c.max_batch * L.kv_max_pages;
    L.kv_layer_elems = (size_t)L.kv_pages * c.n_kv_heads * c.kv_page * c.head_dim;
    L.kv_table = take("kv_table", (size_t)c.max_batch * L.kv_max_pages * 4);
  } else {
    L.kv_layer_elems = (size_t)c.max_batch * c.n_kv_heads * c.max_ctx * c.head_dim;
  }
  L.kcache = take("kcache", L.kv_layer_elems * c.n_layers * eb);
  L.vcache = take("vcache", L.kv_layer_elems * c.n_layers * eb);
  L.rcos = take("rcos", (size_t)c.max_ctx * (c.head_dim / 2) * 4);
  L.rsin = take("rsin", (size_t)c.max_ctx * (c.head_dim / 2) * 4);
  const size_t R = L.max_rows;
  L.x = take("x", R * d * 4);
  L.h = take("h", R * d * eb);
  L.q = take("q", R * qd * eb);
  L.o = take("o", R * qd * eb);
  L.act = take("act", R * c.ffn_dim * eb);
  L.hf = take("hf", (size_t)c.max_batch * d * eb);
  L.part_o = take("part_o", (size_t)c.max_batch * c.n_heads * L.attn.nsplit * c.head_dim * 4);
  L.part_ml = take("part_ml", (size_t)c.max_batch * c.n_heads * L.attn.nsplit * 2 * 4);
  {
    const int F = c.ffn_dim;
    const int shapes[4][2] = {{L.n_qkv, (int)d}, {(int)d, (int)qd}, {2 * F, (int)d}, {(int)d, F}};
    // One region serves the decode split-K GEMMs (max_batch rows) and the split prefill GEMMs
    // of short prompts (any row count up to max_prefill_tokens that the split plan takes).
    for (const auto &nk : shapes) {
      L.splitk_bytes = std::max(L.splitk_bytes, splitk_plan(eb, c.max_batch, nk[0], nk[1]).ws_bytes);
      const int mmax = std::min(c.max_prefill_tokens, 64 * kPrefillSplitMinTiles);
      for (int mr = 64; mr < mmax + 64; mr += 64) {
        const int mm = std::min(mr, mmax);
        L.splitk_bytes =
            std::max(L.splitk_bytes, prefill_splitk_plan(eb, mm, nk[0], nk[1]).ws_bytes);
      }
      L.splitk_bytes =
          std::max(L.splitk_bytes, prefill_splitk_plan(eb, mmax, nk[0], nk[1]).ws_bytes);
    }
    L.splitk = take("splitk", L.splitk_bytes);
  }
  L.pval = take("pval", (size_t)c.max_batch * L.n_parts * 4);
  L.pidx = take("pidx", (size_t)c.max_batch * L.n_parts * 4);
  L.cu = take("cu", (c.max_batch + 1) * 4);
  L.row_seq = take("row_seq", R * 4);
  L.row_pos = take("row_pos", R * 4);
  L.last_row = take("last_row", c.max_batch * 4);
  L.lens = take("lens", c.max_batch * 4);
  L.kstart = take("kstart", c.max_batch * 4);
  L.qtiles = take("qtiles", (R / kAttnQTile + c.max_batch + 1) * 8);
  // work list of the grouped-query prefill attention: ceil(L_b / qtile) tiles per sequence and
  // KV head, each sequence at least one token
  if (attn_prefill_gqa(compute_dtype(c), c.n_heads / c.n_kv_heads))
    L.sched = take("sched", (R / attn_gqa_qtile(c.n_heads / c.n_kv_heads) + c.max_batch + 1) *
                   (size_t)c.n_kv_heads * 16);
  L.err = take("err", 4);
  L.total = off;
  return L;
}

}  // namespace

struct ll_model {
  ll_config cfg;
  Layout L;
  char *ws = nullptr;
  hipStream_t stream = nullptr;
  hipStream_t cap_stream = nullptr;  // records decode graphs (graphs then run on `stream`)
  int batch = 0;
  std::vector<int> lens;
  bool use_graph = true;
  int opt[LL_OPT_COUNT] = {1, 1, 1, 0, 0, 0};  // ll_option values (LL_OPT_DECODE_GRAPH mirrors use_graph)
  struct Graph {
    const void *in;
    void *out;
    void *logits;
    int batch;
    hipGraphExec_t exec;
  };
  std::vector<Graph> graphs;
  std::vector<float> rope_host;
  Timer *timer = nullptr;  // per-launch timing (decode then runs without the graph)
  void mark(int cls) const {
    if (timer) timer->cls = cls;
  }

  template <typename P = void> P *at(size_t off) const { return reinterpret_cast<P *>(ws + off); }
  void *kc(int l) const { return ws + L.kcache + L.kv_layer_elems * l * elem_bytes(cfg.dtype); }
  void *vc(int l) const { return ws + L.vcache + L.kv_layer_elems * l * elem_bytes(cfg.dtype); }
  ~ll_model() { delete timer; }

  // Paged cache: the pool's free pages (a stack, so the first pages handed out are the
  // highest ids), each sequence's pages in logical order, and the host copy of the block
  // table whose entries are copied to the device when they are first set.
  std::vector<int> free_pages;
  std::vector<std::vector<int>> seq_pages;
  std::vector<int> table_host;
  bool paged() const { return cfg.kv_page > 0; }
  KvPaging paging() const {
    KvPaging p;
    if (paged()) {
      p.table = reinterpret_cast<const int *>(ws + L.kv_table);
      p.page_len = cfg.kv_page;
      p.max_pages = L.kv_max_pages;
    }
    return p;
  }
  void release_pages() {
    free_pages.resize(L.kv_pages);
    for (int i = 0; i < L.kv_pages; ++i) free_pages[i] = i;
    seq_pages.assign(cfg.max_batch, {});
  }
  // Pages sequence b lacks to hold `len` positions.
  int pages_short(int b, long len) const {
    const long need = (len + cfg.kv_page - 1) / cfg.kv_page;
    return (int)std::max(0L, need - (long)seq_pages[b].size());
  }
  // Give sequence b pages up to `len` positions and copy the new table entries to the device
  // (the caller has checked the pool).
  hipError_t grow(int b, long len, hipStream_t s) {
    const int first = (int)seq_pages[b].size(), n = pages_short(b, len);
    if (n == 0) return hipSuccess;
    int *row = table_host.data() + (size_t)b * L.kv_max_pages;
    for (int i = 0; i < n; ++i) {
      row[first + i] = free_pages.back();
      seq_pages[b].push_back(free_pages.back());
      free_pages.pop_back();
    }
    return hipMemcpyAsync(ws + L.kv_table + ((size_t)b * L.kv_max_pages + first) * 4, row + first,
                          (size_t)n * 4, hipMemcpyHostToDevice, s);
  }
  void drop_graphs() {
    for (auto &g : graphs) (void)hipGraphExecDestroy(g.exec);
    graphs.clear();
  }
  // Decode-attention plan: the load-time plan, or the keys-per-block override of
  // LL_OPT_ATTN_DECODE_CHUNK (never more splits than the workspace holds).
  AttnDecodePlan attn_plan() const {
    AttnDecodePlan p = L.attn;
    const int kpb = opt[LL_OPT_ATTN_DECODE_CHUNK];
    if (kpb >= p.kpb) {
      p.kpb = kpb;
      p.nsplit = (cfg.max_ctx + kpb - 1) / kpb;
    }
    return p;
  }
};

namespace {

EpiParams qkv_epi(const ll_model *m, int l, const int *row_seq, const int *row_pos) {
  EpiParams ep;
  ep.kind = kEpiQkv;
  ep.act = m->at(m->L.q);
  ep.ld_act = m->cfg.n_heads * m->cfg.head_dim;
  ep.kcache = m->kc(l);
  ep.vcache = m->vc(l);
  ep.row_seq = row_seq;
  ep.row_pos = row_pos;
  ep.rope_cos = m->at<float>(m->L.rcos);
  ep.rope_sin = m->at<float>(m->L.rsin);
  ep.n_heads = m->cfg.n_heads;
  ep.n_kv_heads = m->cfg.n_kv_heads;
  ep.head_dim = m->cfg.head_dim;
  ep.max_ctx = m->cfg.max_ctx;
  ep.kv_paging = m->paging();
  return ep;
}

EpiParams resid_epi(const ll_model *m) {
  EpiParams ep;
  ep.kind = kEpiResid;
  ep.out_f32 = m->at<float>(m->L.x);
  ep.ld_out = m->cfg.d_model;
  return ep;
}

EpiParams swiglu_epi(const ll_model *m) {
  EpiParams ep;
  ep.kind = kEpiSwiglu;
  ep.act = m->at(m->L.act);
  ep.ld_act = m->cfg.ffn_dim;
  return ep;
}

EpiParams argmax_epi(const ll_model *m, float *logits) {
  EpiParams ep;
  ep.kind = kEpiArgmax;
  ep.out_f32 = logits;
  ep.ld_out = m->cfg.vocab;
  ep.part_val = m->at<float>(m->L.pval);
  ep.part_idx = m->at<int>(m->L.pidx);
  ep.n_parts = m->L.n_parts;
  return ep;
}

// Decode batches up to this size normalise inside the decode GEMM (the fp32 rows are then
// read by every column block, which stays cheap only for a few rows).
constexpr int kFusedNormMaxRows = 16;
// The decoder layers for `rows` rows.  decode: one row per sequence at position len[b].
// *hf_ready: the last layer's down projection also wrote the final RMSNorm rows into hf.
ll_status enqueue_layers(ll_model *m, int rows, bool decode, int n_qtiles, hipStream_t s,
                         bool *hf_ready = nullptr, const AttnSched *as = nullptr) {
  if (hf_ready) *hf_ready = false;
  const ll_config &c = m->cfg;
  const int d = c.d_model, qd = c.n_heads * c.head_dim, F = c.ffn_dim;
  const int dt = compute_dtype(c);
  const bool fuse_norm = decode && rows <= kFusedNormMaxRows &&
                         skinny_norm_lds(elem_bytes(dt), rows, d) <= kSkinnyMaxNormLds;
  const AttnDecodePlan ap = m->attn_plan();
  // LL_OPT_DECODE_FUSED: the O projection merges the attention splits while staging its A rows
  // (the merge kernel is not launched).
  const bool merge_in_o = decode && m->opt[LL_OPT_DECODE_FUSED] && ap.nsplit > 1 &&
                          ap.nsplit <= kCombineDirectSplits && rows <= kFusedNormMaxRows &&
                          skinny_norm_lds(elem_bytes(dt), rows, qd) <= kSkinnyMaxNormLds;
  NormIn merge_a;
  if (merge_in_o)
    merge_a.merge = AttnMergeIn{m->at<float>(m->L.part_o), m->at<float>(m->L.part_ml),
                                m->at<int>(m->L.lens), 1, c.head_dim, ap.kpb, ap.nsplit,
                                c.max_ctx};
  float *x = m->at<float>(m->L.x);
  float *splitk_ws = m->L.splitk_bytes ? m->at<float>(m->L.splitk) : nullptr;
  const bool use_split = decode ? m->opt[LL_OPT_DECODE_SPLITK] : m->opt[LL_OPT_PREFILL_SPLITK];
  float *gemm_ws = use_split ? splitk_ws : nullptr;
  const size_t gemm_ws_bytes = use_split ? m->L.splitk_bytes : 0;
  // h_ready: the previous residual GEMM already wrote the next RMSNorm rows into h (split-K
  // decode GEMMs fold the norm into their final reduction).
  bool h_ready = false;
  auto gemm = [&](const void *a, int lda, const NormIn *nrm, const void *wt, int n, int k,
                  const EpiParams &ep, const PostNorm *post = nullptr, bool *post_done = nullptr) {
    return decode ? launch_gemm_skinny(dt, a, lda, nrm, wt, rows, n, k, ep, s, gemm_ws,
                                       gemm_ws_bytes, post, post_done,
                                       m->opt[LL_OPT_DECODE_SPLITK] == 2 ? 2 : 1)
                  : launch_gemm_tiled(dt, a, lda, wt, rows, n, k, ep, s, gemm_ws, gemm_ws_bytes,
                                      m->opt[LL_OPT_PREFILL_TILE]);
  };
  auto post_norm = [&](size_t gain_off, size_t out_off) {
    PostNorm p;
    p.gain = m->at(gain_off);
    p.eps = c.rms_eps;
    p.out = m->at(out_off);
    p.ld_out = d;
    return p;
  };
  // The A operand of a projection that follows an RMSNorm: normalised in the GEMM, already in
  // h, or normalised by a separate row kernel into h.
  auto normed = [&](size_t gain_off, NormIn *nrm) -> ll_status {
    if (fuse_norm) {
      *nrm = NormIn{x, d, nullptr, m->at(gain_off), c.rms_eps};
      return LL_OK;
    }
    if (h_ready) {
      h_ready = false;
      return LL_OK;
    }
    m->mark(LL_K_RMSNORM);
    LL_HIP(launch_rmsnorm(dt, x, d, nullptr, rows, d, m->at(gain_off), c.rms_eps,
                          m->at(m->L.h), d, s));
    return LL_OK;
  };
  for (int l = 0; l < c.n_layers; ++l) {
    NormIn nrm;
    ll_status st = normed(m->L.attn_norm[l], &nrm);
    if (st != LL_OK) return st;
    const int *row_seq = decode ? nullptr : m->at<int>(m->L.row_seq);
    const int *row_pos = decode ? m->at<int>(m->L.lens) : m->at<int>(m->L.row_pos);
    m->mark(LL_K_QKV);
    LL_HIP(gemm(m->at(m->L.h), d, fuse_norm ? &nrm : nullptr, m->at(m->L.wqkv[l]), m->L.n_qkv,
                d, qkv_epi(m, l, row_seq, row_pos)));
    m->mark(LL_K_ATTN);
    if (decode) {
      LL_HIP(launch_attn_decode(dt, c.head_dim, m->at(m->L.q), qd, m->kc(l), m->vc(l),
                                m->at<int>(m->L.lens), 1, m->at(m->L.o), qd, rows, c.n_heads,
                                c.n_kv_heads, c.max_ctx, ap, m->at<float>(m->L.part_o),
                                m->at<float>(m->L.part_ml), s, merge_in_o, m->paging()));
    } else {
      LL_HIP(launch_attn_prefill(dt, c.head_dim, m->at(m->L.q), qd, m->kc(l), m->vc(l),
                                 m->at(m->L.o), qd, m->at<int>(m->L.cu),
                                 m->at<int>(m->L.kstart), m->at<int2>(m->L.qtiles), n_qtiles,
                                 c.n_heads, c.n_kv_heads, c.max_ctx, s, m->paging(),
                                 m->L.sched ? m->at<int4>(m->L.sched) : nullptr, as));
    }
    m->mark(LL_K_O);
    {
      const PostNorm pn = post_norm(m->L.mlp_norm[l], m->L.h);
      LL_HIP(gemm(m->at(m->L.o), qd, merge_in_o ? &merge_a : nullptr, m->at(m->L.wo[l]), d, qd,
                  resid_epi(m), fuse_norm ? nullptr : &pn, &h_ready));
    }
    st = normed(m->L.mlp_norm[l], &nrm);
    if (st != LL_OK) return st;
    m->mark(LL_K_GATE_UP);
    LL_HIP(gemm(m->at(m->L.h), d, fuse_norm ? &nrm : nullptr, m->at(m->L.wgu[l]), 2 * F, d,
                swiglu_epi(m)));
    m->mark(LL_K_DOWN);
    const bool last = l + 1 == c.n_layers;
    const PostNorm pn = last ? post_norm(m->L.final_norm, m->L.hf)
                             : post_norm(m->L.attn_norm[l + 1], m->L.h);
    bool done = false;
    LL_HIP(gemm(m->at(m->L.act), F, nullptr, m->at(m->L.wd[l]), d, F, resid_epi(m),
                fuse_norm ? nullptr : &pn, &done));
    if (last) {
      if (hf_ready) *hf_ready = done;
    } else {
      h_ready = done;
    }
  }
  return LL_OK;
}

// Final RMSNorm of one row per sequence, the LM head with per-block argmax partials, and the
// reduction that writes `next` (and advances `lens_inc`).
ll_status enqueue_head(ll_model *m, int batch, const int *rowmap, int *next, float *logits,
                       int *lens_inc, hipStream_t s, bool hf_ready = false) {
  const ll_config &c = m->cfg;
  EpiParams ep = argmax_epi(m, logits);
  NormIn nrm{m->at<float>(m->L.x), c.d_model, rowmap, m->at(m->L.final_norm), c.rms_eps};
  const bool fuse_norm = batch <= kFusedNormMaxRows &&
                         skinny_norm_lds(elem_bytes(compute_dtype(c)), batch, c.d_model) <= kSkinnyMaxNormLds;
  if (!fuse_norm && !hf_ready) {
    m->mark(LL_K_RMSNORM);
    LL_HIP(launch_rmsnorm(compute_dtype(c), m->at<float>(m->L.x), c.d_model, rowmap, batch, c.d_model,
                          m->at(m->L.final_norm), c.rms_eps, m->at(m->L.hf), c.d_model, s));
  }
  m->mark(LL_K_LM_HEAD);
  LL_HIP(launch_gemm_skinny(compute_dtype(c), m->at(m->L.hf), c.d_model, fuse_norm ? &nrm : nullptr,
                            m->at(m->L.lm_head), batch, c.vocab, c.d_model, ep, s));
  m->mark(LL_K_ARGMAX);
  LL_HIP(launch_argmax_reduce(ep.part_val, ep.part_idx, batch, ep.n_parts, next, lens_inc, s));
  return LL_OK;
}

ll_status enqueue_decode(ll_model *m, const int32_t *in, int32_t *out, float *logits,
                         hipStream_t s) {
  const ll_config &c = m->cfg;
  m->mark(LL_K_EMBED);
  LL_HIP(launch_embed(compute_dtype(c), in, m->batch, m->at(m->L.embed), c.vocab, c.d_model,
                      m->at<float>(m->L.x), m->at<int>(m->L.err), s));
  bool hf_ready = false;
  ll_status st = enqueue_layers(m, m->batch, true, 0, s, &hf_ready);
  if (st != LL_OK) return st;
  return enqueue_head(m, m->batch, nullptr, out, logits, m->at<int>(m->L.lens), s, hf_ready);
}

}  // namespace

extern "C" {

const char *ll_last_error(void) { return ll::g_err.c_str(); }

ll_status ll_workspace_size(const ll_config *cfg, size_t *bytes) {
  g_err.clear();
  if (!bytes) return fail(LL_ERR_INVALID_ARGUMENT, "bytes is NULL");
  ll_status st = validate_config(cfg);
  if (st != LL_OK) return st;
  *bytes = make_layout(*cfg).total;
  return LL_OK;
}

ll_status ll_model_load(const ll_config *cfg, const ll_weights *w, void *workspace,
                        size_t workspace_bytes, void *hip_stream, ll_model **out) {
  g_err.clear();
  if (!out) return fail(LL_ERR_INVALID_ARGUMENT, "out is NULL");
  *out = nullptr;
  ll_status st = validate_config(cfg);
  if (st != LL_OK) return st;
  if (!w) return fail(LL_ERR_INVALID_ARGUMENT, "weights is NULL");
  if (!w->tok_embed || !w->final_norm || !w->lm_head)
    return fail(LL_ERR_INVALID_ARGUMENT, "tok_embed, final_norm and lm_head must be set");
  const void *const *arrays[] = {w->attn_norm, w->wq, w->wk, w->wv, w->wo,
                                 w->mlp_norm, w->w_gate, w->w_up, w->w_down};
  for (auto a : arrays) {
    if (!a) return fail(LL_ERR_INVALID_ARGUMENT, "a per-layer weight array is NULL");
    for (int l = 0; l < cfg->n_layers; ++l)
      if (!a[l]) return fail(LL_ERR_INVALID_ARGUMENT, "layer %d weight pointer is NULL", l);
  }
  if ((st = check_ws(workspace)) != LL_OK) return st;
  const Layout L = make_layout(*cfg);
  if (workspace_bytes < L.total)
    return fail(LL_ERR_WORKSPACE, "workspace has %zu bytes, needs %zu", workspace_bytes, L.total);

  ll_model *m = new ll_model();
  m->cfg = *cfg;
  m->L = L;
  m->ws = reinterpret_cast<char *>(workspace);
  m->stream = reinterpret_cast<hipStream_t>(hip_stream);
  const ll_config &c = *cfg;
  const size_t eb = elem_bytes(c.dtype);
  const int d = c.d_model, qd = c.n_heads * c.head_dim, kvd = c.n_kv_heads * c.head_dim;
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

  const int cdt = compute_dtype(c);
  int *err = m->at<int>(L.err);
  LOAD_HIP(hipMemsetAsync(err, 0, 4, s));
  // Vectors copied as they are, or converted to fp16 (f16_compute).
  auto copy_vec = [&](size_t off, const void *src, size_t n) {
    return cdt == c.dtype ? hipMemcpyAsync(m->at(off), src, n * eb, hipMemcpyDeviceToDevice, s)
                          : launch_bf16_to_f16(src, m->at(off), n, err, s);
  };
  auto repack = [&](const RepackSrc &src, int n, int k, int perm, size_t off) {
    return launch_repack(cdt, src, n, k, perm, c.head_dim, c.ffn_dim, m->at(off), s, c.dtype, err);
  };
  LOAD_HIP(copy_vec(L.embed, w->tok_embed, (size_t)c.vocab * d));
  LOAD_HIP(copy_vec(L.final_norm, w->final_norm, d));
  for (int l = 0; l < c.n_layers; ++l) {
    RepackSrc qkv{{w->wq[l], w->wk[l], w->wv[l]}, {qd, kvd, kvd}};
    LOAD_HIP(repack(qkv, L.n_qkv, d, kPermRope, L.wqkv[l]));
    RepackSrc wo{{w->wo[l], nullptr, nullptr}, {d, 0, 0}};
    LOAD_HIP(repack(wo, d, qd, kPermNone, L.wo[l]));
    RepackSrc gu{{w->w_gate[l], w->w_up[l], nullptr}, {c.ffn_dim, c.ffn_dim, 0}};
    LOAD_HIP(repack(gu, 2 * c.ffn_dim, d, kPermGlu, L.wgu[l]));
    RepackSrc wd{{w->w_down[l], nullptr, nullptr}, {d, 0, 0}};
    LOAD_HIP(repack(wd, d, c.ffn_dim, kPermNone, L.wd[l]));
    LOAD_HIP(copy_vec(L.attn_norm[l], w->attn_norm[l], d));
    LOAD_HIP(copy_vec(L.mlp_norm[l], w->mlp_norm[l], d));
  }
  RepackSrc lm{{w->lm_head, nullptr, nullptr}, {c.vocab, 0, 0}};
  LOAD_HIP(repack(lm, c.vocab, d, kPermNone, L.lm_head));
  // RoPE table in fp64 on the host, stored as fp32: [pos][i] = cos / sin(pos * theta^(-2i/hd)).
  const int half = c.head_dim / 2;
  m->rope_host.resize((size_t)2 * c.max_ctx * half);
  float *hc = m->rope_host.data(), *hs = hc + (size_t)c.max_ctx * half;
  for (int p = 0; p < c.max_ctx; ++p)
    for (int i = 0; i < half; ++i) {
      const double ang = (double)p * std::pow(c.rope_theta, -2.0 * i / c.head_dim);
      hc[(size_t)p * half + i] = (float)std::cos(ang);
      hs[(size_t)p * half + i] = (float)std::sin(ang);
    }
  LOAD_HIP(hipMemcpyAsync(m->at(L.rcos), hc, (size_t)c.max_ctx * half * 4, hipMemcpyHostToDevice, s));
  LOAD_HIP(hipMemcpyAsync(m->at(L.rsin), hs, (size_t)c.max_ctx * half * 4, hipMemcpyHostToDevice, s));
  if (m->paged()) {
    const size_t entries = (size_t)c.max_batch * L.kv_max_pages;
    LOAD_HIP(hipMemsetAsync(m->at(L.kv_table), 0, entries * 4, s));
    m->table_host.assign(entries, 0);
    m->release_pages();
  }

#undef LOAD_HIP
  *out = m;
  return LL_OK;
}

ll_status ll_prefill(ll_model *m, int32_t batch, const int32_t *seq_lens_host,
                     const int32_t *tokens_dev, int32_t *next_tokens_dev, float *logits_dev) {
  g_err.clear();
  if (!m) return fail(LL_ERR_INVALID_ARGUMENT, "model is NULL");
  if (!seq_lens_host || !tokens_dev || !next_tokens_dev)
    return fail(LL_ERR_INVALID_ARGUMENT, "seq_lens_host, tokens_dev and next_tokens_dev must be set");
  if (batch < 1) return fail(LL_ERR_INVALID_ARGUMENT, "batch %d < 1", batch);
  const ll_config &c = m->cfg;
  if (batch > c.max_batch) return fail(LL_ERR_CAPACITY, "batch %d > max_batch %d", batch, c.max_batch);
  // A prefill on a populated cache (chunked prefill) extends the same sequences.
  const bool chunk = m->batch != 0;
  if (chunk && batch != m->batch)
    return fail(LL_ERR_STATE, "prefill of %d sequences on a cache holding %d (a further prefill "
                "chunk extends the same sequences; ll_kv_reset starts new ones)", batch, m->batch);
  long total = 0;
  int n_qtiles = 0;
  const int qtile = attn_prefill_qtile(compute_dtype(c));
  PrefillMeta pm;
  pm.batch = batch;
  for (int b = 0; b < batch; ++b) {
    const int L = seq_lens_host[b];
    const int P0 = chunk ? m->lens[b] : 0;
    if (L < 1) return fail(LL_ERR_INVALID_ARGUMENT, "seq_lens[%d] = %d < 1", b, L);
    if ((long)P0 + L > c.max_ctx)
      return fail(LL_ERR_CAPACITY, "sequence %d: %d cached + %d new tokens > max_ctx %d", b, P0,
                  L, c.max_ctx);
    total += L;
    n_qtiles += (L + qtile - 1) / qtile;
    pm.lens[b] = L;
    pm.start[b] = P0;
  }
  if (total > c.max_prefill_tokens)
    return fail(LL_ERR_CAPACITY, "%ld prompt tokens > max_prefill_tokens %d", total, c.max_prefill_tokens);
  const int T = (int)total;
  hipStream_t s = m->stream;
  const Layout &L = m->L;
  if (m->paged()) {
    long short_pages = 0;
    for (int b = 0; b < batch; ++b)
      short_pages += m->pages_short(b, (long)pm.start[b] + pm.lens[b]);
    if (short_pages > (long)m->free_pages.size())
      return fail(LL_ERR_CAPACITY, "the prefill needs %ld new KV pages, %zu are free", short_pages,
                  m->free_pages.size());
    for (int b = 0; b < batch; ++b) LL_HIP(m->grow(b, (long)pm.start[b] + pm.lens[b], s));
  }
  TimerScope scope(m->timer, 0);
  m->mark(LL_K_META);
  const AttnSched as = attn_prefill_sched(pm, c.n_heads / c.n_kv_heads, c.n_kv_heads);
  LL_HIP(launch_prefill_meta(pm, T, qtile, m->at<int>(L.cu), m->at<int>(L.row_seq),
                             m->at<int>(L.row_pos), m->at<int>(L.last_row), m->at<int>(L.lens),
                             m->at<int>(L.kstart), m->at<int2>(L.qtiles), s,
                             L.sched ? m->at<int4>(L.sched) : nullptr, &as, c.n_kv_heads));
  m->mark(LL_K_EMBED);
  LL_HIP(launch_embed(compute_dtype(c), tokens_dev, T, m->at(L.embed), c.vocab, c.d_model,
                      m->at<float>(L.x), m->at<int>(L.err), s));
  ll_status st = enqueue_layers(m, T, false, n_qtiles, s, nullptr, &as);
  if (st != LL_OK) return st;
  st = enqueue_head(m, batch, m->at<int>(L.last_row), next_tokens_dev, logits_dev, nullptr, s);
  if (st != LL_OK) return st;
  if (chunk) {
    for (int b = 0; b < batch; ++b) m->lens[b] += seq_lens_host[b];
  } else {
    m->batch = batch;
    m->lens.assign(seq_lens_host, seq_lens_host + batch);
  }
  return LL_OK;
}

ll_status ll_decode_step(ll_model *m, const int32_t *in_tokens_dev, int32_t *next_tokens_dev,
                         float *logits_dev) {
  g_err.clear();
  if (!m) return fail(LL_ERR_INVALID_ARGUMENT, "model is NULL");
  if (!in_tokens_dev || !next_tokens_dev)
    return fail(LL_ERR_INVALID_ARGUMENT, "in_tokens_dev and next_tokens_dev must be set");
  if (m->batch == 0) return fail(LL_ERR_STATE, "decode before prefill");
  for (int b = 0; b < m->batch; ++b)
    if (m->lens[b] + 1 > m->cfg.max_ctx)
      return fail(LL_ERR_CAPACITY, "sequence %d at length %d is full (max_ctx %d)", b, m->lens[b],
                  m->cfg.max_ctx);
  if (m->paged()) {
    long short_pages = 0;
    for (int b = 0; b < m->batch; ++b) short_pages += m->pages_short(b, (long)m->lens[b] + 1);
    if (short_pages > (long)m->free_pages.size())
      return fail(LL_ERR_CAPACITY, "the decode step needs %ld new KV pages, %zu are free",
                  short_pages, m->free_pages.size());
    for (int b = 0; b < m->batch; ++b) LL_HIP(m->grow(b, (long)m->lens[b] + 1, m->stream));
  }
  TimerScope scope(m->timer, 1);
  if (m->use_graph && !m->timer) {
    hipGraphExec_t exec = nullptr;
    for (auto &g : m->graphs)
      if (g.in == in_tokens_dev && g.out == next_tokens_dev && g.logits == logits_dev &&
          g.batch == m->batch)
        exec = g.exec;
    if (!exec) {
      if (!m->cap_stream) LL_HIP(hipStreamCreateWithFlags(&m->cap_stream, hipStreamNonBlocking));
      LL_HIP(hipStreamBeginCapture(m->cap_stream, hipStreamCaptureModeThreadLocal));
      ll_status st = enqueue_decode(m, in_tokens_dev, next_tokens_dev, logits_dev, m->cap_stream);
      hipGraph_t graph = nullptr;
      hipError_t ec = hipStreamEndCapture(m->cap_stream, &graph);
      if (st != LL_OK) {
        if (graph) (void)hipGraphDestroy(graph);
        return st;
      }
      if (ec != hipSuccess) return fail(LL_ERR_HIP, "hipStreamEndCapture: %s", hipGetErrorString(ec));
      ec = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
      (void)hipGraphDestroy(graph);
      if (ec != hipSuccess) return fail(LL_ERR_HIP, "hipGraphInstantiate: %s", hipGetErrorString(ec));
      if (m->graphs.size() >= 8) {
        (void)hipGraphExecDestroy(m->graphs.front().exec);
        m->graphs.erase(m->graphs.begin());
      }
      m->graphs.push_back({in_tokens_dev, next_tokens_dev, logits_dev, m->batch, exec});
    }
    LL_HIP(hipGraphLaunch(exec, m->stream));
  } else {
    ll_status st = enqueue_decode(m, in_tokens_dev, next_tokens_dev, logits_dev, m->stream);
    if (st != LL_OK) return st;
  }
  for (auto &l : m->lens) ++l;
  return LL_OK;
}

ll_status ll_kv_reset(ll_model *m) {
  g_err.clear();
  if (!m) return fail(LL_ERR_INVALID_ARGUMENT, "model is NULL");
  if (m->paged()) {
    // earlier block-table copies read table_host, whose entries are reused from here on
    LL_HIP(hipStreamSynchronize(m->stream));
    m->release_pages();
  }
  m->batch = 0;
  m->lens.clear();
  return LL_OK;
}

ll_status ll_kv_pages(const ll_model *m, int32_t *used, int32_t *total) {
  g_err.clear();
  if (!m || !used || !total) return fail(LL_ERR_INVALID_ARGUMENT, "NULL argument");
  *total = m->paged() ? m->L.kv_pages : 0;
  *used = m->paged() ? m->L.kv_pages - (int32_t)m->free_pages.size() : 0;
  return LL_OK;
}

ll_status ll_workspace_regions(const ll_model *m, int32_t cap, uint64_t *offsets,
                               uint64_t *bytes, const char **names, int32_t *n) {
  g_err.clear();
  if (!m || !n) return fail(LL_ERR_INVALID_ARGUMENT, "model and n must be set");
  if (cap < 0 || (cap > 0 && (!offsets || !bytes || !names)))
    return fail(LL_ERR_INVALID_ARGUMENT, "cap %d needs offsets, bytes and names", cap);
  const auto &rg = m->L.regions;
  for (int32_t i = 0; i < cap && i < (int32_t)rg.size(); ++i) {
    offsets[i] = rg[i].off;
    bytes[i] = rg[i].bytes;
    names[i] = rg[i].name.c_str();
  }
  *n = (int32_t)rg.size();
  return LL_OK;
}

ll_status ll_seq_lengths(const ll_model *m, int32_t *out, int32_t cap, int32_t *n) {
  g_err.clear();
  if (!m || !n || (cap > 0 && !out)) return fail(LL_ERR_INVALID_ARGUMENT, "NULL argument");
  *n = m->batch;
  for (int b = 0; b < m->batch && b < cap; ++b) out[b] = m->lens[b];
  return LL_OK;
}

ll_status ll_set_decode_graph(ll_model *m, int32_t enable) {
  return ll_set_option(m, LL_OPT_DECODE_GRAPH, enable != 0);
}

ll_status ll_set_option(ll_model *m, int32_t option, int32_t value) {
  g_err.clear();
  if (!m) return fail(LL_ERR_INVALID_ARGUMENT, "model is NULL");
  switch (option) {
    case LL_OPT_DECODE_GRAPH:
    case LL_OPT_PREFILL_SPLITK:
      if (value != 0 && value != 1) return fail(LL_ERR_INVALID_ARGUMENT, "option %d takes 0 or 1", option);
      break;
    case LL_OPT_DECODE_SPLITK:
      if (value < 0 || value > 2) return fail(LL_ERR_INVALID_ARGUMENT, "decode split-K 0, 1 or 2");
      break;
    case LL_OPT_PREFILL_TILE:
      if (value < 0 || value > 3) return fail(LL_ERR_INVALID_ARGUMENT, "prefill tile 0..3");
      break;
    case LL_OPT_ATTN_DECODE_CHUNK:
      if (value != 0 && value != 64 && value != 128 && value != 256)
        return fail(LL_ERR_INVALID_ARGUMENT, "decode-attention chunk 0, 64, 128 or 256");
      if (value != 0 && value < m->L.attn.kpb)
        return fail(LL_ERR_UNSUPPORTED, "chunk %d below the load-time plan's %d (the workspace "
                    "holds %d splits)", value, m->L.attn.kpb, m->L.attn.nsplit);
      break;
    case LL_OPT_DECODE_FUSED:
      if (value != 0 && value != 1) return fail(LL_ERR_INVALID_ARGUMENT, "decode fused 0 or 1");
      break;
    default:
      return fail(LL_ERR_INVALID_ARGUMENT, "unknown option %d", option);
  }
  if (m->opt[option] != value) m->drop_graphs();  // captured graphs bake the old choice in
  m->opt[option] = value;
  m->use_graph = m->opt[LL_OPT_DECODE_GRAPH] != 0;
  return LL_OK;
}

ll_status ll_get_option(const ll_model *m, int32_t option, int32_t *value) {
  g_err.clear();
  if (!m || !value) return fail(LL_ERR_INVALID_ARGUMENT, "NULL argument");
  if (option < 0 || option >= LL_OPT_COUNT) return fail(LL_ERR_INVALID_ARGUMENT, "unknown option %d", option);
  *value = m->opt[option];
  return LL_OK;
}

ll_status ll_device_flags(ll_model *m, int32_t *flags) {
  g_err.clear();
  if (!m || !flags) return fail(LL_ERR_INVALID_ARGUMENT, "NULL argument");
  LL_HIP(hipStreamSynchronize(m->stream));
  LL_HIP(hipMemcpy(flags, m->at(m->L.err), 4, hipMemcpyDeviceToHost));
  return LL_OK;
}

ll_status ll_set_kernel_timing(ll_model *m, int32_t enable) {
  g_err.clear();
  if (!m) return fail(LL_ERR_INVALID_ARGUMENT, "model is NULL");
  if (enable && !m->timer) m->timer = new Timer(LL_K_ATTN, LL_K_ATTN_COMBINE);
  if (!enable && m->timer) {
    (void)hipStreamSynchronize(m->stream);
    delete m->timer;
    m->timer = nullptr;
  }
  return LL_OK;
}

ll_status ll_kernel_timing_read(ll_model *m, int32_t *counts, double *ms) {
  g_err.clear();
  if (!m || !counts || !ms) return fail(LL_ERR_INVALID_ARGUMENT, "NULL argument");
  for (int i = 0; i < 2 * LL_K_COUNT; ++i) {
    counts[i] = 0;
    ms[i] = 0.0;
  }
  if (!m->timer) return fail(LL_ERR_STATE, "kernel timing is not enabled");
  return m->timer->drain(m->stream, LL_K_COUNT, counts, ms);
}

const char *ll_kernel_class_name(int32_t cls) {
  return (cls >= 0 && cls < LL_K_COUNT) ? kClassNames[cls] : "";
}

void ll_model_free(ll_model *m) {
  if (!m) return;
  m->drop_graphs();
  if (m->cap_stream) (void)hipStreamDestroy(m->cap_stream);
  delete m;
}

// ----------------------------------------------------------------------------------------
// Per-kernel entry points
// ----------------------------------------------------------------------------------------

static ll_status check_dtype(int32_t dtype) {
  if (dtype != LL_F32 && dtype != LL_BF16 && dtype != LL_F16)
    return fail(LL_ERR_UNSUPPORTED, "dtype %d unknown", dtype);
  return LL_OK;
}

ll_status ll_op_rmsnorm(int32_t dtype, int32_t rows, int32_t d, const float *x, const void *gain,
                        float eps, void *y, void *stream) {
  g_err.clear();
  ll_status st = check_dtype(dtype);
  if (st != LL_OK) return st;
  if (rows < 0 || d < 4 || d % 4) return fail(LL_ERR_INVALID_ARGUMENT, "rows >= 0, d a multiple of 4");
  if (rows && (!x || !gain || !y)) return fail(LL_ERR_INVALID_ARGUMENT, "NULL pointer");
  LL_HIP(launch_rmsnorm(dtype, x, d, nullptr, rows, d, gain, eps, y, d, (hipStream_t)stream));
  return LL_OK;
}

ll_status ll_op_mfma_loop(int32_t blocks, int32_t iters, float *out_dev, void *stream) {
  g_err.clear();
  if (blocks < 1 || iters < 1 || !out_dev)
    return fail(LL_ERR_INVALID_ARGUMENT, "blocks >= 1, iters >= 1 and out_dev must be set");
  LL_HIP(launch_mfma_loop(blocks, iters, out_dev, (hipStream_t)stream));
  return LL_OK;
}

ll_status ll_op_read_stream(const float *src_dev, int64_t n, int32_t blocks, float *out_dev,
                            void *stream) {
  g_err.clear();
  if (n < 0 || n % 4 || blocks < 1 || !out_dev)
    return fail(LL_ERR_INVALID_ARGUMENT, "n >= 0 a multiple of 4, blocks >= 1 and out_dev required");
  if (n > 0 && (!src_dev || (reinterpret_cast<uintptr_t>(src_dev) & 15)))
    return fail(LL_ERR_INVALID_ARGUMENT, "src_dev must be set and 16-byte aligned");
  LL_HIP(launch_read_stream(src_dev, (long)n, blocks, out_dev, (hipStream_t)stream));
  return LL_OK;
}

ll_status ll_op_repack(int32_t dtype, int32_t n, int32_t k, const void *w, void *wt, void *stream) {
  g_err.clear();
  ll_status st = check_dtype(dtype);
  if (st != LL_OK) return st;
  if (n < 16 || n % 16 || k < 64 || k % 64) return fail(LL_ERR_UNSUPPORTED, "n %% 16, k %% 64 required");
  if (!w || !wt) return fail(LL_ERR_INVALID_ARGUMENT, "NULL pointer");
  RepackSrc src{{w, nullptr, nullptr}, {n, 0, 0}};
  LL_HIP(launch_repack(dtype, src, n, k, kPermNone, 64, 64, wt, (hipStream_t)stream));
  return LL_OK;
}

ll_status ll_op_gemm(int32_t path, int32_t dtype, int32_t m, int32_t n, int32_t k, const void *a,
                     const void *wt, float *c, int32_t accumulate, void *stream) {
  g_err.clear();
  ll_status st = check_dtype(dtype);
  if (st != LL_OK) return st;
  if (path != 0 && path != 1) return fail(LL_ERR_INVALID_ARGUMENT, "path must be 0 or 1");
  if (m < 0 || n < 1 || k < 1) return fail(LL_ERR_INVALID_ARGUMENT, "bad sizes");
  if (k % 64 || n % (path == 0 ? 128 : 32))
    return fail(LL_ERR_UNSUPPORTED, "k %% 64 and n %% %d required", path == 0 ? 128 : 32);
  if (m && (!a || !wt || !c)) return fail(LL_ERR_INVALID_ARGUMENT, "NULL pointer");
  EpiParams ep;
  ep.kind = accumulate ? kEpiResid : kEpiStore;
  ep.out_f32 = c;
  ep.ld_out = n;
  LL_HIP(path == 0 ? launch_gemm_tiled(dtype, a, k, wt, m, n, k, ep, (hipStream_t)stream)
                   : launch_gemm_skinny(dtype, a, k, nullptr, wt, m, n, k, ep, (hipStream_t)stream));
  return LL_OK;
}

ll_status ll_op_gemm_swiglu(int32_t dtype, int32_t m, int32_t n, int32_t k, const void *a,
                            const void *wt, void *act, void *stream) {
  g_err.clear();
  ll_status st = check_dtype(dtype);
  if (st != LL_OK) return st;
  if (m < 0 || n < 1 || k < 1) return fail(LL_ERR_INVALID_ARGUMENT, "bad sizes");
  if (k % 64 || n % 128) return fail(LL_ERR_UNSUPPORTED, "k %% 64 and n %% 128 required");
  if (m && (!a || !wt || !act)) return fail(LL_ERR_INVALID_ARGUMENT, "NULL pointer");
  EpiParams ep;
  ep.kind = kEpiSwiglu;
  ep.act = act;
  ep.ld_act = n / 2;
  LL_HIP(launch_gemm_tiled(dtype, a, k, wt, m, n, k, ep, (hipStream_t)stream));
  return LL_OK;
}

size_t ll_op_gemm_prefill_splitk_scratch(int32_t dtype, int32_t m, int32_t n, int32_t k) {
  if ((dtype != LL_F32 && dtype != LL_BF16 && dtype != LL_F16) || m < 1 || n < 1 || k < 1 ||
      k % 64)
    return 0;
  return prefill_splitk_plan(elem_bytes(dtype), m, n, k).ws_bytes;
}
ll_status ll_op_gemm_prefill_splitk(int32_t dtype, int32_t m, int32_t n, int32_t k,
                                    const void *a, const void *wt, float *c, int32_t accumulate,
                                    void *scratch, size_t scratch_bytes, void *stream) {
  g_err.clear();
  ll_status st = check_dtype(dtype);
  if (st != LL_OK) return st;
  if (m < 1 || n < 1 || k < 1) return fail(LL_ERR_INVALID_ARGUMENT, "bad sizes");
  const size_t need = ll_op_gemm_prefill_splitk_scratch(dtype, m, n, k);
  if (!need)
    return fail(LL_ERR_UNSUPPORTED, "n %% 128, k %% 64 and fewer than %d tiles of 64 x 128 "
                "required", kPrefillSplitMinTiles);
  if (!a || !wt || !c || !scratch) return fail(LL_ERR_INVALID_ARGUMENT, "NULL pointer");
  if (scratch_bytes < need) return fail(LL_ERR_WORKSPACE, "scratch needs %zu bytes", need);
  EpiParams ep;
  ep.kind = accumulate ? kEpiResid : kEpiStore;
  ep.out_f32 = c;
  ep.ld_out = n;
  LL_HIP(launch_gemm_tiled(dtype, a, k, wt, m, n, k, ep, (hipStream_t)stream,
                           reinterpret_cast<float *>(scratch), scratch_bytes));
  return LL_OK;
}

size_t ll_op_gemm_splitk_scratch(int32_t dtype, int32_t m, int32_t n, int32_t k) {
  if ((dtype != LL_F32 && dtype != LL_BF16 && dtype != LL_F16) || m < 1 || n < 1 || k < 1 ||
      k % 64)
    return 0;
  return splitk_plan(elem_bytes(dtype), m, n, k).ws_bytes;
}

ll_status ll_op_gemm_splitk(int32_t dtype, int32_t m, int32_t n, int32_t k, const void *a,
                            const void *wt, float *c, int32_t accumulate, void *scratch,
                            size_t scratch_bytes, void *stream) {
  g_err.clear();
  ll_status st = check_dtype(dtype);
  if (st != LL_OK) return st;
  if (m < 1 || n < 1 || k < 1) return fail(LL_ERR_INVALID_ARGUMENT, "bad sizes");
  const size_t need = ll_op_gemm_splitk_scratch(dtype, m, n, k);
  if (!need) return fail(LL_ERR_UNSUPPORTED, "m > 16, n %% 128 and k %% 64 required");
  if (!a || !wt || !c || !scratch) return fail(LL_ERR_INVALID_ARGUMENT, "NULL pointer");
  if (scratch_bytes < need) return fail(LL_ERR_WORKSPACE, "scratch needs %zu bytes", need);
  EpiParams ep;
  ep.kind = accumulate ? kEpiResid : kEpiStore;
  ep.out_f32 = c;
  ep.ld_out = n;
  LL_HIP(launch_gemm_skinny(dtype, a, k, nullptr, wt, m, n, k, ep, (hipStream_t)stream,
                            reinterpret_cast<float *>(scratch), scratch_bytes));
  return LL_OK;
}

static ll_status check_heads(int32_t n_heads, int32_t n_kv_heads, int32_t head_dim) {
  if (head_dim != 64 && head_dim != 128) return fail(LL_ERR_UNSUPPORTED, "head_dim %d", head_dim);
  if (n_heads < 1 || n_kv_heads < 1 || n_heads % n_kv_heads)
    return fail(LL_ERR_UNSUPPORTED, "n_heads %% n_kv_heads");
  const int g = n_heads / n_kv_heads;
  if (g != 1 && g != 2 && g != 4 && g != 8) return fail(LL_ERR_UNSUPPORTED, "group %d", g);
  return LL_OK;
}

}  // extern "C"

namespace {
// Device metadata of ll_op_attn_prefill in its scratch buffer (offsets, 256-byte aligned).
struct OpAttnPrefillLayout {
  size_t cu = 0, seq = 0, pos = 0, last = 0, lens = 0, ks = 0, qt = 0, sched = 0, bytes = 0;
  int n_qtiles = 0, total = 0;
  AttnSched as;
  PrefillMeta pm;
};
ll_status op_attn_prefill_layout(int dtype, int batch, const int32_t *seq_lens_host,
                                 const int32_t *cached_host, int n_heads, int n_kv_heads,
                                 int max_ctx, OpAttnPrefillLayout *lay) {
  if (batch < 1 || batch > LL_MAX_BATCH || !seq_lens_host)
    return fail(LL_ERR_INVALID_ARGUMENT, "batch in [1, %d] and seq_lens_host required", LL_MAX_BATCH);
  PrefillMeta &pm = lay->pm;
  pm.batch = batch;
  long total = 0;
  const int qtile = attn_prefill_qtile(dtype);
  for (int b = 0; b < batch; ++b) {
    const int L = seq_lens_host[b], P0 = cached_host ? cached_host[b] : 0;
    if (L < 1 || P0 < 0 || (long)P0 + L > max_ctx)
      return fail(LL_ERR_INVALID_ARGUMENT, "sequence %d: %d cached + %d new keys outside "
                  "[1, max_ctx]", b, P0, L);
    pm.lens[b] = L;
    pm.start[b] = P0;
    total += L;
    lay->n_qtiles += (L + qtile - 1) / qtile;
  }
  if (total > INT32_MAX / 4) return fail(LL_ERR_INVALID_ARGUMENT, "%ld tokens", total);
  lay->total = (int)total;
  if (attn_prefill_gqa(dtype, n_heads / n_kv_heads))
    lay->as = attn_prefill_sched(pm, n_heads / n_kv_heads, n_kv_heads);
  size_t off = 0;
  auto take = [&](size_t bytes) { size_t o2 = off; off = align_up(off + bytes); return o2; };
  lay->cu = take((batch + 1) * 4);
  lay->seq = take(total * 4);
  lay->pos = take(total * 4);
  lay->last = take(batch * 4);
  lay->lens = take(batch * 4);
  lay->ks = take(batch * 4);
  lay->qt = take((size_t)lay->n_qtiles * 8);
  lay->sched = take((size_t)lay->as.n_entries * 16);
  lay->bytes = off;
  return LL_OK;
}
}  // namespace

extern "C" {

size_t ll_op_attn_prefill_scratch(int32_t dtype, int32_t batch, const int32_t *seq_lens_host,
                                  const int32_t *cached_host, int32_t n_heads,
                                  int32_t n_kv_heads, int32_t head_dim, int32_t max_ctx) {
  if (check_dtype(dtype) != LL_OK || check_heads(n_heads, n_kv_heads, head_dim) != LL_OK)
    return 0;
  OpAttnPrefillLayout lay;
  if (op_attn_prefill_layout(dtype, batch, seq_lens_host, cached_host, n_heads, n_kv_heads,
                             max_ctx, &lay) != LL_OK)
    return 0;
  return lay.bytes;
}

ll_status ll_op_attn_prefill(int32_t dtype, int32_t batch, const int32_t *seq_lens_host,
                             const int32_t *cached_host, int32_t n_heads, int32_t n_kv_heads,
                             int32_t head_dim, int32_t max_ctx, const void *q,
                             const void *kcache, const void *vcache, void *o, void *scratch,
                             size_t scratch_bytes, void *stream) {
  g_err.clear();
  ll_status st = check_dtype(dtype);
  if (st == LL_OK) st = check_heads(n_heads, n_kv_heads, head_dim);
  if (st != LL_OK) return st;
  OpAttnPrefillLayout lay;
  if ((st = op_attn_prefill_layout(dtype, batch, seq_lens_host, cached_host, n_heads, n_kv_heads,
                                   max_ctx, &lay)) != LL_OK)
    return st;
  if (!q || !kcache || !vcache || !o || !scratch) return fail(LL_ERR_INVALID_ARGUMENT, "NULL pointer");
  if ((st = check_ws(scratch)) != LL_OK) return st;
  if (lay.bytes > scratch_bytes) return fail(LL_ERR_WORKSPACE, "scratch needs %zu bytes", lay.bytes);
  char *sc = reinterpret_cast<char *>(scratch);
  hipStream_t s = (hipStream_t)stream;
  int4 *sched = lay.as.n_entries ? (int4 *)(sc + lay.sched) : nullptr;
  LL_HIP(launch_prefill_meta(lay.pm, lay.total, attn_prefill_qtile(dtype), (int *)(sc + lay.cu),
                             (int *)(sc + lay.seq), (int *)(sc + lay.pos), (int *)(sc + lay.last),
                             (int *)(sc + lay.lens), (int *)(sc + lay.ks), (int2 *)(sc + lay.qt),
                             s, sched, &lay.as, n_kv_heads));
  const int qd = n_heads * head_dim;
  LL_HIP(launch_attn_prefill(dtype, head_dim, q, qd, kcache, vcache, o, qd, (int *)(sc + lay.cu),
                             (int *)(sc + lay.ks), (int2 *)(sc + lay.qt), lay.n_qtiles, n_heads,
                             n_kv_heads, max_ctx, s, KvPaging{}, sched, &lay.as));
  return LL_OK;
}

size_t ll_op_attn_decode_scratch(int32_t batch, int32_t n_heads, int32_t n_kv_heads,
                                 int32_t head_dim, int32_t max_ctx) {
  if (batch < 1 || n_heads < 1 || n_kv_heads < 1 || head_dim < 1 || max_ctx < 1) return 0;
  const size_t nsplit = std::max(attn_decode_plan(head_dim, 4, batch, n_kv_heads, max_ctx).nsplit,
                                 attn_decode_plan(head_dim, 2, batch, n_kv_heads, max_ctx).nsplit);
  return align_up((size_t)batch * n_heads * nsplit * head_dim * 4) +
         align_up((size_t)batch * n_heads * nsplit * 2 * 4);
}

ll_status ll_op_attn_decode(int32_t dtype, int32_t batch, int32_t n_heads, int32_t n_kv_heads,
                            int32_t head_dim, int32_t max_ctx, const void *q, const void *kcache,
                            const void *vcache, const int32_t *ctx_lens_dev, void *o,
                            void *scratch, size_t scratch_bytes, void *stream) {
  g_err.clear();
  ll_status st = check_dtype(dtype);
  if (st == LL_OK) st = check_heads(n_heads, n_kv_heads, head_dim);
  if (st != LL_OK) return st;
  if (batch < 1 || max_ctx < 1) return fail(LL_ERR_INVALID_ARGUMENT, "batch, max_ctx >= 1");
  if (!q || !kcache || !vcache || !ctx_lens_dev || !o) return fail(LL_ERR_INVALID_ARGUMENT, "NULL pointer");
  if ((st = check_ws(scratch)) != LL_OK) return st;
  const size_t need = ll_op_attn_decode_scratch(batch, n_heads, n_kv_heads, head_dim, max_ctx);
  if (scratch_bytes < need) return fail(LL_ERR_WORKSPACE, "scratch needs %zu bytes", need);
  const AttnDecodePlan plan =
      attn_decode_plan(head_dim, (int)elem_bytes(dtype), batch, n_kv_heads, max_ctx);
  const size_t nsplit = plan.nsplit;
  float *po = reinterpret_cast<float *>(scratch);
  float *pml = reinterpret_cast<float *>(reinterpret_cast<char *>(scratch) +
                                         align_up((size_t)batch * n_heads * nsplit * head_dim * 4));
  const int qd = n_heads * head_dim;
  if (max_ctx > attn_decode_max_ctx())
    return fail(LL_ERR_UNSUPPORTED, "max_ctx %d > %d", max_ctx, attn_decode_max_ctx());
  LL_HIP(launch_attn_decode(dtype, head_dim, q, qd, kcache, vcache, ctx_lens_dev, 0, o, qd, batch,
                            n_heads, n_kv_heads, max_ctx, plan, po, pml, (hipStream_t)stream));
  return LL_OK;
}

ll_status ll_op_lmhead_argmax(int32_t dtype, int32_t rows, int32_t vocab, int32_t k, const void *h,
                              const void *wt, float *logits, int32_t *next, void *scratch,
                              size_t scratch_bytes, void *stream) {
  g_err.clear();
  ll_status st = check_dtype(dtype);
  if (st != LL_OK) return st;
  if (rows < 1 || vocab < 32 || vocab % 32 || k < 64 || k % 64)
    return fail(LL_ERR_UNSUPPORTED, "rows >= 1, vocab %% 32, k %% 64 required");
  if (!h || !wt || !next || !scratch) return fail(LL_ERR_INVALID_ARGUMENT, "NULL pointer");
  const size_t parts = (size_t)rows * (vocab / 32);
  if (scratch_bytes < parts * 8) return fail(LL_ERR_WORKSPACE, "scratch needs %zu bytes", parts * 8);
  EpiParams ep;
  ep.kind = kEpiArgmax;
  ep.out_f32 = logits;
  ep.ld_out = vocab;
  ep.part_val = reinterpret_cast<float *>(scratch);
  ep.part_idx = reinterpret_cast<int *>(reinterpret_cast<char *>(scratch) + parts * 4);
  ep.n_parts = vocab / 32;
  hipStream_t s = (hipStream_t)stream;
  LL_HIP(launch_gemm_skinny(dtype, h, k, nullptr, wt, rows, vocab, k, ep, s));
  LL_HIP(launch_argmax_reduce(ep.part_val, ep.part_idx, rows, ep.n_parts, next, nullptr, s));
  return LL_OK;
}

}  // extern "C"
