// Host-side launch interface of the gfx950 kernels (implemented in the .hip files).
// Every launcher enqueues on `s`, checks hipGetLastError and returns hipSuccess or the error.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace ll {

// Optional per-launch timing.  While a timer is installed on the calling thread, every kernel
// launch takes a (start, stop) event pair from it and goes through hipExtLaunchKernel, which
// stamps the events with the dispatch's own begin and end times.
struct LaunchTimer {
  virtual bool next(hipEvent_t *start, hipEvent_t *stop) = 0;
  // The launcher is about to launch its follow-up kernel (e.g. a split-K combine).
  virtual void secondary() {}
  virtual ~LaunchTimer() {}
};
extern thread_local LaunchTimer *g_launch_timer;

// Operand types.  kF16 carries a bf16 model's weights converted exactly to fp16 (bf16's 8-bit
// significand fits fp16's 11; magnitudes in [2^-17, 65504]) with activations, KV cache and MFMA
// operands in fp16: the same bytes and MFMA rate as bf16 at 8x finer rounding.
enum DType : int { kF32 = 0, kBF16 = 1, kF16 = 2 };

inline size_t elem_bytes(int dtype) { return dtype == kF32 ? 4 : 2; }

// Contraction-axis span of one 1 KiB weight tile (16 rows): 32 bf16 or 16 fp32 elements.
inline int tile_k(int dtype) { return dtype == kF32 ? 16 : 32; }

// Row order of a repacked weight.  Output columns are produced in units of 32 "physical"
// columns: a first half of 16 and a second half of 16 that land in the same lanes, so an
// epilogue can combine the two without moving data between lanes.
enum RepackPerm : int {
  kPermNone = 0,  // physical column == logical row
  kPermRope = 1,  // per head of hd: unit j = dims [16j, 16j+16) | [hd/2 + 16j, hd/2 + 16j + 16)
  kPermGlu = 2,   // unit u = gate rows [16u, 16u+16) | up rows [16u, 16u+16)
};

// Up to three row-major sources stacked along N (e.g. W_q, W_k, W_v), then permuted; rows past
// the sources (when the rows sum to less than N) are written as zeros.
struct RepackSrc {
  const void *src[3];
  int rows[3];
};

// src_dtype (-1: dtype) is the sources' element type: kBF16 sources may be repacked into kF16
// tiles (exact conversion; a value beyond the fp16 range sets bit 1 of *err when err is given).
hipError_t launch_repack(int dtype, const RepackSrc &src, int n, int k, int perm, int head_dim,
                         int ffn_dim, void *wt, hipStream_t s, int src_dtype = -1,
                         int *err = nullptr);

// KV cache addressing.  Contiguous (table null): row pos of (sequence b, kv head h) at
// element ((b hkv + h) max_ctx + pos) hd.  Paged: the cache of a layer is a pool of pages
// [page][hkv][page_len][hd]; table[b * max_pages + pos / page_len] names the physical page
// holding logical page pos / page_len of sequence b.  page_len is a multiple of 256, so every
// 64-key tile of the prefill attention and every decode chunk (at most 256 keys, aligned)
// lies in one page.
struct KvPaging {
  const int *table = nullptr;
  int page_len = 0, max_pages = 0;
};
__host__ __device__ inline size_t kv_row_off(const KvPaging &pg, int b, int kvh, int hkv,
                                             int max_ctx, int pos, int hd) {
  if (!pg.table) return (((size_t)b * hkv + kvh) * max_ctx + pos) * hd;
  const int lp = pos / pg.page_len;
  return (((size_t)pg.table[(size_t)b * pg.max_pages + lp] * hkv + kvh) * pg.page_len +
          (pos - lp * pg.page_len)) * hd;
}

enum EpiKind : int {
  kEpiStore = 0,   // out_f32[m, n] = acc
  kEpiResid = 1,   // out_f32[m, n] += acc   (residual stream update)
  kEpiSwiglu = 2,  // act[m, j] = silu(gate) * up   (kPermGlu weights)
  kEpiQkv = 3,     // RoPE on q, k; q -> act, k / v -> KV cache  (kPermRope weights)
  kEpiArgmax = 4,  // logits (optional) + per-32-column (max, argmax) partials
  kEpiConv = 5,    // Mamba decode in_proj: columns [conv_col0, + conv_n) -> conv step + SiLU
                   // -> act (element type T, row stride conv_n), conv state shifted; the other
                   // columns -> out_f32 (fp32, row stride ld_out) at their own index
  kEpiConvF32 = 6, // the same with act in fp32
  kEpiBiasResid = 7,  // out_f32[m, n] += acc + bias[n]
  kEpiGeglu = 8,      // act[m, j] = gelu_tanh(gate + bias[j]) * (up + bias2[j])  (kPermGlu)
  kEpiRgIn = 9,       // recurrent-block input projection, columns [0, W) | [W, 2W):
                      //   act[m, n] = gelu_tanh(acc + bias[n]) (type T, row stride W);
                      //   v = acc + bias2[n - W]: with conv_state (decode, row = sequence) the
                      //   conv step without activation -> act2 (type T, stride W), conv state
                      //   shifted; without, v -> out_f32[m, n - W] (fp32, stride ld_out)
  kEpiRglru = 10,     // RG-LRU gates on block-diagonal weights: per group of group_n output
                      //   columns (a head: its recurrence-gate and input-gate rows interleaved
                      //   as kPermGlu with ffn = group_n / 2) the A operand starts group_k
                      //   columns further; pair (ra, ix) of channel j gives
                      //   r = sigmoid(ra + bias[j]), i = sigmoid(ix + bias2[j]),
                      //   log a = lam[j] r, g = x[m, j] i (reset ? 1 : sqrt(1 - a^2));
                      //   prefill (no rg_state): out_f32 = (reset ? 0 : a), out2 = g, reset at
                      //   the first row of a sequence of a fresh prefill (row_seq, cu);
                      //   decode: h = a rg_state[m, j] + g -> rg_state, act = T(h * gy[m, j])
};

struct EpiParams {
  int kind = kEpiStore;
  float *out_f32 = nullptr;  // Store / Resid target, Argmax logits (nullable)
  int ld_out = 0;
  void *act = nullptr;       // Swiglu output, Qkv query output (element type T)
  int ld_act = 0;
  // Qkv
  void *kcache = nullptr, *vcache = nullptr;  // [max_batch][n_kv][max_ctx][hd] of this layer
  const int *row_seq = nullptr;  // sequence of each row (nullptr: row index)
  const int *row_pos = nullptr;  // position of each row
  const float *rope_cos = nullptr, *rope_sin = nullptr;  // [max_ctx][hd/2]
  int n_heads = 0, n_kv_heads = 0, head_dim = 0, max_ctx = 0;
  KvPaging kv_paging;  // Qkv: where a cached row lives (default: contiguous)
  // Argmax
  float *part_val = nullptr;
  int *part_idx = nullptr;
  int n_parts = 0;  // partials per row (= N / 32)
  // Conv (row = sequence): conv_state [rows][K-1][conv_n], taps [conv_n][K], bias [conv_n]
  float *conv_state = nullptr;
  const float *conv_w = nullptr, *conv_b = nullptr;
  int conv_k = 0, conv_col0 = 0, conv_n = 0;
  // Bias epilogues and the recurrent block (kEpiBiasResid, kEpiGeglu, kEpiRgIn, kEpiRglru)
  const float *bias = nullptr, *bias2 = nullptr;
  void *act2 = nullptr;
  float *out2 = nullptr;
  const float *lam = nullptr;      // -c softplus(lambda) per channel
  float *rg_state = nullptr;       // [rows][width] recurrent state (decode)
  const void *rg_x = nullptr;      // the gates' A operand (type T, [rows][width])
  const void *rg_gy = nullptr;     // gelu branch (type T, [rows][width]) (decode)
  const int *cu = nullptr;         // first row of each sequence (prefill)
  int rg_fresh = 0, width = 0, group_n = 0, group_k = 0;
};

// Decode attention merges at most this many splits in one pass (all loads up front).
constexpr int kCombineDirectSplits = 16;

// A operand of the decode O projection built from the decode attention's split partials
// (part_o [row][head][split][head_dim], part_ml [row][head][split][2] = (max, sum), as
// launch_attn_decode leaves them with skip_merge): row b, column h * head_dim + d holds the
// merged output of head h, rounded to the GEMM type -- the value the merge kernel would have
// written.  2 <= nsplit <= kCombineDirectSplits; rows use min(lens[b] + len_add, max_ctx) keys.
struct AttnMergeIn {
  const float *part_o = nullptr, *part_ml = nullptr;
  const int *lens = nullptr;
  int len_add = 0, head_dim = 0, kpb = 0, nsplit = 0, max_ctx = 0;
};

// RMSNorm computed inside the decode GEMM (A = RMSNorm(x[rowmap[r]]) * gain), or, when
// merge.part_o is set (x and gain unused), the attention merge above.
struct NormIn {
  const float *x = nullptr;
  int ldx = 0;
  const int *rowmap = nullptr;  // nullable
  const void *gain = nullptr;
  float eps = 0.f;
  AttnMergeIn merge;
};

// Prefill GEMM: MFMA on tiles streamed into LDS through a 4-stage ring (256 x 256 or
// 128 x 256 tiles when they fill the CUs, else 64 x 128).  Requires N % 128 == 0, K % 64 == 0.
// When the 64 x 128 tiles are too few to fill the CUs and `ws` holds
// prefill_splitk_plan(...).ws_bytes bytes, K is split over blocks and a second kernel adds the
// fp32 partials in split order and runs the epilogue (not for the argmax epilogue).
// `tile` forces a tile family where the shape allows it (256-column tiles need N % 256 == 0).
enum GemmTile : int { kTileAuto = 0, kTile256 = 1, kTile128x256 = 2, kTileMid = 3 };
hipError_t launch_gemm_tiled(int dtype, const void *a, int lda, const void *wt, int m, int n,
                             int k, const EpiParams &ep, hipStream_t s, float *ws = nullptr,
                             size_t ws_bytes = 0, int tile = kTileAuto);
// Decode GEMM: weights streamed once from HBM into MFMA operands, A read from L2.
// Requires N % 32 == 0, K % 64 == 0; any M (rows handled 32 at a time).  With `norm` the A
// operand is RMSNorm of fp32 rows computed in the kernel (`a` is then unused); that needs
// M <= 16 and skinny_norm_lds(elem, M, K) <= kSkinnyMaxNormLds (the rows are staged in LDS).
constexpr size_t kSkinnyMaxNormLds = 48 * 1024;
inline size_t skinny_norm_lds(size_t elem, int rows, int k) {
  return (size_t)(rows < 16 ? rows : 16) * (k + 16 / elem) * elem;
}
// Above 16 rows, with a workspace of at least splitk_plan(...).ws_bytes bytes (`ws`), the
// decode GEMM splits K over blocks of 128 columns and reduces the fp32 partials in a second
// kernel (not for the argmax epilogue); without one it takes the whole-K path.
// With `post` and the residual epilogue, the split-K path also writes the RMSNorm of the
// updated residual rows (post->out = rows of x times 1/rms times gain, in the workload dtype),
// and sets *post_done; the other paths leave that to a separate RMSNorm launch.
struct PostNorm {
  const void *gain = nullptr;
  float eps = 0.f;
  void *out = nullptr;
  int ld_out = 0;
};
// ksplit = 2 (residual epilogues, up to 16 rows): K is split over two blocks per column block,
// each adding its partial sum into the fp32 rows with atomics (the bias once), so twice the
// blocks stream the weights; the summation order is then not fixed.  Other epilogues ignore
// it.
hipError_t launch_gemm_skinny(int dtype, const void *a, int lda, const NormIn *norm,
                              const void *wt, int m, int n, int k, const EpiParams &ep,
                              hipStream_t s, float *ws = nullptr, size_t ws_bytes = 0,
                              const PostNorm *post = nullptr, bool *post_done = nullptr,
                              int ksplit = 1);
constexpr int kSplitKMaxTiles = 64;  // k-tiles per split-K block (A slice of up to 128 KiB in LDS)
constexpr int kSplitKBlocks = 256;   // blocks the decode split-K plan aims for
struct SplitKPlan {
  int nsplit = 0;  // 0: split-K not used for this shape
  int kts = 0;     // k-tiles per split
  size_t ws_bytes = 0;
};
SplitKPlan splitk_plan(size_t elem, int m, int n, int k);
// Split of the 64 x 128-tile prefill GEMM (kts = k-tiles per split, even).
constexpr int kPrefillSplitMinTiles = 96;  // tiles from which the GEMM is not split
constexpr int kPrefillSplitBlocks = 256;   // blocks the split aims for
constexpr int kPrefillSplitMax = 8;
SplitKPlan prefill_splitk_plan(size_t elem, int m, int n, int k);

hipError_t launch_embed(int dtype, const int *tokens, int ntok, const void *table, int vocab,
                        int d, float *x, int *err_flags, hipStream_t s, float scale = 1.f);
// dst[i] = fp16(src[i]) for n bf16 values (see kF16); an out-of-range value sets bit 1 of *err.
hipError_t launch_bf16_to_f16(const void *src, void *dst, size_t n, int *err, hipStream_t s);
hipError_t launch_rmsnorm(int dtype, const float *x, int ldx, const int *rowmap, int rows,
                          int d, const void *gain, float eps, void *y, int ldy, hipStream_t s);
// next[r] = column of the largest argmax partial of row r (lowest column on ties); lens_inc[r]
// += 1 when lens_inc is given.
// MFMA-only calibration loop: `blocks` blocks of 4 waves, each wave iters x 8 MFMAs of
// 16x16x32 bf16 (2 * 16 * 16 * 32 flops each); out receives 4 floats per block.
hipError_t launch_mfma_loop(int blocks, int iters, float *out, hipStream_t s);
hipError_t launch_read_stream(const float *src, long n, int blocks, float *out, hipStream_t s);
hipError_t launch_argmax_reduce(const float *part_val, const int *part_idx, int rows,
                                int n_parts, int *next, int *lens_inc, hipStream_t s);

// Prefill metadata from host lengths (passed by value).  Sequence b contributes lens[b] new
// tokens at positions start[b] .. start[b] + lens[b] - 1 (start[b] = tokens already cached;
// 0 for a prefill on an empty cache).  Writes cu_seqlens[B+1] (packed query offsets),
// row_seq[T], row_pos[T], last_row[B], lens_dev[B] = start + lens, kstart[B] = start
// (nullable) and the query-tile list ordered by decreasing causal work.
struct PrefillMeta {
  int batch;
  int lens[256];
  int start[256];
};
// Grouped-query prefill attention (bf16, group = n_heads / n_kv_heads >= 2): one block of 8
// waves per (query tile of attn_gqa_qtile(group) queries, KV head) covers every query head of
// the group, so each K / V tile is read from memory once for the whole group.  The blocks'
// work list (sequence, query tile, KV head) is written on the device in a fixed order --
// sequence, KV head, query tiles from the last (the longest) -- and cut into kXcds contiguous
// ranges of near-equal causal work: workgroup i runs on XCD i % kXcds, which takes range
// i % kXcds entry by entry, so the tiles of one (sequence, KV head) share that XCD's L2.
constexpr int kXcds = 8;
struct AttnSched {
  int qtile = 0;      // queries per block
  int n_entries = 0;  // blocks with work
  int grid = 0;       // workgroups launched (kXcds x the longest range)
  int cut[kXcds + 1] = {};
};
inline bool attn_prefill_gqa(int dtype, int group) { return dtype != kF32 && group >= 2; }
inline int attn_gqa_qtile(int group) { return 256 / group; }
AttnSched attn_prefill_sched(const PrefillMeta &pm, int group, int n_kv_heads);
// sched (nullable): the work list of the grouped-query kernel, sized by as->n_entries.
hipError_t launch_prefill_meta(const PrefillMeta &pm, int total, int qtile, int *cu_seqlens,
                               int *row_seq, int *row_pos, int *last_row, int *lens_dev,
                               int *kstart, int2 *qtiles, hipStream_t s, int4 *sched = nullptr,
                               const AttnSched *as = nullptr, int n_kv_heads = 0);
constexpr int kAttnQTile = 64;       // queries per block, fp32 prefill attention
constexpr int kAttnQTileWide = 128;  // queries per block, bf16 prefill attention
// Query-tile size the prefill attention kernel for (dtype, head_dim) expects in `qtiles`.
inline int attn_prefill_qtile(int dtype) { return dtype == kF32 ? kAttnQTile : kAttnQTileWide; }

// Causal prefill attention of the packed queries over each sequence's cache: query i of
// sequence b sits at position kstart[b] + i and attends to cached keys 0 .. kstart[b] + i
// (kstart nullable: every sequence starts at 0).
// With attn_prefill_gqa(dtype, group) the grouped-query kernel runs over `sched` / `as`
// (qtiles / n_qtiles unused); otherwise one block per (query tile, query head) over qtiles.
hipError_t launch_attn_prefill(int dtype, int head_dim, const void *q, int ldq,
                               const void *kcache, const void *vcache, void *o, int ldo,
                               const int *cu_seqlens, const int *kstart, const int2 *qtiles,
                               int n_qtiles, int n_heads, int n_kv_heads, int max_ctx,
                               hipStream_t s, const KvPaging &pg = KvPaging{},
                               const int4 *sched = nullptr, const AttnSched *as = nullptr);

// Decode attention: split over the cache length (chunk keys per block), then a merge kernel.
// Keys attended per sequence: lens[b] + len_add (clamped to max_ctx).
struct AttnDecodePlan {
  int kpb = 0;     // cached keys per block
  int nsplit = 0;  // blocks per (sequence, kv head); 1 = no merge kernel
};
AttnDecodePlan attn_decode_plan(int head_dim, int elem_bytes, int batch, int n_kv_heads,
                                int max_ctx);
int attn_decode_max_ctx();
// part_o [batch][n_heads][nsplit][head_dim] and part_ml [batch][n_heads][nsplit][2] fp32 are
// used only when plan.nsplit > 1.
hipError_t launch_attn_decode(int dtype, int head_dim, const void *q, int ldq,
                              const void *kcache, const void *vcache, const int *lens,
                              int len_add, void *o, int ldo, int batch, int n_heads,
                              int n_kv_heads, int max_ctx, const AttnDecodePlan &plan,
                              float *part_o, float *part_ml, hipStream_t s,
                              bool skip_merge = false, const KvPaging &pg = KvPaging{});

// ------------------------------------------------------------------------------------------
// Selective state-space (Mamba) mixer
// ------------------------------------------------------------------------------------------
// Per layer: x (rows of the fp32 in_proj output, columns [0, di)) goes through the causal
// depthwise convolution + SiLU (-> u), x_proj gives (dt_low | B | C) per row, and the scan
// runs h <- exp(dt A) h + dt u B, y = C.h + D u, y * silu(z) per channel with the state in
// registers.  Prefill splits each sequence's tokens into chunks scanned in parallel: pass 1
// scans every chunk but the last from a zero state and keeps its end state and sum of dt,
// pass 2 chains those per sequence into each chunk's incoming state, pass 3 rescans every
// chunk from its incoming state and writes y.  Decode is pass 3 alone on one-token chunks.
constexpr int kScanChannels = 64;   // channels per scan block (one wave)
constexpr int kScanMinChunk = 16;   // shortest prefill chunk
constexpr int kScanTargetWaves = 2048;
constexpr int kChunkLast = 1;       // chunk flag: last chunk of its sequence in this call

// Prefill metadata: cu[B+1] packed row offsets, row_seq[T], last_row[B], the chunk list
// (seq, first row, rows, flags) in sequence order and seq_chunk0[B+1] (first chunk of each
// sequence).
struct MambaMeta {
  int batch;
  int lens[256];
};
hipError_t launch_mamba_meta(const MambaMeta &mm, int total, int chunk_len, int *cu,
                             int *row_seq, int *last_row, int4 *chunks, int *seq_chunk0,
                             hipStream_t s);
// Chunk length of a prefill of `total` rows over `di` channels, and the largest chunk count
// any prefill of at most `max_total` rows over `max_batch` sequences produces.
int mamba_chunk_len(int total, int di);
int mamba_max_chunks(int max_total, int max_batch, int di);

// u[r, c] = act(b[c] + sum_k w[c][k] * xs[i - (K-1) + k]) where xs is row r's sequence: the
// K-1 conv-state rows (zeros when `fresh`), then this call's x rows (fp32 xz[., c]); i is
// r's index among its sequence's rows (row_seq / cu null: row r is sequence r, index 0);
// act = 1: SiLU, 0: none.
// conv_state [batch][K-1][di] fp32 (read only here), w [di][K], b [di].
hipError_t launch_mamba_conv(int dtype, const float *xz, int ldxz, const int *row_seq,
                             const int *cu, const float *conv_state, int fresh,
                             const float *w, const float *b, int rows, int di, int K, void *u,
                             hipStream_t s, int act = 1);

struct ScanArgs {
  const float *xdbl = nullptr;  // [rows][ldx]: dt_low (R) | B (N) | C (N), fp32
  int ldx = 0;
  const void *u = nullptr;      // T [rows][di] (conv output)
  const float *xz = nullptr;    // fp32 [rows][ldxz]: x at columns [0, di), z at [di, 2 di)
  int ldxz = 0;
  const float *dtwT = nullptr;  // [R16][di] dt projection, transposed, rows >= R zero
                                //   (R16 = R rounded up to a multiple of 16)
  const float *dt_b = nullptr;  // [di]
  const float *A2 = nullptr;    // [N][di]  A * log2(e)
  const float *D = nullptr;     // [di]
  float *ssm = nullptr;         // [batch][di][N] SSM state of this layer
  float *conv = nullptr;        // [batch][K-1][di] conv state of this layer
  void *y = nullptr;            // T [rows][di] gated output
  float *hloc = nullptr;        // [chunks][N][di] chunk end / incoming states
  float *dtsum = nullptr;       // [chunks][di] sum of dt over each chunk
  const int4 *chunks = nullptr; // null: decode, chunk j = row j = sequence j, one row
  const int *seq_chunk0 = nullptr;
  const int *cu = nullptr;      // packed row offsets (null in decode)
  int di = 0, R = 0, N = 0, K = 0;
  int fresh = 0;                // sequences start from zero conv and SSM state
  int carry = 0;                // pass 3 incoming state: 0 zero, 1 SSM state, 2 hloc
};
// pass 1 over n_chunks chunks, pass 2 over `batch` sequences, pass 3 over n_chunks chunks
hipError_t launch_scan_chunks(int dtype, const ScanArgs &a, int n_chunks, hipStream_t s);
hipError_t launch_scan_carry(const ScanArgs &a, int batch, hipStream_t s);
hipError_t launch_scan_out(int dtype, const ScanArgs &a, int n_chunks, hipStream_t s);
// One fused decode step of the mixer for rows <= kSsmDecodeMaxRows sequences (row = sequence)
// and X = R + 2 N <= kSsmDecodeMaxX: x_proj of the conv output u (wx = the repacked x_proj,
// rows zero-padded to a multiple of 128) for every row, then per
// channel the dt projection, softplus, the state update h <- exp(dt A) h + dt u B (ssm state
// [rows][di][N] read and written), y = C.h + D u, y * silu(z), and optionally out_proj with
// the residual add.  One block per 32 channels; each block forms the whole x_proj product of
// its rows (from L2) so that no second launch is needed.
constexpr int kSsmDecodeMaxRows = 4;
constexpr int kSsmDecodeMaxX = 128;
struct SsmDecodeArgs {
  const void *u = nullptr;     // T [rows][di]
  const float *z = nullptr;    // fp32 [rows][ldz]
  int ldz = 0;
  const void *wx = nullptr;    // repacked x_proj (ll_op_repack layout), >= 128 rows
  const float *dtwT = nullptr, *dt_b = nullptr, *A2 = nullptr, *D = nullptr;
  float *ssm = nullptr;        // [rows][di][N]
  void *y = nullptr;           // T [rows][di] gated output (when wout is null)
  int rows = 0, di = 0, R = 0, N = 0;
  // With wout (the repacked out_proj [d][di]): x[r][0, d) += out_proj(y) instead of writing y,
  // each block adding its 32-channel share with fp32 atomics (summation order not fixed).
  const void *wout = nullptr;
  float *x = nullptr;
  int ldx = 0, d = 0;
};
hipError_t launch_ssm_decode(int dtype, const SsmDecodeArgs &a, hipStream_t s);

// dst[j][i] = src[i][j] * scale (after exp when `neg_exp`: dst = -exp(src) * scale) for
// j < cols, zero rows for cols <= j < cols_pad; fp32.
hipError_t launch_transpose_f32(const float *src, int rows, int cols, int cols_pad, float *dst,
                                int neg_exp, float scale, hipStream_t s);

// ------------------------------------------------------------------------------------------
// Mamba2 mixer
// ------------------------------------------------------------------------------------------
// Per layer the in_proj output rows hold z | x B C | dt (fp32, row stride ldz); the causal
// conv + SiLU over the x B C channels gives xbc.  Each head h (group h / (H / G) of B and C)
// keeps a state [P][N]: h <- exp(dt A_h) h + dt x B^T, y = h C + D_h x, and the scan writes
// g = y * silu(z) (fp32) for the gated RMSNorm that precedes out_proj.  One block of 256
// threads covers 16 rows of a head (16 lanes per row, N / 16 states per lane).  Prefill uses
// the three passes of the Mamba scan over time chunks; decode is pass 3 on one-token chunks.
constexpr int kM2Rows = 16;              // head rows per scan block
constexpr int kM2TargetBlocks = 1024;
int mamba2_chunk_len(int total, int n_heads, int head_dim);
// The matrix-form prefill scan: chunk length, and the shapes it is instantiated for.
constexpr int kM2SsdChunk = 64;
bool mamba2_ssd_ok(int head_dim, int d_state);
int mamba2_max_chunks(int max_total, int max_batch, int n_heads, int head_dim);
struct M2ScanArgs {
  const float *zxd = nullptr;   // in_proj rows: z at [0, di), dt at [dt_col, dt_col + H)
  int ldz = 0, dt_col = 0;
  const float *xbc = nullptr;   // conv output rows [rows][conv_n]: x | B (G N) | C (G N)
  const float *dt_b = nullptr, *A2 = nullptr, *D = nullptr;  // [H]; A2 = A * log2(e)
  float *ssm = nullptr;         // [batch][H][P][N]
  float *g = nullptr;           // fp32 [rows][di]
  float *hloc = nullptr;        // [chunks][H][P][N]
  float *dtsum = nullptr;       // [chunks][H]
  const int4 *chunks = nullptr; // null: decode (chunk j = row j = sequence j)
  const int *seq_chunk0 = nullptr, *cu = nullptr;
  float *conv = nullptr;        // conv state [batch][K-1][conv_n] (updated when update_conv)
  int conv_col = 0, conv_n = 0, K = 0, update_conv = 0;
  int di = 0, H = 0, P = 0, N = 0, G = 0;
  int fresh = 0, carry = 0;     // carry: 0 zero, 1 SSM state, 2 hloc
  int mfma = 0;                 // prefill chunks through the matrix-form scan (k_m2_ssd):
                                // chunks of at most kM2SsdChunk steps, fp16 operands
};
hipError_t launch_m2_scan_chunks(const M2ScanArgs &a, int n_chunks, hipStream_t s);
hipError_t launch_m2_scan_carry(const M2ScanArgs &a, int batch, hipStream_t s);
hipError_t launch_m2_scan_out(const M2ScanArgs &a, int n_chunks, hipStream_t s);

// ------------------------------------------------------------------------------------------
// RG-LRU recurrent block (Griffin).  The gate GEMM's epilogue (kEpiRglru) writes a (decay, 0 at
// a reset) and g (normalised, gated input) per (row, channel); the prefill scan runs
// h_t = a_t h_{t-1} + g_t per channel over time chunks and writes out = T(h * gy).
// Pass 1 (launch_rg_scan_chunks): (prod a, h_end from zero) of every chunk but each sequence's
// last.  Pass 3 (launch_rg_scan_out): incoming state chained from the sequence's state (zero
// when fresh) through its earlier chunks, rescan, output, and at a sequence's last chunk the
// recurrent state and the last K-1 conv inputs (from raw, after the old conv state).
// Chunks come from launch_mamba_meta with chunk length rg_chunk_len(longest sequence), so a
// sequence has at most kRgMaxChunksPerSeq chunks.
constexpr int kRgMaxChunksPerSeq = 64;
int rg_chunk_len(int max_len);
struct RgScanArgs {
  const float *a = nullptr, *g = nullptr;  // [rows][W]
  const void *gy = nullptr;                // T [rows][W]
  void *out = nullptr;                     // T [rows][W]
  float *state = nullptr;                  // [batch][W]
  float *hend = nullptr, *aprod = nullptr; // [chunks][W]
  const int4 *chunks = nullptr;
  const int *seq_chunk0 = nullptr, *cu = nullptr;
  float *conv = nullptr;                   // [batch][K-1][W]
  const float *raw = nullptr;              // conv inputs of this call [rows][ld_raw]
  int ld_raw = 0, W = 0, K = 0, fresh = 0;
};
// gain_t / gain_c = 1 + norm_t / norm_c (type T, [d]); lam_out = -c softplus(lam) ([W]) when
// lam is given.
hipError_t launch_rg_prep(int dtype, const void *norm_t, const void *norm_c, int d,
                          const float *lam, int W, float c, void *gain_t, void *gain_c,
                          float *lam_out, hipStream_t s);
// x[i] = cap * tanh(x[i] / cap) over n floats (soft-capped logits).
hipError_t launch_softcap(float *x, long n, float cap, hipStream_t s);
hipError_t launch_rg_scan_chunks(const RgScanArgs &a, int n_chunks, hipStream_t s);
hipError_t launch_rg_scan_out(int dtype, const RgScanArgs &a, int n_chunks, hipStream_t s);

}  // namespace ll
