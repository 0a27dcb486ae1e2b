// Phase-specialised causal grouped-query attention (appendix "Deployment Kernel Families",
// Table A.4: a prefill kernel over query tiles with the causal mask inside the score update
// and fp32 online-softmax statistics, and a decode kernel that loads each KV tile once for
// the whole query-head group).
//
// Prefill: scores are computed transposed, S^T = K Q^T, so that each lane owns one query
// column: the softmax statistics and the O^T = V^T P^T accumulator are then lane-local, and
// P feeds the second MFMA as its B operand without leaving registers.  bf16 uses 32x32x16
// MFMAs over 128-query tiles (k_attn_prefill_wide); fp32 uses 16x16 MFMAs over 64-query
// tiles (k_attn_prefill).  K and V^T tiles are staged in LDS in MFMA operand order.
//
// Decode: grid (split, kv head, sequence); a block streams `chunk` cached keys once for all
// query heads of the group, keeps exact chunk scores in LDS and writes (max, sum, partial
// output) per head; a second kernel merges the splits with
// log-sum-exp weights (fixed order, so the result does not depend on block order).
#include <algorithm>
#include <cmath>
#include <type_traits>

#include "device_common.h"
#include "kernels.h"

namespace ll {
namespace {

template <typename T, int HD>
__global__ __launch_bounds__(256) void k_attn_prefill(
    const T *__restrict__ Q, int ldq, const T *__restrict__ Kc, const T *__restrict__ Vc,
    T *__restrict__ O, int ldo, const int *__restrict__ cu, const int *__restrict__ kstart,
    const int2 *__restrict__ qtiles, int hq, int hkv, int max_ctx, float scale_log2,
    KvPaging pg) {
  using F = typename Frag<T>::type;
  constexpr int EPL = Frag<T>::EPL;
  constexpr int KT = 4 * EPL;       // head dims per Q K^T chunk
  constexpr int NQC = HD / KT;
  constexpr int BKV = 64, NKS = BKV / 16;
  constexpr int PVK = 4 * EPL;      // keys per P V chunk
  constexpr int NPV = BKV / PVK;
  constexpr int NDS = HD / 16;
  constexpr int CPR = HD / EPL;     // 16-byte chunks per cached row
  __shared__ F sK[NKS * NQC * 64];
  __shared__ __attribute__((aligned(16))) T sV[NDS * NPV * 64 * EPL];

  // grid (head, query tile): blocks are dealt round-robin to the 8 XCDs in dispatch order, so
  // head-fastest order gives every XCD the same mix of short and long causal tiles; the tile
  // list is ordered longest first and its second half is walked backwards, so that the blocks
  // dispatched second to a CU's slots are the short ones
  const int ny = gridDim.y, yh = (ny + 1) / 2;
  const int yi = blockIdx.y < yh ? blockIdx.y : ny - 1 - (blockIdx.y - yh);
  const int2 qt = qtiles[yi];
  const int b = qt.x, h = blockIdx.x, kvh = h / (hq / hkv);
  const int tok0 = cu[b], L = cu[b + 1] - tok0;
  // queries sit at positions P0 + i after P0 cached keys; KL keys in all
  const int P0 = kstart ? kstart[b] : 0, KL = P0 + L;
  const int q0 = qt.y * kAttnQTile;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int my_q = q0 + wave * 16 + (lane & 15);
  const F fz = frag_zero<F>();

  F qf[NQC];
#pragma unroll
  for (int c = 0; c < NQC; ++c)
    qf[c] = my_q < L ? load_frag<F>(Q + (size_t)(tok0 + my_q) * ldq + h * HD + c * KT +
                                    (lane >> 4) * EPL)
                     : fz;
  f32x4 acc[NDS];
#pragma unroll
  for (int ds = 0; ds < NDS; ++ds) acc[ds] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;

  const int q_last = min(q0 + kAttnQTile - 1, L - 1);
  const int ntiles = (P0 + q_last) / BKV + 1;
  for (int kt = 0; kt < ntiles; ++kt) {
    __syncthreads();
    // the tile's 64 keys lie in one page (its first key is a cached position)
    const size_t tb = kv_row_off(pg, b, kvh, hkv, max_ctx, kt * BKV, HD);
    for (int c = tid; c < BKV * CPR; c += 256) {
      const int key = c / CPR, dc = c % CPR;
      const int gk = kt * BKV + key;
      F kv = fz, vv = fz;
      if (gk < KL) {
        kv = load_frag<F>(Kc + tb + (size_t)key * HD + dc * EPL);
        vv = load_frag<F>(Vc + tb + (size_t)key * HD + dc * EPL);
      }
      sK[((key >> 4) * NQC + dc / 4) * 64 + (key & 15) + 16 * (dc & 3)] = kv;
      const int kc = key / PVK, kk = key % PVK;
      const int g = (kk & 15) >> 2, ee = (kk >> 4) * 4 + (kk & 3);
#pragma unroll
      for (int e = 0; e < EPL; ++e) {
        const int d = dc * EPL + e;
        sV[(((d >> 4) * NPV + kc) * 64 + (d & 15) + 16 * g) * EPL + ee] = vv[e];
      }
    }
    __syncthreads();

    f32x4 s[NKS];
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      s[ks] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int c = 0; c < NQC; ++c) s[ks] = mma_chunk(sK[(ks * NQC + c) * 64 + lane], qf[c], s[ks]);
    }
    float tmax = -INFINITY;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int key = kt * BKV + ks * 16 + (lane >> 4) * 4 + r;
        const float v = (key <= P0 + my_q && my_q < L) ? s[ks][r] * scale_log2 : -INFINITY;
        s[ks][r] = v;
        tmax = fmaxf(tmax, v);
      }
    tmax = fmaxf(tmax, __shfl_xor(tmax, 16));
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32));
    const float m_new = fmaxf(m_run, tmax);
    const float base = m_new == -INFINITY ? 0.f : m_new;
    const float alpha = exp2f(m_run - base);
    m_run = m_new;
    l_run *= alpha;
#pragma unroll
    for (int ds = 0; ds < NDS; ++ds) acc[ds] *= alpha;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float p = exp2f(s[ks][r] - base);
        s[ks][r] = p;
        l_run += p;
      }
#pragma unroll
    for (int kc = 0; kc < NPV; ++kc) {
      F pb;
#pragma unroll
      for (int e = 0; e < EPL; ++e) pb[e] = from_f32<T>(s[kc * (PVK / 16) + e / 4][e & 3]);
#pragma unroll
      for (int ds = 0; ds < NDS; ++ds)
        acc[ds] = mma_chunk(*reinterpret_cast<const F *>(&sV[((ds * NPV + kc) * 64 + lane) * EPL]),
                            pb, acc[ds]);
    }
  }
  l_run += __shfl_xor(l_run, 16);
  l_run += __shfl_xor(l_run, 32);
  if (my_q < L) {
    const float inv = 1.0f / l_run;
    T *dst = O + (size_t)(tok0 + my_q) * ldo + h * HD + (lane >> 4) * 4;
#pragma unroll
    for (int ds = 0; ds < NDS; ++ds)
#pragma unroll
      for (int r = 0; r < 4; ++r) dst[ds * 16 + r] = from_f32<T>(acc[ds][r] * inv);
  }
}

// V tile of a stage: the tile's 64 keys as natural [key][dim] rows, DMA'd straight from the
// cache like K, with the 16-byte chunks of each row XOR-swizzled: chunk c of row k sits at
// slot c ^ vswz(k).  The transposed fragment reads of the P V product (below) then hit 64
// distinct banks per 32 lanes.
template <int HD> __device__ __forceinline__ constexpr int vswz(int row) {
  return 4 * ((row / (128 / HD)) % (HD / 32));
}

// Per-lane source of DMA instruction q of a stage's V tile (HD / 8 of them per 64 keys): lane l
// fills slot (64 q + l) % (HD / 8) of row (64 q + l) / (HD / 8), i.e. 8 elements of that key
// row from column 8 (slot ^ vswz(row)).
template <int HD> __device__ __forceinline__ int2 v_src(int q, int lane) {
  constexpr int SPR = HD / 8;
  const int idx = 64 * q + lane, row = idx / SPR, slot = idx % SPR;
  return make_int2(row, 8 * (slot ^ vswz<HD>(row)));
}

// One 1 KiB DMA of a K or V tile: rows past the sequence (row > lim, the tile's last valid
// row) read row lim instead; their probabilities are 0.  `base` is the tile's first key row.
template <typename H, int HD>
__device__ __forceinline__ void kv_dma(const H *base, int2 rc, int lim, uint4 *dst) {
  load_tile_to_lds(base + (unsigned)(min(rc.x, lim) * HD + rc.y), dst);
}

// Byte offsets, within a V tile, of lane l's transposed reads for 32-dim block d (key step 0,
// first half).  ds_read_b64_tr_b16 (measured on gfx950): in each group of 16 lanes, lane
// 4 r + c supplies the address of 4 consecutive 16-bit elements, and lane j receives element
// j % 4 of the elements of lanes 4 r + j / 4, r = 0..3.  Lane 4 r + c of group G therefore
// points at key row 4 (G / 2) + r, dims 32 d + 16 (G % 2) + 4 c: lane j of the group gets
// dim 32 d + 16 (G % 2) + j of four consecutive keys, which is the A operand of V^T P^T with
// the keys in the order the score registers hold them (4 (l / 32) + e, then 8 + 4 (l / 32) + e).
template <int HD>
__device__ __forceinline__ void v_tr_offsets(int lane, int *voff) {
  const int G = lane >> 4, j = lane & 15, r = j >> 2, c = j & 3;
  const int row = 4 * (G >> 1) + r, x = vswz<HD>(row) / 4;
#pragma unroll
  for (int d = 0; d < HD / 32; ++d)
    voff[d] = row * HD * 2 + (4 * (d ^ x) + 2 * (G & 1) + (c >> 1)) * 16 + 8 * (c & 1);
}

typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));
template <typename V, int HD>
__device__ __forceinline__ V v_frag_tr(const char *vtile, int off) {
  typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
  const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(vtile + off));
  const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(vtile + off + 8 * HD * 2));
  return __builtin_bit_cast(V, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
}

// Value of lane l ^ 32 combined with lane l's own (v_permlane32_swap exchanges the two
// halves of the wave; the pair it returns holds both values in some order).
__device__ __forceinline__ float xhalf_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float xhalf_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
// acc + the 8 probabilities of a packed P^T operand, as rounded to the operand type (the
// weights the P V product applies), two at a time with fp32 accumulation (v_dot2).
typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ float sum_frag(const f16x8 &p, float acc) {
  const f16x2_t one = {(_Float16)1.f, (_Float16)1.f};
  acc = __builtin_amdgcn_fdot2(__builtin_shufflevector(p, p, 0, 1), one, acc, false);
  acc = __builtin_amdgcn_fdot2(__builtin_shufflevector(p, p, 2, 3), one, acc, false);
  acc = __builtin_amdgcn_fdot2(__builtin_shufflevector(p, p, 4, 5), one, acc, false);
  return __builtin_amdgcn_fdot2(__builtin_shufflevector(p, p, 6, 7), one, acc, false);
}
__device__ __forceinline__ float sum_frag(const bf16x8 &p, float acc) {
  const bf16x2_t one = {(__bf16)1.f, (__bf16)1.f};
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(p, p, 0, 1), one, acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(p, p, 2, 3), one, acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(p, p, 4, 5), one, acc, false);
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(p, p, 6, 7), one, acc, false);
}

// One 64-key tile of 16-bit prefill attention for one wave of 32 queries (lane l owns query
// qw + l % 32), on v_mfma_f32_32x32x16, from an LDS stage `st` that holds the tile's K in
// operand order ([32-key block][16-dim step] tiles of 64 x 16 B) followed by its V tile
// (natural rows, swizzled; voff from v_tr_offsets).
//   S^T = K Q^T: A = K rows from LDS, B = the wave's Q^T fragments (registers).  Lane l holds,
//     of each 32-key block, rows 8 (i / 4) + 4 (l / 32) + i % 4: the online-softmax
//     statistics need one exchange with lane l ^ 32.
//   O^T += V^T P^T: A = V^T by transposed LDS reads, B = P^T straight from the score registers.
// S^T of one 64-key tile.  K fragments are requested two 16-dim steps ahead of their MFMAs
// (LDS latency off the MFMA chain at modest register cost), and the two 32-key chains
// alternate so that MFMA result latency is not exposed either.
template <typename H, int HD>
__device__ __forceinline__ void attn_s16(const uint4 *__restrict__ st,
                                         const typename Frag<H>::type *qf, int lane, f32x16 *sc) {
  using V = typename Frag<H>::type;
  constexpr int NKC = HD / 16, AHEAD = 2;
  V kf[NKC][2];
  auto kload = [&](int c) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) kf[c][kb] = *reinterpret_cast<const V *>(&st[(kb * NKC + c) * 64 + lane]);
  };
#pragma unroll
  for (int c = 0; c < AHEAD; ++c) kload(c);
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int i = 0; i < 16; ++i) sc[kb][i] = 0.f;
#pragma unroll
  for (int c = 0; c < NKC; ++c) {
    if (c + AHEAD < NKC) kload(c + AHEAD);
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) sc[kb] = mma32(kf[c][kb], qf[c], sc[kb]);
  }
}

// Online softmax of a tile's scores: causal / length mask (only on tiles that reach past the
// wave's first query), running maximum and sum, rescale of the accumulator, and the
// probabilities packed as the P^T operands of the four 16-key steps.
// The reference maximum moves lazily: only when some row's score maximum exceeds it by more
// than kSoftmaxSlack (log2 units) are the accumulator and sum rescaled (for every row, to the
// true running maximum).  Until then the probabilities are taken against the smaller, stale
// reference and lie in (0, 2^kSoftmaxSlack]; the common factor cancels exactly in the final
// division by the sum, and fp16 / bf16 hold such values with the same relative precision as
// values below 1.  On most tiles the 64 accumulator multiplies per lane are skipped.
constexpr float kSoftmaxSlack = 8.f;
template <typename H, int HD>
__device__ __forceinline__ void attn_softmax16(f32x16 *sc, f32x16 *acc, float &m_run,
                                               float &l_run, int kt, int P0, int L, int qw,
                                               int my_q, bool q_ok, float scale_log2, int lane,
                                               typename Frag<H>::type *pf) {
  constexpr int BKV = 64, NDB = HD / 32, NPC = BKV / 16;
  const int g = lane >> 5;
  if (kt * BKV + BKV - 1 > P0 + qw || qw + 31 >= L) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int key = kt * BKV + 32 * kb + 8 * (i / 4) + 4 * g + (i % 4);
        sc[kb][i] = (q_ok & (key <= P0 + my_q)) ? sc[kb][i] : -INFINITY;
      }
  }
  // row maximum of the raw scores; scaling by a positive constant commutes with max
  float tmax = -INFINITY;
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int i = 0; i < 16; ++i) tmax = fmaxf(tmax, sc[kb][i]);
  tmax = xhalf_max(tmax);
  const float m_cand = tmax * scale_log2;
  if (__any(m_cand > m_run + kSoftmaxSlack)) {
    const float m_new = fmaxf(m_run, m_cand);
    const float alpha = __builtin_amdgcn_exp2f(m_run - (m_new == -INFINITY ? 0.f : m_new));
    l_run *= alpha;
#pragma unroll
    for (int d = 0; d < NDB; ++d) acc[d] *= alpha;
    m_run = m_new;
  }
  const float base = m_run == -INFINITY ? 0.f : m_run;
  // p = 2^(s * scale - m); arguments are <= kSoftmaxSlack, so the hardware exp2 is exact
  // enough (results below the fp32 normal range flush to 0)
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int i = 0; i < 16; ++i) sc[kb][i] = __builtin_amdgcn_exp2f(fmaf(sc[kb][i], scale_log2, -base));
#pragma unroll
  for (int c = 0; c < NPC; ++c) {
#pragma unroll
    for (int e = 0; e < 8; ++e) pf[c][e] = static_cast<H>(sc[c / 2][8 * (c % 2) + e]);
    l_run = sum_frag(pf[c], l_run);
  }
}

// V^T fragments of a stage's V tile.
template <typename H, int HD>
__device__ __forceinline__ void attn_vload16(const uint4 *__restrict__ st, const int *voff,
                                             typename Frag<H>::type (*vf)[HD / 32]) {
  constexpr int NPC = 4, KTILES = 2 * (HD / 16);
  const char *vt = reinterpret_cast<const char *>(st + KTILES * 64);
#pragma unroll
  for (int c = 0; c < NPC; ++c)
#pragma unroll
    for (int d = 0; d < HD / 32; ++d)
      vf[c][d] = v_frag_tr<typename Frag<H>::type, HD>(vt, voff[d] + 16 * c * HD * 2);
}

template <typename H, int HD>
__device__ __forceinline__ void attn_pv16(typename Frag<H>::type (*vf)[HD / 32],
                                          const typename Frag<H>::type *pf, f32x16 *acc) {
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int d = 0; d < HD / 32; ++d) acc[d] = mma32(vf[c][d], pf[c], acc[d]);
}

// One whole tile: scores, then the V^T fragments are requested (the softmax covers their
// latency), softmax, P V.
template <typename H, int HD>
__device__ __forceinline__ void attn_tile16(const uint4 *__restrict__ st,
                                            const typename Frag<H>::type *qf, f32x16 *acc,
                                            float &m_run, float &l_run, int kt, int P0, int L,
                                            int qw, int my_q, bool q_ok, float scale_log2,
                                            int lane, const int *voff) {
  using V = typename Frag<H>::type;
  f32x16 sc[2];
  attn_s16<H, HD>(st, qf, lane, sc);
  V vf[4][HD / 32];
  attn_vload16<H, HD>(st, voff, vf);
  __builtin_amdgcn_sched_barrier(0);
  V pf[4];
  attn_softmax16<H, HD>(sc, acc, m_run, l_run, kt, P0, L, qw, my_q, q_ok, scale_log2, lane, pf);
  attn_pv16<H, HD>(vf, pf, acc);
}

// Normalised output rows of one wave: lane l writes dims 32 d + 8 j + 4 (l / 32) .. + 3 of its
// query (the O^T accumulator layout), 8 bytes at a time.
template <typename H, int HD>
__device__ __forceinline__ void attn_store16(H *dst, const f32x16 *acc, float inv, int g) {
  constexpr int NDB = HD / 32;
  dst += 4 * g;
#pragma unroll
  for (int d = 0; d < NDB; ++d)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const H v0 = static_cast<H>(acc[d][4 * j] * inv), v1 = static_cast<H>(acc[d][4 * j + 1] * inv);
      const H v2 = static_cast<H>(acc[d][4 * j + 2] * inv), v3 = static_cast<H>(acc[d][4 * j + 3] * inv);
      uint2 pk;
      pk.x = (uint32_t)__builtin_bit_cast(uint16_t, v0) | ((uint32_t)__builtin_bit_cast(uint16_t, v1) << 16);
      pk.y = (uint32_t)__builtin_bit_cast(uint16_t, v2) | ((uint32_t)__builtin_bit_cast(uint16_t, v3) << 16);
      *reinterpret_cast<uint2 *>(dst + 32 * d + 8 * j) = pk;
    }
}

// 16-bit prefill attention, one query head per block (the MHA workloads): one block per
// (128-query tile, query head), 4 waves of 32 queries, key tiles of 64 through a
// double-buffered LDS stage.  K (operand order) and V (natural rows, swizzled) are DMA'd from
// the cache straight into LDS (global_load_lds), the work split evenly over the 4 waves; the
// loads for tile t + 1 are in flight while tile t computes (attn_tile16).
template <typename H, int HD>
__global__ __launch_bounds__(256, 2) void k_attn_prefill_wide(
    const H *__restrict__ Q, int ldq, const H *__restrict__ Kc, const H *__restrict__ Vc,
    H *__restrict__ O, int ldo, const int *__restrict__ cu, const int *__restrict__ kstart,
    const int2 *__restrict__ qtiles, int hq, int hkv, int max_ctx, float scale_log2,
    KvPaging pg) {
  constexpr int QT = kAttnQTileWide, BKV = 64;
  constexpr int NKC = HD / 16;                 // 16-dim steps of S^T
  constexpr int NDB = HD / 32;                 // 32-dim output blocks
  constexpr int KTILES = 2 * NKC;              // K tiles per stage: [32-key block][16-dim step]
  constexpr int VINS = BKV * HD * 2 / 1024;    // 1 KiB DMA instructions of a V tile
  constexpr int STAGE = (KTILES + VINS) * 64;  // uint4 per stage
  static_assert(QT == 128 && KTILES % 4 == 0 && VINS % 4 == 0, "4 waves of 32 queries");
  __shared__ uint4 smem[2 * STAGE];

  // grid (head, query tile): blocks are dealt round-robin to the 8 XCDs in dispatch order, so
  // head-fastest order gives every XCD the same mix of short and long causal tiles; the tile
  // list is ordered longest first and its second half is walked backwards, so that the blocks
  // dispatched second to a CU's slots are the short ones
  const int ny = gridDim.y, yh = (ny + 1) / 2;
  const int yi = blockIdx.y < yh ? blockIdx.y : ny - 1 - (blockIdx.y - yh);
  const int2 qt = qtiles[yi];
  const int b = qt.x, h = blockIdx.x, kvh = h / (hq / hkv);
  const int tok0 = cu[b], L = cu[b + 1] - tok0;
  // queries sit at positions P0 + i after P0 cached keys; KL keys in all
  const int P0 = kstart ? kstart[b] : 0, KL = P0 + L;
  const int q0 = qt.y * QT;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 5;
  const int qw = q0 + wave * 32;  // first query of this wave
  const int my_q = qw + (lane & 31);
  const bool q_ok = my_q < L;
  using V = typename Frag<H>::type;
  const V fz = frag_zero<V>();

  V qf[NKC];
#pragma unroll
  for (int c = 0; c < NKC; ++c)
    qf[c] = q_ok ? load_frag<V>(Q + (size_t)(tok0 + my_q) * ldq + h * HD + 16 * c + 8 * g) : fz;
  f32x16 acc[NDB];
#pragma unroll
  for (int d = 0; d < NDB; ++d)
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[d][i] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;
  int voff[NDB];
  v_tr_offsets<HD>(lane, voff);

  const int ntiles = (P0 + min(q0 + QT, L) - 1) / BKV + 1;

  // K tile (kb, c): lane l reads key 32 kb + l % 32 (clamped into the sequence; rows past KL
  // are masked), dims 16 c + 8 g.  A tile's keys lie in one page (tiles start at cached
  // positions and the clamp stays in the tile), so one base per tile serves every row.
  int2 ksrc[KTILES / 4], vsrc[VINS / 4];   // (row in the tile, column) of each DMA of the wave
#pragma unroll
  for (int i = 0; i < KTILES / 4; ++i) {
    const int ti = wave + 4 * i;
    ksrc[i] = make_int2(32 * (ti / NKC) + (lane & 31), 16 * (ti % NKC) + 8 * g);
  }
#pragma unroll
  for (int i = 0; i < VINS / 4; ++i) vsrc[i] = v_src<HD>(wave + 4 * i, lane);
  auto issue = [&](int kt, int buf) {
    const size_t tb = kv_row_off(pg, b, kvh, hkv, max_ctx, kt * BKV, HD);
    const int lim = KL - 1 - kt * BKV;
#pragma unroll
    for (int i = 0; i < KTILES / 4; ++i)
      kv_dma<H, HD>(Kc + tb, ksrc[i], lim, &smem[buf * STAGE + (wave + 4 * i) * 64]);
#pragma unroll
    for (int i = 0; i < VINS / 4; ++i)
      kv_dma<H, HD>(Vc + tb, vsrc[i], lim, &smem[buf * STAGE + (KTILES + wave + 4 * i) * 64]);
  };

  issue(0, 0);
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  // tile kt from stage CUR (= kt % 2; the loop is unrolled by two so that stage offsets are
  // compile-time constants)
  auto tile = [&](int kt, auto CUR) {
    constexpr int cur = decltype(CUR)::value;
    if (kt + 1 < ntiles) issue(kt + 1, cur ^ 1);
    if (qw < L && kt * BKV <= P0 + qw + 31)  // else nothing for this wave in this tile
      attn_tile16<H, HD>(&smem[cur * STAGE], qf, acc, m_run, l_run, kt, P0, L, qw, my_q, q_ok,
                         scale_log2, lane, voff);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
  };
  for (int kt = 0; kt < ntiles; kt += 2) {
    tile(kt, std::integral_constant<int, 0>());
    if (kt + 1 < ntiles) tile(kt + 1, std::integral_constant<int, 1>());
  }

  l_run = xhalf_sum(l_run);
  if (q_ok) attn_store16<H, HD>(O + (size_t)(tok0 + my_q) * ldo + h * HD, acc, 1.0f / l_run, g);
}

// 16-bit prefill attention for grouped heads (group G = H_q / H_kv >= 2), after the paper's
// prefill kernel that shares KV loads according to the head grouping (appendix "Deployment
// Kernel Families", Table A.4): one block of 8 waves per (query tile, KV head) holds every
// query head of the group -- wave w takes head kvh G + w / QB and 32 queries of block w % QB
// (QB = 8 / G; tiles of 32 QB queries) -- so each 64-key K / V tile is read from memory and
// staged in LDS once for G heads.  The 8 waves share the K and V DMA evenly.  Blocks take
// their (sequence, query tile, KV head) from the work list in XCD-owned ranges (AttnSched).
template <typename H, int HD, int G>
__global__ __launch_bounds__(512, 1) void k_attn_prefill_gqa(
    const H *__restrict__ Q, int ldq, const H *__restrict__ Kc, const H *__restrict__ Vc,
    H *__restrict__ O, int ldo, const int *__restrict__ cu, const int *__restrict__ kstart,
    const int4 *__restrict__ sched, AttnSched as, int hkv, int max_ctx, float scale_log2,
    KvPaging pg) {
  constexpr int NW = 8, QB = NW / G, QT = 32 * QB, BKV = 64;
  constexpr int NKC = HD / 16, NDB = HD / 32, NPC = BKV / 16;
  constexpr int KTILES = 2 * NKC;
  constexpr int VINS = BKV * HD * 2 / 1024;        // 1 KiB DMA instructions of a V tile
  constexpr int STAGE = (KTILES + VINS) * 64;      // uint4 per stage
  static_assert(G >= 2 && G <= NW && NW % G == 0 && KTILES % NW == 0 && VINS % NW == 0,
                "8 waves over the group");
  __shared__ uint4 smem[2 * STAGE];

  const int x = blockIdx.x % kXcds, e = as.cut[x] + (int)(blockIdx.x / kXcds);
  if (e >= as.cut[x + 1]) return;   // this XCD's range is shorter than the longest one
  const int4 en = sched[e];
  const int b = en.x, kvh = en.z;
  const int tok0 = cu[b], L = cu[b + 1] - tok0;
  const int P0 = kstart ? kstart[b] : 0, KL = P0 + L;
  const int q0 = en.y * QT;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 5;
  const int h = kvh * G + wave / QB;
  const int qw = q0 + 32 * (wave % QB);
  const int my_q = qw + (lane & 31);
  const bool q_ok = my_q < L;
  using V = typename Frag<H>::type;
  const V fz = frag_zero<V>();

  V qf[NKC];
#pragma unroll
  for (int c = 0; c < NKC; ++c)
    qf[c] = q_ok ? load_frag<V>(Q + (size_t)(tok0 + my_q) * ldq + h * HD + 16 * c + 8 * g) : fz;
  f32x16 acc[NDB];
#pragma unroll
  for (int d = 0; d < NDB; ++d)
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[d][i] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;

  int voff[NDB];
  v_tr_offsets<HD>(lane, voff);

  const int ntiles = (P0 + min(q0 + QT, L) - 1) / BKV + 1;
  int2 ksrc[KTILES / NW], vsrc[VINS / NW];   // (row in the tile, column) of each DMA of the wave
#pragma unroll
  for (int i = 0; i < KTILES / NW; ++i) {
    const int ti = wave + NW * i;
    ksrc[i] = make_int2(32 * (ti / NKC) + (lane & 31), 16 * (ti % NKC) + 8 * g);
  }
#pragma unroll
  for (int i = 0; i < VINS / NW; ++i) vsrc[i] = v_src<HD>(wave + NW * i, lane);
  auto issue = [&](int kt, int buf) {
    const size_t tb = kv_row_off(pg, b, kvh, hkv, max_ctx, kt * BKV, HD);
    const int lim = KL - 1 - kt * BKV;
#pragma unroll
    for (int i = 0; i < KTILES / NW; ++i)
      kv_dma<H, HD>(Kc + tb, ksrc[i], lim, &smem[buf * STAGE + (wave + NW * i) * 64]);
#pragma unroll
    for (int i = 0; i < VINS / NW; ++i)
      kv_dma<H, HD>(Vc + tb, vsrc[i], lim, &smem[buf * STAGE + (KTILES + wave + NW * i) * 64]);
  };

  issue(0, 0);
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  // tile kt from stage CUR (= kt % 2; the loop is unrolled by two so that stage offsets are
  // compile-time constants)
  auto tile = [&](int kt, auto CUR) {
    constexpr int cur = decltype(CUR)::value;
    if (kt + 1 < ntiles) issue(kt + 1, cur ^ 1);
    if (qw < L && kt * BKV <= P0 + qw + 31)  // else nothing for this wave in this tile
      attn_tile16<H, HD>(&smem[cur * STAGE], qf, acc, m_run, l_run, kt, P0, L, qw, my_q, q_ok,
                         scale_log2, lane, voff);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
  };
  for (int kt = 0; kt < ntiles; kt += 2) {
    tile(kt, std::integral_constant<int, 0>());
    if (kt + 1 < ntiles) tile(kt + 1, std::integral_constant<int, 1>());
  }

  l_run = xhalf_sum(l_run);
  if (q_ok) attn_store16<H, HD>(O + (size_t)(tok0 + my_q) * ldo + h * HD, acc, 1.0f / l_run, g);
}

constexpr int kMaxSplit = 128;  // blocks per (sequence, kv head)

// Decode attention for one (split, kv head, sequence): the block covers up to KPT * NSLOT
// cached keys in one pass.  Every thread requests all of its K rows before using the first
// (then all of its V rows), so a block has its whole chunk in flight at once; each K and V row
// is read once for all G query heads of the group.  With a single split the block normalises
// and writes the attention output; otherwise it writes (max, sum, unnormalised output) for the
// merge kernel.  The merge is a separate kernel: a kernel boundary makes every block's
// partials visible across XCDs once per launch, where a device-scope fence in each block
// would write back the L2 once per block.
template <typename T, int HD, int G, int KPT>
__global__ __launch_bounds__(256) void k_attn_decode(
    const T *__restrict__ Q, int ldq, const T *__restrict__ Kc, const T *__restrict__ Vc,
    const int *__restrict__ lens, int len_add, int hkv, int max_ctx, int kpb, int nsplit,
    float *__restrict__ part_o, float *__restrict__ part_ml, T *__restrict__ O, int ldo,
    float scale_log2, KvPaging pg) {
  using F = typename Frag<T>::type;
  constexpr int EPL = Frag<T>::EPL;
  constexpr int LPK = HD / EPL;         // lanes per cached row
  constexpr int NSLOT = 256 / LPK;      // rows in flight per pass
  constexpr int CH = KPT * NSLOT;       // largest chunk
  const int split = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
  const int S = min(lens[b] + len_add, max_ctx);  // never read past the cache capacity
  const int j0 = split * kpb;
  if (j0 >= S) return;
  const int n = min(min(kpb, CH), S - j0);
  const int tid = threadIdx.x, dl = tid % LPK, slot = tid / LPK;
  const int lane = tid & 63, wave = tid >> 6;
  const int hq = hkv * G;
  __shared__ float s_p[G][CH];
  __shared__ float s_red[8][G][HD];  // [wave][32-lane half]
  __shared__ float s_m[G], s_l[G];
  const F fz = frag_zero<F>();

  float qv[G][EPL];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const F qq = load_frag<F>(Q + (size_t)b * ldq + (kvh * G + g) * HD + dl * EPL);
#pragma unroll
    for (int e = 0; e < EPL; ++e) qv[g][e] = to_f32(qq[e]) * scale_log2;
  }
  // the chunk (kpb <= 256 keys, aligned) lies in one page
  const size_t kvbase = kv_row_off(pg, b, kvh, hkv, max_ctx, j0, HD);
  const T *Kb = Kc + kvbase + dl * EPL;
  const T *Vb = Vc + kvbase + dl * EPL;

  F rows[KPT];
#pragma unroll
  for (int i = 0; i < KPT; ++i) {
    if (i * NSLOT >= n) break;
    const int jj = slot + i * NSLOT;
    rows[i] = jj < n ? load_frag_stream<F>(Kb + (size_t)jj * HD) : fz;
  }
#pragma unroll
  for (int i = 0; i < KPT; ++i) {
    if (i * NSLOT >= n) break;
    float d[G];
#pragma unroll
    for (int g = 0; g < G; ++g) {
      float a = 0.f;
#pragma unroll
      for (int e = 0; e < EPL; ++e) a += qv[g][e] * to_f32(rows[i][e]);
      d[g] = a;
    }
#pragma unroll
    for (int g = 0; g < G; ++g) d[g] = group_sum<LPK>(d[g]);
    const int jj = slot + i * NSLOT;
    if (dl == 0 && jj < n)
#pragma unroll
      for (int g = 0; g < G; ++g) s_p[g][jj] = d[g];
  }
  // V rows, requested while the chunk softmax runs
#pragma unroll
  for (int i = 0; i < KPT; ++i) {
    if (i * NSLOT >= n) break;
    const int jj = slot + i * NSLOT;
    rows[i] = jj < n ? load_frag_stream<F>(Vb + (size_t)jj * HD) : fz;
  }
  __syncthreads();
  for (int g = wave; g < G; g += 4) {
    float mx = -INFINITY;
    for (int i = lane; i < n; i += 64) mx = fmaxf(mx, s_p[g][i]);
    mx = wave_max(mx);
    float sum = 0.f;
    for (int i = lane; i < n; i += 64) {
      const float p = exp2f(s_p[g][i] - mx);
      s_p[g][i] = p;
      sum += p;
    }
    sum = wave_sum(sum);
    if (lane == 0) {
      s_m[g] = mx;
      s_l[g] = sum;
    }
  }
  __syncthreads();
  float acc[G][EPL];
#pragma unroll
  for (int g = 0; g < G; ++g)
#pragma unroll
    for (int e = 0; e < EPL; ++e) acc[g][e] = 0.f;
#pragma unroll
  for (int i = 0; i < KPT; ++i) {
    if (i * NSLOT >= n) break;
    const int jj = slot + i * NSLOT;
    if (jj < n) {
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const float p = s_p[g][jj];
#pragma unroll
        for (int e = 0; e < EPL; ++e) acc[g][e] += p * to_f32(rows[i][e]);
      }
    }
  }
  // Slots of one 32-lane half are summed across lanes, the 8 halves of the block in LDS.
  if constexpr (LPK < 32) {
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
      for (int e = 0; e < EPL; ++e) acc[g][e] = stride_sum32<LPK>(acc[g][e]);
  }
  if ((lane & 31) < LPK)
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
      for (int e = 0; e < EPL; ++e) s_red[2 * wave + (lane >> 5)][g][dl * EPL + e] = acc[g][e];
  __syncthreads();
  for (int i = tid; i < G * HD; i += 256) {
    const int g = i / HD, d = i % HD;
    float v = 0.f;
#pragma unroll
    for (int w = 0; w < 8; ++w) v += s_red[w][g][d];
    if (nsplit == 1)
      O[(size_t)b * ldo + (kvh * G + g) * HD + d] = from_f32<T>(v / s_l[g]);
    else
      part_o[(((size_t)b * hq + kvh * G + g) * nsplit + split) * HD + d] = v;
  }
  if (nsplit > 1 && tid < G) {
    float *ml = part_ml + (((size_t)b * hq + kvh * G + tid) * nsplit + split) * 2;
    ml[0] = s_m[tid];
    ml[1] = s_l[tid];
  }
}

// Merge of the splits of one (query head, sequence): log-sum-exp weights in a fixed split
// order, so the result does not depend on which block finished first.
template <typename T, int HD>
__global__ __launch_bounds__(HD) void k_attn_combine(const float *__restrict__ part_o,
                                                      const float *__restrict__ part_ml,
                                                      const int *__restrict__ lens, int len_add,
                                                      int hq, int kpb, int nsplit, int max_ctx,
                                                      T *__restrict__ O, int ldo) {
  __shared__ float s_m[kMaxSplit], s_l[kMaxSplit], s_w[kMaxSplit];
  const int h = blockIdx.x, b = blockIdx.y, d = threadIdx.x;
  const int S = min(lens[b] + len_add, max_ctx);
  const int ns = (S + kpb - 1) / kpb;
  const size_t base = ((size_t)b * hq + h) * nsplit;
  // All split statistics are fetched at once, then every step runs out of LDS.
  for (int sp = d; sp < ns; sp += HD) {
    s_m[sp] = part_ml[(base + sp) * 2];
    s_l[sp] = part_ml[(base + sp) * 2 + 1];
  }
  __syncthreads();
  float mx = -INFINITY;
  for (int sp = 0; sp < ns; ++sp) mx = fmaxf(mx, s_m[sp]);
  for (int sp = d; sp < ns; sp += HD) s_w[sp] = exp2f(s_m[sp] - mx);
  __syncthreads();
  O[(size_t)b * ldo + h * HD + d] = from_f32<T>(merge_splits(part_o + base * HD + d, HD, s_w, s_l, ns));
}

// The merge for up to kCombineDirectSplits splits: one thread per output element, every
// load issued up front (one memory round trip, no block-wide steps).
template <typename T, int HD>
__global__ __launch_bounds__(HD) void k_attn_combine_direct(const float *__restrict__ part_o,
                                                            const float *__restrict__ part_ml,
                                                            const int *__restrict__ lens,
                                                            int len_add, int hq, int kpb,
                                                            int nsplit, int max_ctx,
                                                            T *__restrict__ O, int ldo) {
  const int h = blockIdx.x, b = blockIdx.y, d = threadIdx.x;
  const int S = min(lens[b] + len_add, max_ctx);
  const int ns = (S + kpb - 1) / kpb;
  const size_t base = ((size_t)b * hq + h) * nsplit;
  O[(size_t)b * ldo + h * HD + d] = from_f32<T>(
      merge_splits_direct<kCombineDirectSplits>(part_ml + base * 2, part_o + base * HD + d, HD, ns));
}

template <typename H, int HD>
hipError_t run_prefill_gqa(int group, const void *q, int ldq, const void *kc, const void *vc,
                           void *o, int ldo, const int *cu, const int *kstart, const int4 *sched,
                           const AttnSched &as, int hkv, int max_ctx, hipStream_t s,
                           const KvPaging &pg) {
  const float scale_log2 = kLog2e / sqrtf((float)HD);
#define LL_GQA(G)                                                                             \
  LL_LAUNCH((k_attn_prefill_gqa<H, HD, G>), dim3(as.grid), dim3(512), 0, s,                   \
            reinterpret_cast<const H *>(q), ldq, reinterpret_cast<const H *>(kc),              \
            reinterpret_cast<const H *>(vc), reinterpret_cast<H *>(o), ldo, cu, kstart,        \
            sched, as, hkv, max_ctx, scale_log2, pg)
  switch (group) {
    case 2: LL_GQA(2); break;
    case 4: LL_GQA(4); break;
    case 8: LL_GQA(8); break;
    default: return hipErrorInvalidValue;
  }
#undef LL_GQA
  return hipGetLastError();
}

template <typename T, int HD>
hipError_t run_prefill(const void *q, int ldq, const void *kc, const void *vc, void *o, int ldo,
                       const int *cu, const int *kstart, const int2 *qtiles, int n_qtiles,
                       int hq, int hkv, int max_ctx, hipStream_t s, const KvPaging &pg) {
  const float scale_log2 = kLog2e / sqrtf((float)HD);
  if constexpr (!std::is_same<T, float>::value) {
    LL_LAUNCH((k_attn_prefill_wide<T, HD>), dim3(hq, n_qtiles), dim3(256), 0, s,
              reinterpret_cast<const T *>(q), ldq, reinterpret_cast<const T *>(kc),
              reinterpret_cast<const T *>(vc), reinterpret_cast<T *>(o), ldo, cu, kstart,
              qtiles, hq, hkv, max_ctx, scale_log2, pg);
  } else {
    LL_LAUNCH((k_attn_prefill<T, HD>), dim3(hq, n_qtiles), dim3(256), 0, s,
              reinterpret_cast<const T *>(q), ldq, reinterpret_cast<const T *>(kc),
              reinterpret_cast<const T *>(vc), reinterpret_cast<T *>(o), ldo, cu, kstart, qtiles,
              hq, hkv, max_ctx, scale_log2, pg);
  }
  return hipGetLastError();
}

// Rows per thread so that a block covers kMaxChunk keys.  (Measured on MI355X: fewer, larger
// blocks -- a whole short cache per block, or a loop over chunks inside a block -- were
// slower than more blocks plus the merge kernel: one CU cannot stream a cache fast enough.)
constexpr int kMaxChunk = 256;
template <int HD, int EPL> constexpr int kChunkKpt = kMaxChunk / (256 / (HD / EPL));

template <typename T, int HD, int G>
hipError_t run_decode_g(const void *q, int ldq, const void *kc, const void *vc, const int *lens,
                        int len_add, void *o, int ldo, int batch, int hkv, int max_ctx,
                        const AttnDecodePlan &plan, float *part_o, float *part_ml,
                        hipStream_t s, bool skip_merge, const KvPaging &pg) {
  const float scale_log2 = kLog2e / sqrtf((float)HD);
  constexpr int EPL = Frag<T>::EPL;
  LL_LAUNCH((k_attn_decode<T, HD, G, kChunkKpt<HD, EPL>>), dim3(plan.nsplit, hkv, batch),
            dim3(256), 0, s, reinterpret_cast<const T *>(q), ldq,
            reinterpret_cast<const T *>(kc), reinterpret_cast<const T *>(vc), lens, len_add,
            hkv, max_ctx, plan.kpb, plan.nsplit, part_o, part_ml, reinterpret_cast<T *>(o), ldo,
            scale_log2, pg);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || plan.nsplit == 1 || skip_merge) return e;
  if (g_launch_timer) g_launch_timer->secondary();
  if (plan.nsplit <= kCombineDirectSplits)
    LL_LAUNCH((k_attn_combine_direct<T, HD>), dim3(hkv * G, batch), dim3(HD), 0, s, part_o,
              part_ml, lens, len_add, hkv * G, plan.kpb, plan.nsplit, max_ctx,
              reinterpret_cast<T *>(o), ldo);
  else
    LL_LAUNCH((k_attn_combine<T, HD>), dim3(hkv * G, batch), dim3(HD), 0, s, part_o, part_ml,
              lens, len_add, hkv * G, plan.kpb, plan.nsplit, max_ctx, reinterpret_cast<T *>(o),
              ldo);
  return hipGetLastError();
}

template <typename T, int HD>
hipError_t run_decode(int group, const void *q, int ldq, const void *kc, const void *vc,
                      const int *lens, int len_add, void *o, int ldo, int batch, int hkv,
                      int max_ctx, const AttnDecodePlan &plan, float *part_o, float *part_ml,
                      hipStream_t s, bool skip_merge, const KvPaging &pg) {
#define LL_DECODE_G(G)                                                                       \
  return run_decode_g<T, HD, G>(q, ldq, kc, vc, lens, len_add, o, ldo, batch, hkv, max_ctx, \
                                plan, part_o, part_ml, s, skip_merge, pg)
  switch (group) {
    case 1: LL_DECODE_G(1);
    case 2: LL_DECODE_G(2);
    case 4: LL_DECODE_G(4);
    case 8: LL_DECODE_G(8);
  }
#undef LL_DECODE_G
  return hipErrorInvalidValue;
}

}  // namespace

AttnSched attn_prefill_sched(const PrefillMeta &pm, int group, int hkv) {
  AttnSched as;
  if (group < 2 || group > 8 || 8 % group || hkv < 1 || pm.batch < 1 || pm.batch > 256) return as;
  as.qtile = attn_gqa_qtile(group);
  // causal work of an entry ~ key tiles its queries scan; entries in the device's order
  long total_work = 0;
  for (int b = 0; b < pm.batch; ++b) {
    const int nq = (pm.lens[b] + as.qtile - 1) / as.qtile;
    for (int t = 0; t < nq; ++t)
      total_work += (long)hkv * ((pm.start[b] + std::min((t + 1) * as.qtile, pm.lens[b]) + 63) / 64);
    as.n_entries += nq * hkv;
  }
  // cut[x] = first entry at which the work done before it reaches x / kXcds of the total
  long done = 0;
  int e = 0, x = 1;
  as.cut[0] = 0;
  for (int b = 0; b < pm.batch; ++b) {
    const int nq = (pm.lens[b] + as.qtile - 1) / as.qtile;
    for (int k = 0; k < hkv; ++k)
      for (int j = 0; j < nq; ++j, ++e) {
        while (x < kXcds && done * kXcds >= total_work * x) as.cut[x++] = e;
        const int t = nq - 1 - j;
        done += (pm.start[b] + std::min((t + 1) * as.qtile, pm.lens[b]) + 63) / 64;
      }
  }
  while (x <= kXcds) as.cut[x++] = as.n_entries;
  int longest = 0;
  for (int i = 0; i < kXcds; ++i) longest = std::max(longest, as.cut[i + 1] - as.cut[i]);
  as.grid = kXcds * longest;
  return as;
}

hipError_t launch_attn_prefill(int dtype, int head_dim, const void *q, int ldq, const void *kc,
                               const void *vc, void *o, int ldo, const int *cu,
                               const int *kstart, const int2 *qtiles, int n_qtiles, int hq,
                               int hkv, int max_ctx, hipStream_t s, const KvPaging &pg,
                               const int4 *sched, const AttnSched *as) {
  if (pg.table && (pg.page_len < 256 || pg.page_len % 256 || pg.max_pages < 1))
    return hipErrorInvalidValue;
  if (hkv < 1 || hq % hkv) return hipErrorInvalidValue;
  if (attn_prefill_gqa(dtype, hq / hkv)) {
    if (!sched || !as || as->qtile != attn_gqa_qtile(hq / hkv)) return hipErrorInvalidValue;
    if (as->n_entries <= 0) return hipSuccess;
#define LL_GQA_HD(H, HD)                                                                      \
  return run_prefill_gqa<H, HD>(hq / hkv, q, ldq, kc, vc, o, ldo, cu, kstart, sched, *as, hkv, \
                                max_ctx, s, pg)
    if (dtype == kF16) {
      if (head_dim == 64) LL_GQA_HD(f16, 64);
      if (head_dim == 128) LL_GQA_HD(f16, 128);
    } else {
      if (head_dim == 64) LL_GQA_HD(bf16, 64);
      if (head_dim == 128) LL_GQA_HD(bf16, 128);
    }
#undef LL_GQA_HD
    return hipErrorInvalidValue;
  }
  if (n_qtiles <= 0) return hipSuccess;
#define LL_PREFILL(TT, HD)                                                                   \
  return run_prefill<TT, HD>(q, ldq, kc, vc, o, ldo, cu, kstart, qtiles, n_qtiles, hq, hkv, \
                             max_ctx, s, pg)
  if (dtype == kF32) {
    if (head_dim == 64) LL_PREFILL(float, 64);
    if (head_dim == 128) LL_PREFILL(float, 128);
  } else if (dtype == kF16) {
    if (head_dim == 64) LL_PREFILL(f16, 64);
    if (head_dim == 128) LL_PREFILL(f16, 128);
  } else {
    if (head_dim == 64) LL_PREFILL(bf16, 64);
    if (head_dim == 128) LL_PREFILL(bf16, 128);
  }
#undef LL_PREFILL
  return hipErrorInvalidValue;
}

AttnDecodePlan attn_decode_plan(int head_dim, int elem_bytes, int batch, int hkv,
                                int max_ctx) {
  AttnDecodePlan p;
  (void)head_dim;
  (void)elem_bytes;
  // Chunks of 256 keys, halved (down to 64) until there are ~1024 blocks; a cache that fits
  // one chunk needs no merge.
  int chunk = kMaxChunk;
  while (chunk > 64 && (long)batch * hkv * ((max_ctx + chunk - 1) / chunk) < 1024) chunk >>= 1;
  while ((max_ctx + chunk - 1) / chunk > kMaxSplit) chunk <<= 1;  // only for caches > 8192 keys
  p.kpb = chunk;
  p.nsplit = (max_ctx + chunk - 1) / chunk;
  return p;
}

int attn_decode_max_ctx() { return kMaxSplit * 256; }

hipError_t launch_attn_decode(int dtype, int head_dim, const void *q, int ldq, const void *kc,
                              const void *vc, const int *lens, int len_add, void *o, int ldo,
                              int batch, int hq, int hkv, int max_ctx, const AttnDecodePlan &plan,
                              float *part_o, float *part_ml, hipStream_t s, bool skip_merge,
                              const KvPaging &pg) {
  if (batch <= 0) return hipSuccess;
  if (pg.table && (pg.page_len < 256 || pg.page_len % 256 || pg.max_pages < 1 ||
                   pg.page_len % plan.kpb))
    return hipErrorInvalidValue;
  if (plan.kpb <= 0 || plan.nsplit < 1 || plan.nsplit > kMaxSplit || hq % hkv ||
      (long)plan.kpb * plan.nsplit < max_ctx || plan.kpb > kMaxChunk)
    return hipErrorInvalidValue;
  if (!q || !kc || !vc || !lens || !o || (plan.nsplit > 1 && (!part_o || !part_ml)))
    return hipErrorInvalidValue;
  const int g = hq / hkv;
#define LL_DECODE_HD(TT, HD)                                                                 \
  return run_decode<TT, HD>(g, q, ldq, kc, vc, lens, len_add, o, ldo, batch, hkv, max_ctx,  \
                            plan, part_o, part_ml, s, skip_merge, pg)
  if (dtype == kF32) {
    if (head_dim == 64) LL_DECODE_HD(float, 64);
    if (head_dim == 128) LL_DECODE_HD(float, 128);
  } else if (dtype == kF16) {
    if (head_dim == 64) LL_DECODE_HD(f16, 64);
    if (head_dim == 128) LL_DECODE_HD(f16, 128);
  } else {
    if (head_dim == 64) LL_DECODE_HD(bf16, 64);
    if (head_dim == 128) LL_DECODE_HD(bf16, 128);
  }
#undef LL_DECODE_HD
  return hipErrorInvalidValue;
}

}  // namespace ll
