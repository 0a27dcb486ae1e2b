// Projection GEMMs of the decoder: C = A W^T with W in nn.Linear [out][in] layout.
//
//  * Weights are repacked once into 1 KiB tiles (16 output rows x one MFMA contraction chunk)
//    stored in MFMA operand order, all tiles of a 16-row block contiguous along K.  A wave
//    then fetches an operand with one fully coalesced 1 KiB read and LDS reads are
//    conflict-free.
//  * Prefill (M = prompt tokens): 256 x 256 or 128 x 256 block tiles for 16-bit operands
//    (k_gemm_pp: whole-cache-line loads into LDS rings, two wave groups in a ping-pong of
//    memory and MFMA phases, v_mfma_f32_16x16x32), 256 x 256, 128 x 256 or 64 x 128 tiles
//    through a 4-stage ring otherwise (k_gemm_big; fp32 workloads: v_mfma_f32_16x16x4_f32);
//    short prompts split K over blocks.
//  * Decode (M = batch <= 32 per launch): every weight byte is read once straight from HBM
//    into MFMA B operands (non-temporal), A comes from L2; 8 waves split K, reduced in LDS.
//  * Output columns come in units of 32 = two halves of 16 that land in the same lane, so the
//    epilogues (RoPE pairs (i, i + hd/2), SwiGLU gate/up pairs) need no cross-lane traffic.
#include <algorithm>
#include <type_traits>

#include "device_common.h"
#include "kernels.h"

namespace ll {
namespace {

// ------------------------------------------------------------------------------------------
// Repack
// ------------------------------------------------------------------------------------------
// S: element type of the sources, T: of the tiles (bf16 -> fp16 converts each element; every
// bf16 value of magnitude in [2^-17, 65504] is exact in fp16, smaller ones round to fp16's
// subnormal grid of 2^-24; larger ones become inf, flagged in err bit 1).
template <typename T> struct Chunk16 {  // 16 bytes of elements
  T e[16 / sizeof(T)];
};
template <typename S, typename T>
__device__ __forceinline__ uint4 convert16(uint4 v, int *err) {
  if constexpr (std::is_same<S, T>::value) {
    return v;
  } else {
    static_assert(sizeof(S) == 2 && sizeof(T) == 2, "16-bit conversions only");
    const Chunk16<S> in = __builtin_bit_cast(Chunk16<S>, v);
    Chunk16<T> out;
    bool bad = false;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float f = to_f32(in.e[e]);
      bad |= fabsf(f) > 65504.f && !__builtin_isnan(f);
      out.e[e] = from_f32<T>(f);
    }
    if (bad && err) atomicOr(err, 2);
    return __builtin_bit_cast(uint4, out);
  }
}

template <typename S, typename T = S>
__global__ void k_repack(RepackSrc src, int n, int k, int perm, int hd, int ffn, uint8_t *wt,
                         int *err) {
  static_assert(sizeof(S) == sizeof(T), "same element size");
  constexpr int EPL = Frag<T>::EPL, TK = 4 * EPL;
  const int kb_n = k / TK;
  const size_t total = (size_t)n * k / EPL;  // 16-byte chunks
  for (size_t c = (size_t)blockIdx.x * blockDim.x + threadIdx.x; c < total;
       c += (size_t)gridDim.x * blockDim.x) {
    const size_t tile = c >> 6;
    const int ln = (int)(c & 63);
    const int nb = (int)(tile / kb_n), kb = (int)(tile % kb_n);
    const int nphys = nb * 16 + (ln & 15);
    const int kk = kb * TK + (ln >> 4) * EPL;
    int nlog = nphys;
    if (perm == kPermRope) {
      const int head = nphys / hd, within = nphys % hd;
      const int j = within >> 5, half = (within >> 4) & 1, cc = within & 15;
      nlog = head * hd + (half ? hd / 2 : 0) + 16 * j + cc;
    } else if (perm == kPermGlu) {
      const int u = nphys >> 5, half = (nphys >> 4) & 1, cc = nphys & 15;
      nlog = half * ffn + 16 * u + cc;
    }
    int s = 0;
    while (s < 2 && nlog >= src.rows[s]) nlog -= src.rows[s++];
    // rows past the stacked sources (padding up to n) are zero
    uint4 v = make_uint4(0u, 0u, 0u, 0u);
    if (src.src[s] && nlog < src.rows[s])
      v = convert16<S, T>(*reinterpret_cast<const uint4 *>(reinterpret_cast<const S *>(src.src[s]) +
                                                           (size_t)nlog * k + kk),
                          err);
    *reinterpret_cast<uint4 *>(wt + c * 16) = v;
  }
}

// ------------------------------------------------------------------------------------------
// Epilogues: called with (row m, 32-column unit u, lane column c, first-half value,
// second-half value).
// ------------------------------------------------------------------------------------------
// Eight consecutive outputs of type T from fp32 values, as 16-byte stores.
template <typename T> __device__ __forceinline__ void store8(T *dst, const float *v);
template <typename H> __device__ __forceinline__ void store8_16(H *dst, const float *v) {
  uint32_t w[4];
#pragma unroll
  for (int j = 0; j < 4; ++j)
    w[j] = (uint32_t)__builtin_bit_cast(uint16_t, static_cast<H>(v[2 * j])) |
           ((uint32_t)__builtin_bit_cast(uint16_t, static_cast<H>(v[2 * j + 1])) << 16);
  *reinterpret_cast<uint4 *>(dst) = make_uint4(w[0], w[1], w[2], w[3]);
}
template <> __device__ __forceinline__ void store8<bf16>(bf16 *dst, const float *v) {
  store8_16(dst, v);
}
template <> __device__ __forceinline__ void store8<f16>(f16 *dst, const float *v) {
  store8_16(dst, v);
}
template <> __device__ __forceinline__ void store8<float>(float *dst, const float *v) {
  reinterpret_cast<float4 *>(dst)[0] = make_float4(v[0], v[1], v[2], v[3]);
  reinterpret_cast<float4 *>(dst)[1] = make_float4(v[4], v[5], v[6], v[7]);
}

// kVec8 epilogues also take eight consecutive columns of each half of a 32-column unit at once
// (vec8(m, u, c0, first[8], second[8]): columns 32 u + c0 .. + 7 and 32 u + 16 + c0 .. + 7),
// which the prefill GEMM feeds from an LDS transpose of its accumulators.
struct EpiStore {
  float *out;
  int ld;
  static constexpr bool kArgmax = false, kPairs = false, kVec8 = false;
  __device__ void operator()(int m, int u, int c, float v0, float v1) const {
    float *p = out + (size_t)m * ld + 32 * u + c;
    p[0] = v0;
    p[16] = v1;
  }
  __device__ void one(int m, int col, float v) const { out[(size_t)m * ld + col] = v; }
};

struct EpiResid {
  float *out;
  int ld;
  static constexpr bool kArgmax = false, kPairs = false, kVec8 = true, kAtomicSplit = true;
  // K split over blocks: each block adds its partial sum (fp32 atomics; order not fixed)
  __device__ void add_atomic(int m, int col, float v, bool) const {
    unsafeAtomicAdd(out + (size_t)m * ld + col, v);
  }
  __device__ void operator()(int m, int u, int c, float v0, float v1) const {
    float *p = out + (size_t)m * ld + 32 * u + c;
    p[0] += v0;
    p[16] += v1;
  }
  __device__ void one(int m, int col, float v) const { out[(size_t)m * ld + col] += v; }
  // 16-byte read-modify-writes when the rows are 16-byte aligned
  __device__ void vec8(int m, int u, int c0, const float *a, const float *b) const {
    float *r = out + (size_t)m * ld + 32 * u + c0;
    if (((ld & 3) | (int)(reinterpret_cast<uintptr_t>(out) & 15)) != 0) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        r[e] += a[e];
        r[16 + e] += b[e];
      }
      return;
    }
    float4 *p = reinterpret_cast<float4 *>(r), *q = reinterpret_cast<float4 *>(r + 16);
    float4 p0 = p[0], p1 = p[1], q0 = q[0], q1 = q[1];
    p0.x += a[0]; p0.y += a[1]; p0.z += a[2]; p0.w += a[3];
    p1.x += a[4]; p1.y += a[5]; p1.z += a[6]; p1.w += a[7];
    q0.x += b[0]; q0.y += b[1]; q0.z += b[2]; q0.w += b[3];
    q1.x += b[4]; q1.y += b[5]; q1.z += b[6]; q1.w += b[7];
    p[0] = p0; p[1] = p1; q[0] = q0; q[1] = q1;
  }
};

template <typename T> struct EpiSwiglu {
  T *out;
  int ld;
  static constexpr bool kArgmax = false, kPairs = true, kVec8 = true;
  __device__ void operator()(int m, int u, int c, float g, float up) const {
    out[(size_t)m * ld + 16 * u + c] = from_f32<T>(silu_f(g) * up);
  }
  __device__ void vec8(int m, int u, int c0, const float *g, const float *up) const {
    float v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = silu_f(g[e]) * up[e];
    store8<T>(out + (size_t)m * ld + 16 * u + c0, v);
  }
};

template <typename T> struct EpiQkv {
  T *q;
  int ldq;
  T *kc, *vc;
  const int *row_seq, *row_pos;
  const float *rcos, *rsin;
  int hq, hkv, hd, max_ctx;
  KvPaging pg;
  static constexpr bool kArgmax = false, kPairs = true, kVec8 = true;
  __device__ void operator()(int m, int u, int c, float v0, float v1) const {
    const int n0 = u * 32;
    const int head = n0 / hd;
    const int j = (n0 - head * hd) >> 5;
    const int half = hd >> 1;
    const int i1 = 16 * j + c, i2 = half + i1;
    const int pos = row_pos[m];
    if (head < hq + hkv) {  // rotate-half RoPE on queries and keys
      const float co = rcos[(size_t)pos * half + i1], si = rsin[(size_t)pos * half + i1];
      const float a = v0 * co - v1 * si, b = v1 * co + v0 * si;
      v0 = a;
      v1 = b;
    }
    T *dst;
    if (head < hq) {
      dst = q + (size_t)m * ldq + head * hd;
    } else {
      const bool is_k = head < hq + hkv;
      const int kvh = is_k ? head - hq : head - hq - hkv;
      const int seq = row_seq ? row_seq[m] : m;
      dst = (is_k ? kc : vc) + kv_row_off(pg, seq, kvh, hkv, max_ctx, pos, hd);
    }
    dst[i1] = from_f32<T>(v0);
    dst[i2] = from_f32<T>(v1);
  }
  // The same for pair indices i1 = 16 j + c0 .. + 7 of one unit: eight RoPE pairs, two
  // 16-byte stores.
  __device__ void vec8(int m, int u, int c0, const float *a, const float *b) const {
    const int n0 = u * 32;
    const int head = n0 / hd;
    const int j = (n0 - head * hd) >> 5;
    const int half = hd >> 1;
    const int i1 = 16 * j + c0, i2 = half + i1;
    const int pos = row_pos[m];
    float x[8], y[8];
    if (head < hq + hkv) {  // rotate-half RoPE on queries and keys
      const float4 *cp = reinterpret_cast<const float4 *>(rcos + (size_t)pos * half + i1);
      const float4 *sp = reinterpret_cast<const float4 *>(rsin + (size_t)pos * half + i1);
      const float4 c4[2] = {cp[0], cp[1]}, s4[2] = {sp[0], sp[1]};
      const float co[8] = {c4[0].x, c4[0].y, c4[0].z, c4[0].w, c4[1].x, c4[1].y, c4[1].z, c4[1].w};
      const float si[8] = {s4[0].x, s4[0].y, s4[0].z, s4[0].w, s4[1].x, s4[1].y, s4[1].z, s4[1].w};
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        x[e] = a[e] * co[e] - b[e] * si[e];
        y[e] = b[e] * co[e] + a[e] * si[e];
      }
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        x[e] = a[e];
        y[e] = b[e];
      }
    }
    T *dst;
    if (head < hq) {
      dst = q + (size_t)m * ldq + head * hd;
    } else {
      const bool is_k = head < hq + hkv;
      const int kvh = is_k ? head - hq : head - hq - hkv;
      const int seq = row_seq ? row_seq[m] : m;
      dst = (is_k ? kc : vc) + kv_row_off(pg, seq, kvh, hkv, max_ctx, pos, hd);
    }
    store8<T>(dst + i1, x);
    store8<T>(dst + i2, y);
  }
};

// in_proj of a Mamba / Mamba2 decode step (row m = sequence m): columns [col0, col0 + nc) are
// the conv inputs, pushed through one step of the causal depthwise convolution with the
// sequence's conv state (u = silu(b + sum_k w[k] window[k]), the window being the K-1 held
// inputs then the new value; the state then shifts by one and keeps it), written to u (type U,
// row stride nc); every other column is stored as fp32 at its own index of `raw` (row stride
// ld_raw).
template <typename U> struct EpiConv {
  U *u;          // [rows][nc]
  float *raw;    // [rows][ld_raw]
  int ld_raw;
  float *conv;   // [rows][K-1][nc] conv state of this layer
  const float *w, *b;  // [nc][K], [nc]
  int col0, nc, K;
  static constexpr bool kArgmax = false, kPairs = false, kVec8 = false;
  __device__ void one(int m, int col, float v) const {
    const int ch = col - col0;
    if (ch < 0 || ch >= nc) {
      raw[(size_t)m * ld_raw + col] = v;
      return;
    }
    float *st = conv + (size_t)m * (K - 1) * nc + ch;
    const float *wc = w + (size_t)ch * K;
    float old[3];
#pragma unroll
    for (int k = 0; k < 3; ++k)
      if (k < K - 1) old[k] = st[(size_t)k * nc];
    float acc = b[ch];
#pragma unroll
    for (int k = 0; k < 3; ++k)
      if (k < K - 1) acc = fmaf(wc[k], old[k], acc);
    acc = fmaf(wc[K - 1], v, acc);
#pragma unroll
    for (int k = 0; k < 2; ++k)
      if (k < K - 2) st[(size_t)k * nc] = old[k + 1];
    if (K > 1) st[(size_t)(K - 2) * nc] = v;
    u[(size_t)m * nc + ch] = from_f32<U>(silu_f(acc));
  }
  __device__ void operator()(int m, int uu, int c, float v0, float v1) const {
    one(m, 32 * uu + c, v0);
    one(m, 32 * uu + 16 + c, v1);
  }
};

// out[m, n] += acc + bias[n]
struct EpiBiasResid {
  float *out;
  int ld;
  const float *bias;
  static constexpr bool kArgmax = false, kPairs = false, kVec8 = false, kAtomicSplit = true;
  __device__ void add_atomic(int m, int col, float v, bool first) const {
    unsafeAtomicAdd(out + (size_t)m * ld + col, first ? v + bias[col] : v);
  }
  __device__ void one(int m, int col, float v) const {
    out[(size_t)m * ld + col] += v + bias[col];
  }
  __device__ void operator()(int m, int u, int c, float v0, float v1) const {
    one(m, 32 * u + c, v0);
    one(m, 32 * u + 16 + c, v1);
  }
};

template <typename T> struct EpiGeglu {
  T *out;
  int ld;
  const float *bg, *bu;
  static constexpr bool kArgmax = false, kPairs = true, kVec8 = true;
  __device__ void operator()(int m, int u, int c, float g, float up) const {
    const int j = 16 * u + c;
    out[(size_t)m * ld + j] = from_f32<T>(gelu_tanh_f(g + bg[j]) * (up + bu[j]));
  }
  __device__ void vec8(int m, int u, int c0, const float *g, const float *up) const {
    const int j0 = 16 * u + c0;
    float v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = gelu_tanh_f(g[e] + bg[j0 + e]) * (up[e] + bu[j0 + e]);
    store8<T>(out + (size_t)m * ld + j0, v);
  }
};

// Recurrent-block input projection (see kEpiRgIn).
template <typename T> struct EpiRgIn {
  T *gy;             // [rows][W]
  T *xc;             // decode: conv output [rows][W]
  float *raw;        // prefill: linear_x output + bias [rows][ld_raw]
  int ld_raw, W, K;
  const float *by, *bx;
  float *conv;       // decode: [rows][K-1][W]
  const float *w, *b;
  static constexpr bool kArgmax = false, kPairs = false, kVec8 = false;
  __device__ void one(int m, int col, float v) const {
    if (col < W) {
      gy[(size_t)m * W + col] = from_f32<T>(gelu_tanh_f(v + by[col]));
      return;
    }
    const int ch = col - W;
    v += bx[ch];
    if (!conv) {
      raw[(size_t)m * ld_raw + ch] = v;
      return;
    }
    float *st = conv + (size_t)m * (K - 1) * W + ch;
    const float *wc = w + (size_t)ch * K;
    float old[3];
#pragma unroll
    for (int k = 0; k < 3; ++k)
      if (k < K - 1) old[k] = st[(size_t)k * W];
    float acc = b[ch];
#pragma unroll
    for (int k = 0; k < 3; ++k)
      if (k < K - 1) acc = fmaf(wc[k], old[k], acc);
    acc = fmaf(wc[K - 1], v, acc);
#pragma unroll
    for (int k = 0; k < 2; ++k)
      if (k < K - 2) st[(size_t)k * W] = old[k + 1];
    if (K > 1) st[(size_t)(K - 2) * W] = v;
    xc[(size_t)m * W + ch] = from_f32<T>(acc);
  }
  __device__ void operator()(int m, int u, int c, float v0, float v1) const {
    one(m, 32 * u + c, v0);
    one(m, 32 * u + 16 + c, v1);
  }
};

// RG-LRU gates (see kEpiRglru).  kGroupA: the GEMM kernels start the A operand of a block
// whose first output column is n0 at column a_off(n0).
template <typename T> struct EpiRglru {
  const T *x;            // the gates' input rows [rows][W]
  const float *ba, *bi, *lam;
  int W, group_n, group_k;
  float *aout, *gout;    // prefill
  const int *row_seq, *cu;
  int fresh;
  float *state;          // decode
  const T *gy;
  T *out;
  static constexpr bool kArgmax = false, kPairs = true, kVec8 = false, kGroupA = true;
  __device__ size_t a_off(int n0) const { return (size_t)(n0 / group_n) * group_k; }
  __device__ void operator()(int m, int u, int c, float ra, float ix) const {
    const int j = 16 * u + c;
    const float r = sigmoid_f(ra + ba[j]), ig = sigmoid_f(ix + bi[j]);
    const float la = lam[j] * r;
    const float a = __expf(la);
    const bool reset = !state && fresh && m == cu[row_seq[m]];
    const float mult = reset ? 1.f : sqrtf(-expm1f(2.f * la));
    const float g = to_f32(x[(size_t)m * W + j]) * ig * mult;
    if (!state) {
      aout[(size_t)m * W + j] = reset ? 0.f : a;
      gout[(size_t)m * W + j] = g;
      return;
    }
    float *sp = state + (size_t)m * W + j;
    const float h = fmaf(a, *sp, g);
    *sp = h;
    out[(size_t)m * W + j] = from_f32<T>(h * to_f32(gy[(size_t)m * W + j]));
  }
};

template <typename E, typename = void> struct AtomicSplit : std::false_type {};
template <typename E>
struct AtomicSplit<E, std::void_t<decltype(E::kAtomicSplit)>>
    : std::integral_constant<bool, E::kAtomicSplit> {};

template <typename E, typename = void> struct GroupA : std::false_type {};
template <typename E>
struct GroupA<E, std::void_t<decltype(E::kGroupA)>> : std::integral_constant<bool, E::kGroupA> {};

// fp32 partial sums of one K range of a split GEMM: plane blockIdx.z of [split][M][ld].
struct EpiPart {
  float *out;
  int ld;
  size_t plane;
  static constexpr bool kArgmax = false, kPairs = false, kVec8 = false;
  __device__ void operator()(int m, int u, int c, float v0, float v1) const {
    float *p = out + blockIdx.z * plane + (size_t)m * ld + 32 * u + c;
    p[0] = v0;
    p[16] = v1;
  }
};

struct EpiArgmax {
  float *logits;  // nullable
  int ld;
  float *pval;
  int *pidx;
  int n_parts;
  static constexpr bool kArgmax = true, kPairs = true, kVec8 = false;
};

// ------------------------------------------------------------------------------------------
// Prefill GEMM
// ------------------------------------------------------------------------------------------
// ------------------------------------------------------------------------------------------
// Large prefill GEMM: 256 x 256 block tiles, 8 waves of 128 x 64, one 1 KiB k-tile per step.
// Operand tiles go straight from global memory into LDS (global_load_lds_dwordx4: each wave
// fills one 1 KiB tile per instruction, lane l's 16 bytes at offset 16 l, which is exactly the
// MFMA operand order) through a ring of 4 stages, loads issued 3 steps ahead.  Each step is
// software-pipelined around its single barrier: the first half of the step's MFMAs runs from
// fragments already in registers, the wave then waits for the next stage, passes the barrier
// and reads the next step's fragments from LDS while the second half of the MFMAs runs.  The
// barrier is a bare s_barrier after an explicit vmcnt wait (a full __syncthreads would also
// wait for the loads just issued for later stages).  Blocks are renumbered so that each XCD
// (workgroups are dealt round-robin to the 8 XCDs) works on a compact group of output tiles
// and shares A and W tiles in its own L2.
// ------------------------------------------------------------------------------------------
// Bijection from dispatch order to a tile order in which XCD x owns a contiguous range.
__device__ __forceinline__ int xcd_remap(int pid, int n) {
  constexpr int kXcd = 8;
  const int per = (n + kXcd - 1) / kXcd;
  const int tall = n % kXcd == 0 ? kXcd : n % kXcd;
  const int x = pid % kXcd, local = pid / kXcd;
  return x < tall ? x * per + local : tall * per + (x - tall) * (per - 1) + local;
}

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// The same pipeline at BM x BN = 256 x 256, 128 x 256 or 64 x 128: 2 x (BN / 64) waves, each
// owning BM / 2 rows and 64 columns.  With a split of K over blockIdx.z, block z covers
// k-tiles [z * ksteps, (z + 1) * ksteps) (ksteps even) and its epilogue writes that range's
// partial sums (EpiPart).
template <typename T, typename Epi, int BM, int BN>
__global__ __launch_bounds__(BN * 2, 1) void k_gemm_big(const T *__restrict__ A, int lda,
                                                        const uint8_t *__restrict__ Wt, int M,
                                                        int N, int K, int ksteps, Epi epi) {
  using F = typename Frag<T>::type;
  constexpr int EPL = Frag<T>::EPL, TK = 4 * EPL;
  constexpr int GM = 4;  // row tiles per group (measured: 4 beats 1, 2, 8 and 16 at 8B shapes)
  constexpr int NW = BN / 32, WN = BN / 64;    // waves: 2 (M) x WN (N)
  constexpr int NA = BM / 16;                  // A tiles per stage (16-row blocks)
  constexpr int NB = BN / 16;                  // W tiles per stage (16-column blocks)
  constexpr int NI = BM / 32;                  // 16-row blocks per wave
  constexpr int S = 4, TPS = NA + NB, LPW = TPS / NW;  // stages, tiles per stage, loads per wave
  static_assert(TPS % NW == 0, "loads split evenly over the waves");
  static_assert(NI % 2 == 0, "each wave's row blocks split into two halves");
  __shared__ uint4 smem[S * TPS * 64];  // [stage][A: NA row tiles | W: NB column tiles][64]
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave / WN, wn = wave % WN;
  const int ntm = (M + BM - 1) / BM, ntn = N / BN;
  // tile order: XCD-contiguous ranges, each walking groups of GM row-tiles across all columns
  const int t = xcd_remap(blockIdx.x, ntm * ntn);
  const int group = t / (GM * ntn), first_m = group * GM;
  const int gsize = min(ntm - first_m, GM);
  const int tm = first_m + (t % (GM * ntn)) % gsize, tn = (t % (GM * ntn)) / gsize;
  const int m0 = tm * BM, n0 = tn * BN;
  if constexpr (GroupA<Epi>::value) A += epi.a_off(n0);
  const int kt_all = K / TK;                   // k-tiles of one 16-row weight block
  const int kt0 = blockIdx.z * ksteps;
  const int nsteps = min(ksteps, kt_all - kt0);

  // Wave w fills stage tiles LPW w .. LPW w + LPW - 1: A tiles (16-row blocks) first, then
  // the 16 W tiles (16-column blocks).
  const uint8_t *src[LPW];
#pragma unroll
  for (int i = 0; i < LPW; ++i) {
    const int tt = wave * LPW + i;
    if (tt < NA) {
      const int row = min(m0 + tt * 16 + (lane & 15), M - 1);
      src[i] = reinterpret_cast<const uint8_t *>(A + (size_t)row * lda + (size_t)kt0 * TK +
                                                 (lane >> 4) * EPL);
    } else {
      src[i] = Wt + (((size_t)(n0 / 16 + tt - NA) * kt_all + kt0) * 64 + lane) * 16;
    }
  }
  // Steps past the end reload the last tile (the data is never read), so that every step
  // issues the same number of loads and the vmcnt arithmetic stays fixed.
  auto issue = [&](int step, int stage) {
    const int st = min(step, nsteps - 1);
#pragma unroll
    for (int i = 0; i < LPW; ++i) {
      const size_t off = wave * LPW + i < NA ? (size_t)st * TK * sizeof(T) : (size_t)st * 1024;
      load_tile_to_lds(src[i] + off, &smem[(stage * TPS + wave * LPW + i) * 64]);
    }
  };

  f32x4 acc[NI][4];
#pragma unroll
  for (int i = 0; i < NI; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto read_frags = [&](int stage, F *fa, F *fb) {
    const uint4 *base = &smem[stage * TPS * 64];
#pragma unroll
    for (int j = 0; j < 4; ++j) fb[j] = *reinterpret_cast<const F *>(&base[(NA + wn * 4 + j) * 64 + lane]);
#pragma unroll
    for (int i = 0; i < NI; ++i) fa[i] = *reinterpret_cast<const F *>(&base[(wm * NI + i) * 64 + lane]);
  };
  auto mma_half = [&](int h, const F *fa, const F *fb) {
#pragma unroll
    for (int i = 0; i < NI / 2; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        acc[h * (NI / 2) + i][j] = mma_chunk(fa[h * (NI / 2) + i], fb[j], acc[h * (NI / 2) + i][j]);
  };
  // One step: loads for step s+3, MFMAs (first half), barrier for stage s+1, fragments of
  // step s+1, MFMAs (second half).  The scheduling barriers keep the compiler from moving
  // MFMAs that need the new fragments up next to the reads.
  auto step_body = [&](int s, const F *ca, const F *cb, F *na, F *nb) {
    issue(s + 3, (s + 3) & 3);
    mma_half(0, ca, cb);
    __builtin_amdgcn_sched_barrier(0);
    wait_vmcnt<2 * LPW>();  // stage s+1 landed (stages s+2, s+3 may still be in flight)
    asm volatile("s_barrier" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
    read_frags((s + 1) & 3, na, nb);
    __builtin_amdgcn_sched_barrier(0);
    mma_half(1, ca, cb);
    __builtin_amdgcn_sched_barrier(0);
  };

  issue(0, 0);
  issue(1, 1);
  issue(2, 2);
  wait_vmcnt<2 * LPW>();
  __syncthreads();
  F fa0[NI], fb0[4], fa1[NI], fb1[4];
  read_frags(0, fa0, fb0);
  // nsteps is even (K is a multiple of two k-tiles); the last step reads a stage it never uses.
  for (int s = 0; s < nsteps; s += 2) {
    step_body(s, fa0, fb0, fa1, fb1);
    step_body(s + 1, fa1, fb1, fa0, fb0);
  }
  wait_vmcnt<0>();

  const int ubase = (n0 + wn * 64) >> 5;
  if constexpr (Epi::kVec8) {
    // Each 16 x 64 block of the wave's accumulators goes through a wave-private LDS scratch
    // (the ring is free once every wave has passed the barrier), and is read back row-wise:
    // lane l takes row l / 4 and eight consecutive columns of both halves of one 32-column
    // unit, so the epilogue loads and stores 16 bytes at a time.
    constexpr int LD = 68;  // row stride in floats (a 16-float skew between the 4-row groups)
    static_assert(NW * 16 * LD * 4 <= S * TPS * 1024, "epilogue scratch fits in the ring");
    __syncthreads();
    float *sc = reinterpret_cast<float *>(smem) + wave * (16 * LD);
    const int rho = lane >> 2, u = (lane >> 1) & 1, c0 = 8 * (lane & 1);
#pragma unroll
    for (int i = 0; i < NI; ++i) {
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) sc[(4 * (lane >> 4) + r) * LD + 16 * j + (lane & 15)] = acc[i][j][r];
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      const float4 *f0 = reinterpret_cast<const float4 *>(sc + rho * LD + 32 * u + c0);
      const float4 *f1 = reinterpret_cast<const float4 *>(sc + rho * LD + 32 * u + 16 + c0);
      const float4 a0 = f0[0], a1 = f0[1], b0 = f1[0], b1 = f1[1];
      const float av[8] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w};
      const float bv[8] = {b0.x, b0.y, b0.z, b0.w, b1.x, b1.y, b1.z, b1.w};
      const int m = m0 + wm * (BM / 2) + i * 16 + rho;
      if (m < M) epi.vec8(m, ubase + u, c0, av, bv);
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    }
  } else {
#pragma unroll
    for (int i = 0; i < NI; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = m0 + wm * (BM / 2) + i * 16 + (lane >> 4) * 4 + r;
        if (m < M) {
#pragma unroll
          for (int p = 0; p < 2; ++p) epi(m, ubase + p, lane & 15, acc[i][2 * p][r], acc[i][2 * p + 1][r]);
        }
      }
  }
}

// ------------------------------------------------------------------------------------------
// Large prefill GEMM for 16-bit operands: BM x 256 block tiles (BM = 256 or 128), 8 waves of
// BM / 2 x 64, v_mfma_f32_16x16x32, in a ping-pong schedule.
//  * Loads.  The texture path spends its time per cache line touched, so a load instruction
//    is cheapest when its 64 lanes cover whole 128-byte lines.  A W tile (1 KiB, contiguous)
//    does; a 16-row x 32-element A tile would touch 16 half lines.  A is therefore staged 64
//    k-elements (one line per row) at a time: an instruction loads 8 whole rows, lane l
//    taking 16-byte chunk (l % 8) ^ ((r / 2) % 8) of row r = l / 8 (+ 8) of a 16-row block,
//    which lands at byte 16 l of the instruction's 1 KiB.  Row r of the block thus holds its
//    chunk c at 16-byte slot 8 r + (c ^ ((r / 2) % 8)): the MFMA fragment reads (16 rows, one
//    chunk) hit 16 distinct 16-byte bank groups.  W keeps one 32-element tile per stage.
//    Rings: A 3 x (BM x 64), W 4 x (256 x 32) (160 KiB at BM = 256).  At k-step s (32
//    elements) every wave issues its share of the W tiles of step s + 3 and of half s % 2 of
//    the A panel s / 2 + 2.
//  * Schedule: the two wave groups (wm = 0, 1; wave w runs on SIMD w % 4, so every SIMD holds
//    one wave of each) alternate between a memory phase (fragments of step s from LDS,
//    loads) and a compute phase (all MFMAs of step s), half a step apart: group 1 passes one
//    extra barrier first.  While one wave of a SIMD runs its MFMAs back to back, the other
//    issues its LDS reads and loads.  (Raising the compute wave's priority with s_setprio
//    measured 1-2 % slower; reading the next step's fragments inside the compute phase,
//    10 % slower.)
//  * Ordering: before the barrier that ends its memory phase a wave finishes its LDS reads
//    (lgkmcnt 0) and confirms that its loads issued two or more steps earlier have landed
//    (vmcnt: every step issues the same number); a stage is refilled only after the memory
//    phases that last read it (both groups') have ended at a barrier.
// Blocks walk the same XCD-aware tile order as k_gemm_big.  K is a multiple of 64.
// ------------------------------------------------------------------------------------------
template <typename T, typename Epi, int BM>
__global__ __launch_bounds__(512, 1) void k_gemm_pp(const T *__restrict__ A, int lda,
                                                   const uint8_t *__restrict__ Wt, int M, int N,
                                                   int K, Epi epi) {
  using F = typename Frag<T>::type;
  static_assert(sizeof(T) == 2, "16-bit operands");
  constexpr int BN = 256, TK = 32, GM = 4;
  constexpr int NA = BM / 16;       // 16-row blocks of the block tile
  constexpr int NB = BN / 16;       // 16-column W tiles per k-step
  constexpr int NI = BM / 32;       // 16-row blocks per wave
  constexpr int AW = NA / 8;        // A instructions (1 KiB) per wave per k-step
  constexpr int WW = NB / 8;        // W instructions per wave per k-step
  constexpr int LPW = AW + WW;      // loads per wave per k-step
  constexpr int ASTAGE = NA * 128;  // uint4 per A stage (BM rows x 64 elements)
  constexpr int WSTAGE = NB * 64;   // uint4 per W stage
  static_assert(NA % 8 == 0, "an A panel splits evenly over 8 waves and two k-steps");
  __shared__ uint4 smem[3 * ASTAGE + 4 * WSTAGE];
  uint4 *const sA = smem;
  uint4 *const sW = smem + 3 * ASTAGE;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave / 4, wn = wave % 4;
  const int ntm = (M + BM - 1) / BM, ntn = N / BN;
  const int t = xcd_remap(blockIdx.x, ntm * ntn);
  const int group = t / (GM * ntn), first_m = group * GM;
  const int gsize = min(ntm - first_m, GM);
  const int tm = first_m + (t % (GM * ntn)) % gsize, tn = (t % (GM * ntn)) / gsize;
  const int m0 = tm * BM, n0 = tn * BN;
  if constexpr (GroupA<Epi>::value) A += epi.a_off(n0);
  const int nsteps = K / TK, npanels = nsteps / 2;

  // A instruction q (0 .. 2 NA - 1) of a panel covers rows 8 q .. 8 q + 7 of the block tile
  // (16-row block q / 2, half q % 2); k-step parity p issues q = p NA + AW wave + i.
  const T *asrc[2][AW];
#pragma unroll
  for (int p = 0; p < 2; ++p)
#pragma unroll
    for (int i = 0; i < AW; ++i) {
      const int q = p * NA + AW * wave + i, r = 8 * (q & 1) + (lane >> 3);
      const int row = min(m0 + 16 * (q >> 1) + r, M - 1);
      asrc[p][i] = A + (size_t)row * lda + 8 * ((lane & 7) ^ ((r >> 1) & 7));
    }
  const uint8_t *wsrc[WW];
#pragma unroll
  for (int i = 0; i < WW; ++i)
    wsrc[i] = Wt + ((size_t)(n0 / 16 + WW * wave + i) * nsteps * 64 + lane) * 16;
  auto load_w = [&](int step, int stage) {
    const int st = min(step, nsteps - 1);
#pragma unroll
    for (int i = 0; i < WW; ++i)
      load_tile_to_lds(wsrc[i] + (size_t)st * 1024, &sW[stage * WSTAGE + (WW * wave + i) * 64]);
  };
  auto load_a = [&](int panel, int p) {
    const int pn = min(panel, npanels - 1);
#pragma unroll
    for (int i = 0; i < AW; ++i)
      load_tile_to_lds(asrc[p][i] + (size_t)pn * 64,
                       &sA[(panel % 3) * ASTAGE + (p * NA + AW * wave + i) * 64]);
  };
  // Steps and panels past the end reload the last ones (never read), so that every step
  // issues the same number of loads and the vmcnt arithmetic stays fixed.
  load_w(0, 0);
  load_w(1, 1);
  load_w(2, 2);
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    load_a(j, 0);
    load_a(j, 1);
  }
  wait_vmcnt<0>();
  __syncthreads();

  // fragment slots: lane l reads row l % 16 of a 16-row block, chunk 4 kc + l / 16
  const int r16 = lane & 15;
  const int aoff0 = 8 * r16 + ((lane >> 4) ^ ((r16 >> 1) & 7));
  const int aoff1 = 8 * r16 + ((4 + (lane >> 4)) ^ ((r16 >> 1) & 7));
  f32x4 acc[NI][4];
#pragma unroll
  for (int i = 0; i < NI; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  if (wm == 1) asm volatile("s_barrier" ::: "memory");
  F fa[NI], fb[4];
  // one k-step; P = s % 2 (the A chunk within the panel and the half of the panel to load)
  auto step = [&](int s, auto P) {
    constexpr int p = decltype(P)::value;
    __builtin_amdgcn_sched_barrier(0);
    const int panel = s >> 1;
    const uint4 *pa = &sA[(panel % 3) * ASTAGE + wm * NI * 128 + (p ? aoff1 : aoff0)];
#pragma unroll
    for (int i = 0; i < NI; ++i) fa[i] = *reinterpret_cast<const F *>(&pa[i * 128]);
    const uint4 *pw = &sW[(s & 3) * WSTAGE + wn * 4 * 64 + lane];
#pragma unroll
    for (int j = 0; j < 4; ++j) fb[j] = *reinterpret_cast<const F *>(&pw[j * 64]);
    load_w(s + 3, (s + 3) & 3);
    load_a(panel + 2, p);
    wait_vmcnt<2 * LPW>();
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < NI; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = mma_chunk(fa[i], fb[j], acc[i][j]);
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("s_barrier" ::: "memory");
  };
  for (int s = 0; s < nsteps; s += 2) {   // nsteps is even
    step(s, std::integral_constant<int, 0>());
    step(s + 1, std::integral_constant<int, 1>());
  }
  if (wm == 0) asm volatile("s_barrier" ::: "memory");
  wait_vmcnt<0>();

  const int ubase = (n0 + wn * 64) >> 5;
  if constexpr (Epi::kVec8) {
    // Each 16 x 64 block of the wave's accumulators goes through a wave-private LDS scratch
    // (the rings are free once every wave has passed the barrier) and is read back row-wise:
    // lane l takes row l / 4 and eight consecutive columns of both halves of one 32-column
    // unit, so the epilogue loads and stores 16 bytes at a time.
    constexpr int LD = 68;  // row stride in floats (a 16-float skew between the 4-row groups)
    static_assert(8 * 16 * LD * 4 <= (int)sizeof(smem), "epilogue scratch fits in the rings");
    __syncthreads();
    float *sc = reinterpret_cast<float *>(smem) + wave * (16 * LD);
    const int rho = lane >> 2, u = (lane >> 1) & 1, c0 = 8 * (lane & 1);
#pragma unroll
    for (int i = 0; i < NI; ++i) {
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) sc[(4 * (lane >> 4) + r) * LD + 16 * j + (lane & 15)] = acc[i][j][r];
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      const float4 *f0 = reinterpret_cast<const float4 *>(sc + rho * LD + 32 * u + c0);
      const float4 *f1 = reinterpret_cast<const float4 *>(sc + rho * LD + 32 * u + 16 + c0);
      const float4 a0 = f0[0], a1 = f0[1], b0 = f1[0], b1 = f1[1];
      const float av[8] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w};
      const float bv[8] = {b0.x, b0.y, b0.z, b0.w, b1.x, b1.y, b1.z, b1.w};
      const int m = m0 + wm * (BM / 2) + i * 16 + rho;
      if (m < M) epi.vec8(m, ubase + u, c0, av, bv);
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    }
  } else {
#pragma unroll
    for (int i = 0; i < NI; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = m0 + wm * (BM / 2) + i * 16 + (lane >> 4) * 4 + r;
        if (m < M) {
#pragma unroll
          for (int p = 0; p < 2; ++p) epi(m, ubase + p, lane & 15, acc[i][2 * p][r], acc[i][2 * p + 1][r]);
        }
      }
  }
}

// ------------------------------------------------------------------------------------------
// Decode GEMM: one block per NB x 16 output columns (NB = 2: one 32-column pair unit; NB = 1:
// a single 16-column block, for element-wise epilogues when pairs would leave CUs idle), 8
// waves splitting K, partial sums reduced through LDS.  Each wave requests U weight tiles per
// n-block before using the first.
//
// Activation source (AM): kAGlobal reads A fragments from global memory next to the weight
// tiles; kAStaged first copies the block's (up to 16) A rows into LDS, which takes the
// activation traffic off the L1 path the weight stream uses; kANorm stages RMSNorm(x)
// computed on the fly: the fp32 residual rows times the gain, rounded to T, with sum(x^2) on
// the side.  The per-row factor 1/sqrt(mean(x^2) + eps) of RMSNorm does not depend on the
// column, so it scales the finished dot products in the epilogue:
//   (x * s * g) . w = s * ((x * g) . w).
// kAMerge (the decode O projection) stages the merge of the decode attention's split
// partials, computed exactly as the merge kernel computes it, so the attention output never
// goes through global memory and the merge kernel's launch disappears.
// ------------------------------------------------------------------------------------------
enum AMode : int { kAGlobal = 0, kAStaged = 1, kANorm = 2, kAMerge = 3 };

// Rows [m_base, m_base + nrows) of the attention-merge operand into LDS (row stride lds_ld):
// element (r, h * hd + d) is the merge of head h's splits for sequence m_base + r.  MAXS >= the
// split count; slots past a row's split count carry weight 0 and add exact zeros, so the value
// equals the merge kernel's (which merges up to kCombineDirectSplits slots).  Each thread
// merges two elements at once so that both sets of loads are in flight together.
template <int MAXS, typename T>
__device__ __forceinline__ void stage_attn_merge(const AttnMergeIn &mg, T *sA, int lds_ld, int K,
                                                 int nrows, int m_base) {
  const int hd = mg.head_dim, hq = K / hd, total = nrows * K;
  auto merged = [&](int i) -> float {
    const int r = i / K, c = i - r * K, h = c / hd, d = c - h * hd;
    const int b = m_base + r;
    const int S = min(mg.lens[b] + mg.len_add, mg.max_ctx);
    const int ns = max((S + mg.kpb - 1) / mg.kpb, 1);
    const size_t base = ((size_t)b * hq + h) * mg.nsplit;
    return merge_splits_direct<MAXS>(mg.part_ml + base * 2, mg.part_o + base * hd + d, hd, ns);
  };
  for (int i = threadIdx.x; i < total; i += 1024) {
    const int i2 = min(i + 512, total - 1);  // a repeat of the last element when past the end
    const float v0 = merged(i), v1 = merged(i2);
    sA[(size_t)(i / K) * lds_ld + i % K] = from_f32<T>(v0);
    if (i + 512 < total) sA[(size_t)(i2 / K) * lds_ld + i2 % K] = from_f32<T>(v1);
  }
}

template <typename T, int MT, int NB, int AM, typename Epi, int KS = 1>
__global__ __launch_bounds__(512) void k_gemm_skinny(const T *__restrict__ A, int lda,
                                                     NormIn norm,
                                                     const uint8_t *__restrict__ Wt, int M,
                                                     int m_base, int K, Epi epi) {
  using F = typename Frag<T>::type;
  constexpr int EPL = Frag<T>::EPL, TK = 4 * EPL, NW = 8, U = 16 / NB;
  static_assert(AM == kAGlobal || MT == 1, "staged operands cover up to 16 rows");
  constexpr bool NORM = AM == kANorm;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int blk = blockIdx.x;
  if constexpr (GroupA<Epi>::value) A += epi.a_off(16 * NB * blk);
  const int kb_n = K / TK;
  // KS > 1: blockIdx.y takes k-tiles [y kb_n / KS, (y + 1) kb_n / KS), split over the waves
  const int ks0 = KS > 1 ? (int)(blockIdx.y * kb_n / KS) : 0;
  const int ksn = KS > 1 ? (int)((blockIdx.y + 1) * kb_n / KS) - ks0 : kb_n;
  const int kb0 = ks0 + (wave * ksn) / NW, kb1 = ks0 + ((wave + 1) * ksn) / NW;
  const uint8_t *wp[NB];
#pragma unroll
  for (int j = 0; j < NB; ++j) wp[j] = Wt + ((size_t)(NB * blk + j) * kb_n * 64 + lane) * 16;
  const F fz = frag_zero<F>();

  f32x4 acc[MT][NB];
  const T *arow[MT];
  bool aok[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
    for (int j = 0; j < NB; ++j) acc[mt][j] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int row = m_base + mt * 16 + (lane & 15);
    aok[mt] = row < M;
    arow[mt] = A + (size_t)(aok[mt] ? row : 0) * lda + (lane >> 4) * EPL;
  }

  // The first batch of weight tiles is requested before anything else.
  F bw[U][NB];
  auto load_w = [&](int kb) {
#pragma unroll
    for (int q = 0; q < U; ++q)
#pragma unroll
      for (int j = 0; j < NB; ++j)
        bw[q][j] = kb + q < kb1 ? load_frag_stream<F>(wp[j] + (size_t)(kb + q) * 1024) : fz;
  };
  load_w(kb0);

  // Staged modes: the block's rows in LDS, row stride K + EPL elements to spread banks.
  extern __shared__ __attribute__((aligned(16))) uint8_t dyn_smem[];
  T *sA = reinterpret_cast<T *>(dyn_smem);
  __shared__ float s_ss[NW][16];  // RMSNorm mode: sums of squares of row slices
  __shared__ int s_wpr;
  const int nrows = min(M - m_base, 16);
  const int lds_ld = K + EPL;
  if constexpr (NORM) {
    // The 8 waves are spread over the rows (wpr waves per row, each a 1/wpr slice of it), so
    // every row's loads are in flight together.
    const T *g = reinterpret_cast<const T *>(norm.gain);
    const int k4n = K / 4;
    int rows2 = 1;
    while (rows2 < nrows) rows2 <<= 1;
    const int wpr = rows2 >= NW ? 1 : NW / rows2;
    const int sl = wave % wpr;
    for (int r = wave / wpr; r < nrows; r += NW / wpr) {
      const int src = norm.rowmap ? norm.rowmap[m_base + r] : m_base + r;
      const float4 *xr = reinterpret_cast<const float4 *>(norm.x + (size_t)src * norm.ldx);
      float part = 0.f;
#pragma unroll 4
      for (int k4 = sl * 64 + lane; k4 < k4n; k4 += 64 * wpr) {
        const float4 v = xr[k4];
        part += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
        T *d = sA + (size_t)r * lds_ld + 4 * k4;
        d[0] = from_f32<T>(v.x * to_f32(g[4 * k4 + 0]));
        d[1] = from_f32<T>(v.y * to_f32(g[4 * k4 + 1]));
        d[2] = from_f32<T>(v.z * to_f32(g[4 * k4 + 2]));
        d[3] = from_f32<T>(v.w * to_f32(g[4 * k4 + 3]));
      }
      part = wave_sum(part);
      if (lane == 0) s_ss[sl][r] = part;
    }
    s_wpr = wpr;
    __syncthreads();
  } else if constexpr (AM == kAStaged) {
    const int cpr = K / EPL;  // 16-byte chunks per row
#pragma unroll 4
    for (int i = threadIdx.x; i < nrows * cpr; i += 512) {
      const int r = i / cpr, c = i % cpr;
      *reinterpret_cast<F *>(sA + (size_t)r * lds_ld + c * EPL) =
          load_frag<F>(A + (size_t)(m_base + r) * lda + c * EPL);
    }
    __syncthreads();
  } else if constexpr (AM == kAMerge) {
    // weight tiles of the first batch are already in flight
    if (norm.merge.nsplit <= 4) stage_attn_merge<4>(norm.merge, sA, lds_ld, K, nrows, m_base);
    else if (norm.merge.nsplit <= 8) stage_attn_merge<8>(norm.merge, sA, lds_ld, K, nrows, m_base);
    else stage_attn_merge<kCombineDirectSplits>(norm.merge, sA, lds_ld, K, nrows, m_base);
    __syncthreads();
  }
  auto a_frag = [&](int mt, int kb) -> F {
    if constexpr (AM != kAGlobal) {
      const int r = lane & 15;
      return r < nrows ? *reinterpret_cast<const F *>(sA + (size_t)r * lds_ld + kb * TK +
                                                       (lane >> 4) * EPL)
                       : fz;
    } else {
      return aok[mt] ? load_frag<F>(arow[mt] + (size_t)kb * TK) : fz;
    }
  };

  // Batches of U k-tiles, the last one predicated (uniformly per wave); the activation
  // fragments of a batch are requested together with its weight tiles.
  for (int kb = kb0; kb < kb1; kb += U) {
    if (kb != kb0) load_w(kb);
    F av[U][MT];
#pragma unroll
    for (int q = 0; q < U; ++q)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) av[q][mt] = kb + q < kb1 ? a_frag(mt, kb + q) : fz;
    // Tiles past kb1 were loaded as zeros, so their products add exactly nothing.
#pragma unroll
    for (int q = 0; q < U; ++q)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int j = 0; j < NB; ++j) acc[mt][j] = mma_chunk(av[q][mt], bw[q][j], acc[mt][j]);
  }

  __shared__ f32x4 red[NW][MT * NB][64];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int j = 0; j < NB; ++j) red[wave][mt * NB + j][lane] = acc[mt][j];
  __syncthreads();
  if (wave != 0) return;
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    f32x4 sv[NB];
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      sv[j] = red[0][mt * NB + j][lane];
#pragma unroll
      for (int w = 1; w < NW; ++w) sv[j] += red[w][mt * NB + j][lane];
    }
    if constexpr (NORM) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int rr = (lane >> 4) * 4 + r;
        float tot = 0.f;
        if (rr < nrows)
          for (int w = 0; w < s_wpr; ++w) tot += s_ss[w][rr];
        const float sc = 1.0f / sqrtf(tot / (float)K + norm.eps);
#pragma unroll
        for (int j = 0; j < NB; ++j) sv[j][r] *= sc;
      }
    }
    const int c = lane & 15;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = m_base + mt * 16 + (lane >> 4) * 4 + r;
      if constexpr (Epi::kArgmax) {
        static_assert(NB == 2, "argmax partials cover 32-column units");
        const int col0 = 32 * blk + c;
        if (m < M && epi.logits) {
          epi.logits[(size_t)m * epi.ld + col0] = sv[0][r];
          epi.logits[(size_t)m * epi.ld + col0 + 16] = sv[1][r];
        }
        float bv = sv[0][r];
        int bi = col0;
        if (sv[1][r] > bv) {
          bv = sv[1][r];
          bi = col0 + 16;
        }
#pragma unroll
        for (int o = 1; o < 16; o <<= 1) {
          const float ov = __shfl_xor(bv, o);
          const int oi = __shfl_xor(bi, o);
          if (ov > bv || (ov == bv && oi < bi)) {
            bv = ov;
            bi = oi;
          }
        }
        if (m < M && c == 0) {
          epi.pval[(size_t)m * epi.n_parts + blk] = bv;
          epi.pidx[(size_t)m * epi.n_parts + blk] = bi;
        }
      } else if constexpr (KS > 1) {
        if (m < M) {
#pragma unroll
          for (int j = 0; j < NB; ++j)
            epi.add_atomic(m, 16 * NB * blk + 16 * j + c, sv[j][r], blockIdx.y == 0);
        }
      } else if constexpr (NB == 2) {
        if (m < M) epi(m, blk, c, sv[0][r], sv[1][r]);
      } else {
        if (m < M) epi.one(m, 16 * blk + c, sv[0][r]);
      }
    }
  }
}

// ------------------------------------------------------------------------------------------
// Split-K decode GEMM for 17..32 rows (e.g. a batch of 32 sequences).  With whole-K blocks
// of 32 columns, every block re-reads all of A (32 rows x K) through L1, as many bytes as its
// weights: the activation traffic, not HBM, then limits the stream.  Here a block of 8 waves
// owns 128 columns (one 16-column weight tile per wave) and a slice of K; its 32 x slice A
// tile is DMA'd into LDS once and feeds all 8 waves.  Slices are as long as still gives
// every CU a block (splitk_plan); each block writes fp32 partial sums part[split][m][n], and a
// second kernel sums the splits in order (deterministic) and applies the epilogue.
// ------------------------------------------------------------------------------------------
template <typename T, int KTS>
__global__ __launch_bounds__(512) void k_gemm_splitk(const T *__restrict__ A, int lda,
                                                     const uint8_t *__restrict__ Wt, int M,
                                                     int m_base, int N, int K,
                                                     float *__restrict__ part) {
  constexpr int kts = KTS;
  using F = typename Frag<T>::type;
  constexpr int EPL = Frag<T>::EPL, TK = 4 * EPL, NW = 8, U = 32;
  __shared__ uint4 sAk[2 * KTS * 64];  // [k-tile][row block][64]
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int ct = blockIdx.x * NW + wave;  // 16-column weight tile of this wave
  const int kb_n = K / TK;
  const int kt0 = blockIdx.y * kts, nk = min(kts, kb_n - kt0);
  const F fz = frag_zero<F>();
  const uint8_t *wp = Wt + (((size_t)ct * kb_n + kt0) * 64 + lane) * 16;
  // The weight stream starts first: a ring of U tiles (32 KiB per wave) in flight, each slot
  // refilled with the tile U ahead as soon as it has been consumed, so the stream never drains
  // between batches (32 tiles measured 3 % faster than 16 on the 8b-gqa gate/up shape).
  // (The scheduling barriers keep the loads in ring order, so the wait before tile q is for
  // the q-th oldest load only.)
  F bw[U];
#pragma unroll
  for (int q = 0; q < U; ++q) {
    bw[q] = load_frag_stream<F>(wp + (size_t)min(q, nk - 1) * 1024);
    __builtin_amdgcn_sched_barrier(0);
  }
  // Then the A slice, DMA'd into LDS in operand order while the weights are in flight: tile
  // (t, rb) holds rows m_base + 16 rb + l % 16 (clamped to M - 1; those results are never
  // stored), contraction indices (kt0 + t) TK + EPL (l / 16) + e.  A fixed number of tiles
  // per wave (slots past 2 nk receive a copy of a valid tile and are never read), so the code
  // stays straight-line.  Waiting for the slice also waits for the first U weight tiles,
  // which the first steps need anyway; the load latencies overlap instead of adding up.
  static_assert((2 * KTS) % NW == 0, "A tiles split evenly over the waves");
  constexpr int NA = 2 * KTS / NW;
#pragma unroll
  for (int j = 0; j < NA; ++j) {
    const int i = wave + NW * j, t = min(i >> 1, nk - 1), rb = i & 1;
    const int row = min(m_base + 16 * rb + (lane & 15), M - 1);
    load_tile_to_lds(A + (size_t)row * lda + (size_t)(kt0 + t) * TK + (lane >> 4) * EPL,
                     &sAk[(size_t)i * 64]);
  }
  asm volatile("s_waitcnt vmcnt(0)\n\ts_barrier" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);

  // The slice is a compile-time number of tiles, fully unrolled: straight-line code in which
  // the compiler's vmcnt bookkeeping sees one load issued per tile consumed and waits only
  // for the oldest.  Past nk (last split only) the weights are replaced by zeros and A is
  // read at a clamped (written) tile, so those steps add exactly zero.
  f32x4 acc[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
#pragma unroll
  for (int tt = 0; tt < KTS; ++tt) {
    const F w = tt < nk ? bw[tt % U] : fz;
    const int ta = min(tt, nk - 1);
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
      acc[rb] = mma_chunk(*reinterpret_cast<const F *>(&sAk[(ta * 2 + rb) * 64 + lane]), w, acc[rb]);
    if (tt + U < KTS) bw[tt % U] = load_frag_stream<F>(wp + (size_t)min(tt + U, nk - 1) * 1024);
    __builtin_amdgcn_sched_barrier(0);
  }
  float *dst = part + (size_t)blockIdx.y * M * N + 16 * ct + (lane & 15);
#pragma unroll
  for (int rb = 0; rb < 2; ++rb)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = m_base + 16 * rb + 4 * (lane >> 4) + r;
      if (m < M) dst[(size_t)m * N] = acc[rb][r];
    }
}

// Sum of the split partials in split order, then the epilogue: per (row, 32-column unit,
// column c) for pairing epilogues, per (row, column) otherwise.
template <typename Epi>
__global__ __launch_bounds__(256) void k_splitk_reduce(const float *__restrict__ part, int nsplit,
                                                       int M, int N, Epi epi) {
  const long idx = (long)blockIdx.x * 256 + threadIdx.x;
  const size_t plane = (size_t)M * N;
  // The splits are read eight at a time, all eight loads in flight before the first add (a
  // plain loop waits for each load in turn); the sum still runs in split order.
  constexpr int R = 8;
  if constexpr (Epi::kPairs) {
    if (idx >= (long)M * (N / 2)) return;
    const int m = (int)(idx / (N / 2)), rem = (int)(idx % (N / 2));
    const int u = rem / 16, c = rem % 16;
    const float *p = part + (size_t)m * N + 32 * u + c;
    float v0 = 0.f, v1 = 0.f;
    for (int s0 = 0; s0 < nsplit; s0 += R) {
      float a[R] = {}, b[R] = {};
#pragma unroll
      for (int q = 0; q < R; ++q)
        if (s0 + q < nsplit) {
          a[q] = p[(size_t)(s0 + q) * plane];
          b[q] = p[(size_t)(s0 + q) * plane + 16];
        }
#pragma unroll
      for (int q = 0; q < R; ++q)
        if (s0 + q < nsplit) {
          v0 += a[q];
          v1 += b[q];
        }
    }
    epi(m, u, c, v0, v1);
  } else {
    if (idx >= (long)M * N) return;
    const int m = (int)(idx / N), n = (int)(idx % N);
    const float *p = part + (size_t)m * N + n;
    float v = 0.f;
    for (int s0 = 0; s0 < nsplit; s0 += R) {
      float a[R] = {};
#pragma unroll
      for (int q = 0; q < R; ++q)
        if (s0 + q < nsplit) a[q] = p[(size_t)(s0 + q) * plane];
#pragma unroll
      for (int q = 0; q < R; ++q)
        if (s0 + q < nsplit) v += a[q];
    }
    epi.one(m, n, v);
  }
}

// Split sums added to the fp32 residual rows (EpiResid), followed by the RMSNorm of the
// updated rows for the next projection: one block of 1024 threads per row, each thread one
// float4 column group per 4096 columns, all split loads in flight together.
template <typename T>
__global__ __launch_bounds__(1024) void k_splitk_resid_norm(const float *__restrict__ part,
                                                            int nsplit, int M, int N,
                                                            float *__restrict__ x, int ldx,
                                                            const T *__restrict__ gain, float eps,
                                                            T *__restrict__ y, int ldy) {
  const int m = blockIdx.x;
  const size_t plane4 = (size_t)M * N / 4;
  const int n4 = N >> 2;
  const float4 *p4 = reinterpret_cast<const float4 *>(part) + (size_t)m * n4;
  float4 *xr = reinterpret_cast<float4 *>(x + (size_t)m * ldx);
  float ss = 0.f;
  for (int i = threadIdx.x; i < n4; i += 1024) {
    float4 v = xr[i];
    float4 a = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll 8
    for (int sp = 0; sp < nsplit; ++sp) {
      const float4 q = p4[sp * plane4 + i];
      a.x += q.x;
      a.y += q.y;
      a.z += q.z;
      a.w += q.w;
    }
    v.x += a.x;
    v.y += a.y;
    v.z += a.z;
    v.w += a.w;
    xr[i] = v;
    ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  }
  __shared__ float s_part[16];
  ss = wave_sum(ss);
  if ((threadIdx.x & 63) == 0) s_part[threadIdx.x >> 6] = ss;
  __syncthreads();
  float tot = 0.f;
#pragma unroll
  for (int w = 0; w < 16; ++w) tot += s_part[w];
  const float scale = 1.0f / sqrtf(tot / (float)N + eps);
  T *yr = y + (size_t)m * ldy;
  for (int i = threadIdx.x; i < n4; i += 1024) {
    const float4 v = xr[i];
    yr[4 * i + 0] = from_f32<T>(v.x * scale * to_f32(gain[4 * i + 0]));
    yr[4 * i + 1] = from_f32<T>(v.y * scale * to_f32(gain[4 * i + 1]));
    yr[4 * i + 2] = from_f32<T>(v.z * scale * to_f32(gain[4 * i + 2]));
    yr[4 * i + 3] = from_f32<T>(v.w * scale * to_f32(gain[4 * i + 3]));
  }
}

// The 256 x 256 kernel is used once it fills most of the 256 CUs with one block each, else
// (or when its last round of blocks would be mostly empty) the 128 x 256 variant, else the
// 64 x 128 variant.
constexpr int kBigGemmMinTiles = 192;

template <typename Epi>
__global__ __launch_bounds__(256) void k_splitk_reduce(const float *__restrict__ part, int nsplit,
                                                       int M, int N, Epi epi);

template <typename T, typename Epi>
hipError_t run_tiled(const void *a, int lda, const void *wt, int m, int n, int k, const Epi &epi,
                     hipStream_t s, float *ws = nullptr, size_t ws_bytes = 0, int tile = 0) {
  const int big_tiles = ((m + 255) / 256) * (n / 256);
  const int half_tiles = ((m + 127) / 128) * (n / 256);
  // Fraction of the last round of 256 blocks that has work; the 128-row tiles are preferred
  // when they fill the rounds clearly better (they run about 5-10 % below the big tiles).
  auto fill = [](int tiles) { return (double)tiles / (((tiles + 255) / 256) * 256); };
  bool prefer_half = fill(half_tiles) * 0.9 > fill(big_tiles);
  // Grouped-A epilogues: a block's columns must stay in one group, and K is not split.
  if constexpr (GroupA<Epi>::value) {
    if (epi.group_n % 256 != 0) tile = kTileMid;
    ws = nullptr;
  }
  // A forced tile family (kTile256, kTile128x256, kTileMid) where the shape allows it.
  if (n % 256 != 0 && tile != kTileMid) tile = kTileAuto;
  if (tile == kTile256) prefer_half = false;
  const int min_tiles = tile == kTileAuto ? kBigGemmMinTiles : 1;
  if (tile == kTileMid) prefer_half = true;
  const int kt = k / tile_k(sizeof(T) == 4 ? kF32 : kBF16);  // k-tiles
  const T *ap = reinterpret_cast<const T *>(a);
  const uint8_t *wp = reinterpret_cast<const uint8_t *>(wt);
  if (n % 256 == 0 && big_tiles >= min_tiles && !prefer_half && tile != kTile128x256) {
    if constexpr (sizeof(T) == 2)
      LL_LAUNCH((k_gemm_pp<T, Epi, 256>), dim3(big_tiles), dim3(512), 0, s, ap, lda, wp, m, n, k,
                epi);
    else
      LL_LAUNCH((k_gemm_big<T, Epi, 256, 256>), dim3(big_tiles), dim3(512), 0, s, ap, lda, wp, m,
                n, k, kt, epi);
    return hipGetLastError();
  }
  if (n % 256 == 0 && half_tiles >= min_tiles && tile != kTileMid) {
    if constexpr (sizeof(T) == 2)
      LL_LAUNCH((k_gemm_pp<T, Epi, 128>), dim3(half_tiles), dim3(512), 0, s, ap, lda, wp, m, n, k,
                epi);
    else
      LL_LAUNCH((k_gemm_big<T, Epi, 128, 256>), dim3(half_tiles), dim3(512), 0, s, ap, lda, wp, m,
                n, k, kt, epi);
    return hipGetLastError();
  }
  // Short prompts: 64 x 128 tiles; when even those are too few to fill the CUs, K is split
  // over blockIdx.z and a second kernel adds the partial sums in split order and runs the
  // epilogue on the totals.
  const int mid_tiles = ((m + 63) / 64) * (n / 128);
  const SplitKPlan sp = prefill_splitk_plan(sizeof(T), m, n, k);
  if (sp.nsplit > 1 && ws && ws_bytes >= sp.ws_bytes) {
    LL_LAUNCH((k_gemm_big<T, EpiPart, 64, 128>), dim3(mid_tiles, 1, sp.nsplit), dim3(256), 0, s,
              ap, lda, wp, m, n, k, sp.kts, EpiPart{ws, n, (size_t)m * n});
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (g_launch_timer) g_launch_timer->secondary();
    const long items = Epi::kPairs ? (long)m * (n / 2) : (long)m * n;
    LL_LAUNCH((k_splitk_reduce<Epi>), dim3((unsigned)((items + 255) / 256)), dim3(256), 0, s, ws,
              sp.nsplit, m, n, epi);
    return hipGetLastError();
  }
  LL_LAUNCH((k_gemm_big<T, Epi, 64, 128>), dim3(mid_tiles), dim3(256), 0, s, ap, lda, wp, m, n,
            k, kt, epi);
  return hipGetLastError();
}

template <typename T, int MT, int NB, int AM, typename Epi>
hipError_t launch_skinny_one(const T *ap, int lda, const NormIn &nz,
                             const uint8_t *w, int m, int mb, int n, int k, const Epi &epi,
                             hipStream_t s, int ksplit = 1) {
  const size_t lds = AM != kAGlobal ? skinny_norm_lds(sizeof(T), m - mb, k) : 0;
  if (lds > kSkinnyMaxNormLds) return hipErrorInvalidValue;
  if constexpr (AtomicSplit<Epi>::value && !Epi::kPairs) {
    if (ksplit == 2) {
      LL_LAUNCH((k_gemm_skinny<T, MT, NB, AM, Epi, 2>), dim3(n / (16 * NB), 2), dim3(512), lds,
                s, ap, lda, nz, w, m, mb, k, epi);
      return hipGetLastError();
    }
  }
  if (ksplit != 1) return hipErrorInvalidValue;
  LL_LAUNCH((k_gemm_skinny<T, MT, NB, AM, Epi>), dim3(n / (16 * NB)), dim3(512), lds, s, ap,
            lda, nz, w, m, mb, k, epi);
  return hipGetLastError();
}


template <typename T, typename Epi>
hipError_t run_splitk(const void *a, int lda, const void *wt, int m, int n, int k, const Epi &epi,
                      const SplitKPlan &plan, float *ws, hipStream_t s,
                      const PostNorm *post = nullptr) {
  const size_t lds = 0;
  for (int mb = 0; mb < m; mb += 32) {
#define LL_SPLITK(KTS)                                                                        \
  LL_LAUNCH((k_gemm_splitk<T, KTS>), dim3(n / 128, plan.nsplit), dim3(512), lds, s,            \
            reinterpret_cast<const T *>(a), lda, reinterpret_cast<const uint8_t *>(wt), m, mb, \
            n, k, ws)
    switch (plan.kts) {
      case 8: LL_SPLITK(8); break;
      case 16: LL_SPLITK(16); break;
      case 24: LL_SPLITK(24); break;
      case 32: LL_SPLITK(32); break;
      case 40: LL_SPLITK(40); break;
      case 48: LL_SPLITK(48); break;
      case 56: LL_SPLITK(56); break;
      case 64: LL_SPLITK(64); break;
      default: return hipErrorInvalidValue;
    }
#undef LL_SPLITK
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (g_launch_timer) g_launch_timer->secondary();
  if constexpr (std::is_same<Epi, EpiResid>::value) {
    if (post) {
      LL_LAUNCH((k_splitk_resid_norm<T>), dim3(m), dim3(1024), 0, s, ws, plan.nsplit, m, n, epi.out,
                epi.ld, reinterpret_cast<const T *>(post->gain), post->eps,
                reinterpret_cast<T *>(post->out), post->ld_out);
      return hipGetLastError();
    }
  }
  const long items = Epi::kPairs ? (long)m * (n / 2) : (long)m * n;
  LL_LAUNCH((k_splitk_reduce<Epi>), dim3((unsigned)((items + 255) / 256)), dim3(256), 0, s, ws,
            plan.nsplit, m, n, epi);
  return hipGetLastError();
}

template <typename T, typename Epi>
hipError_t run_skinny(const void *a, int lda, const NormIn *norm,
                      const void *wt, int m, int n, int k, const Epi &epi, hipStream_t s,
                      int ksplit = 1) {
  const T *ap = reinterpret_cast<const T *>(a);
  const uint8_t *w = reinterpret_cast<const uint8_t *>(wt);
  const NormIn nz = norm ? *norm : NormIn{};
  // Element-wise epilogues take 16-column blocks when 32-column ones would not fill the CUs.
  const bool single = !Epi::kPairs && n / 32 < 256;
  for (int mb = 0; mb < m; mb += 32) {
    const bool one = m - mb <= 16;
    if (norm && !one) return hipErrorInvalidValue;
    // up to 16 rows: A from LDS when the rows fit, else from global memory
    const int am = !one ? kAGlobal
                   : norm && norm->merge.part_o ? kAMerge
                   : norm ? kANorm
                   : skinny_norm_lds(sizeof(T), m - mb, k) <= kSkinnyMaxNormLds ? kAStaged : kAGlobal;
    hipError_t e = hipErrorInvalidValue;
#define LL_SKINNY(MT, NB, AM) \
  e = launch_skinny_one<T, MT, NB, AM>(ap, lda, nz, w, m, mb, n, k, epi, s, MT == 1 ? ksplit : 1)
#define LL_SKINNY_NB(NB)                        \
  do {                                          \
    if (!one) LL_SKINNY(2, NB, kAGlobal);        \
    else if (am == kANorm) LL_SKINNY(1, NB, kANorm); \
    else if (am == kAMerge) {                    \
      if constexpr (std::is_same<Epi, EpiResid>::value) LL_SKINNY(1, NB, kAMerge); \
    }                                            \
    else if (am == kAStaged) LL_SKINNY(1, NB, kAStaged); \
    else LL_SKINNY(1, NB, kAGlobal);             \
  } while (0)
    if constexpr (Epi::kPairs) {
      LL_SKINNY_NB(2);
    } else {
      if (single) LL_SKINNY_NB(1); else LL_SKINNY_NB(2);
    }
#undef LL_SKINNY_NB
#undef LL_SKINNY
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

template <typename T, bool kTiled>
hipError_t dispatch_epi(const void *a, int lda, const NormIn *norm,
                        const void *wt, int m, int n, int k, const EpiParams &ep, hipStream_t s,
                        float *ws = nullptr, size_t ws_bytes = 0, const PostNorm *post = nullptr,
                        bool *post_done = nullptr, int tile = kTileAuto, int ksplit = 1) {
  if (post_done) *post_done = false;
  const SplitKPlan plan = splitk_plan(elem_bytes(sizeof(T) == 4 ? kF32 : kBF16), m, n, k);
  auto run = [&](const auto &epi) {
    using E = std::decay_t<decltype(epi)>;
    if constexpr (kTiled) {
      if constexpr (E::kArgmax) return hipErrorInvalidValue;
      else return run_tiled<T>(a, lda, wt, m, n, k, epi, s, ws, ws_bytes, tile);
    } else {
      if constexpr (!E::kArgmax && !GroupA<E>::value) {
        if (plan.nsplit > 0 && !norm && ws && ws_bytes >= plan.ws_bytes) {
          const bool fuse_post = post && std::is_same<E, EpiResid>::value && n % 4 == 0;
          if (fuse_post && post_done) *post_done = true;
          return run_splitk<T>(a, lda, wt, m, n, k, epi, plan, ws, s, fuse_post ? post : nullptr);
        }
      }
      return run_skinny<T>(a, lda, norm, wt, m, n, k, epi, s,
                           AtomicSplit<E>::value ? ksplit : 1);
    }
  };
  // Refuse, before any launch, pointer sets that a kernel would dereference as null.
  if (ep.kind == kEpiArgmax &&
      (!ep.part_val || !ep.part_idx || ep.n_parts != n / 32))
    return hipErrorInvalidValue;
  if ((ep.kind == kEpiStore || ep.kind == kEpiResid) && !ep.out_f32) return hipErrorInvalidValue;
  if (ep.kind == kEpiSwiglu && !ep.act) return hipErrorInvalidValue;
  if ((ep.kind == kEpiConv || ep.kind == kEpiConvF32) &&
      (!ep.act || !ep.out_f32 || !ep.conv_state || !ep.conv_w || !ep.conv_b || ep.conv_k < 1 ||
       ep.conv_k > 4 || ep.conv_col0 < 0 || ep.conv_n < 1 || ep.conv_col0 + ep.conv_n > n ||
       ep.ld_out < n))
    return hipErrorInvalidValue;
  if (ep.kind == kEpiQkv && (!ep.act || !ep.kcache || !ep.vcache || !ep.row_pos ||
                             !ep.rope_cos || !ep.rope_sin))
    return hipErrorInvalidValue;
  if (norm && !norm->merge.part_o && (!norm->x || !norm->gain)) return hipErrorInvalidValue;
  if (norm && norm->merge.part_o) {
    // The attention-merge operand: decode GEMMs of at most 16 rows with the residual epilogue.
    const AttnMergeIn &mg = norm->merge;
    if (kTiled || ep.kind != kEpiResid || m > 16 || !mg.part_ml || !mg.lens ||
        mg.head_dim < 1 || k % mg.head_dim || mg.kpb < 1 || mg.max_ctx < 1 || mg.nsplit < 2 ||
        mg.nsplit > kCombineDirectSplits || (long)mg.kpb * mg.nsplit < mg.max_ctx)
      return hipErrorInvalidValue;
  }
  if (ep.kind == kEpiBiasResid && (!ep.out_f32 || !ep.bias)) return hipErrorInvalidValue;
  if (ep.kind == kEpiGeglu && (!ep.act || !ep.bias || !ep.bias2)) return hipErrorInvalidValue;
  if (ep.kind == kEpiRgIn &&
      (!ep.act || !ep.bias || !ep.bias2 || ep.width < 1 || n != 2 * ep.width ||
       (ep.conv_state ? (!ep.act2 || !ep.conv_w || !ep.conv_b || ep.conv_k < 1 || ep.conv_k > 4)
                      : (!ep.out_f32 || ep.ld_out < ep.width))))
    return hipErrorInvalidValue;
  if (ep.kind == kEpiRglru &&
      (!ep.rg_x || !ep.bias || !ep.bias2 || !ep.lam || ep.width < 1 || n != 2 * ep.width ||
       ep.group_n < 128 || ep.group_n % 128 != 0 || n % ep.group_n != 0 ||
       ep.group_k != ep.group_n / 2 || lda < ep.width || norm || k != ep.group_k ||
       (ep.rg_state ? (!ep.rg_gy || !ep.act)
                    : (!ep.out_f32 || !ep.out2 || (ep.rg_fresh && (!ep.row_seq || !ep.cu))))))
    return hipErrorInvalidValue;
  switch (ep.kind) {
    case kEpiStore: return run(EpiStore{ep.out_f32, ep.ld_out});
    case kEpiResid: return run(EpiResid{ep.out_f32, ep.ld_out});
    case kEpiSwiglu: return run(EpiSwiglu<T>{reinterpret_cast<T *>(ep.act), ep.ld_act});
    case kEpiQkv:
      return run(EpiQkv<T>{reinterpret_cast<T *>(ep.act), ep.ld_act,
                           reinterpret_cast<T *>(ep.kcache), reinterpret_cast<T *>(ep.vcache),
                           ep.row_seq, ep.row_pos, ep.rope_cos, ep.rope_sin, ep.n_heads,
                           ep.n_kv_heads, ep.head_dim, ep.max_ctx, ep.kv_paging});
    case kEpiArgmax:
      return run(EpiArgmax{ep.out_f32, ep.ld_out, ep.part_val, ep.part_idx, ep.n_parts});
    case kEpiConv:
      return run(EpiConv<T>{reinterpret_cast<T *>(ep.act), ep.out_f32, ep.ld_out, ep.conv_state,
                            ep.conv_w, ep.conv_b, ep.conv_col0, ep.conv_n, ep.conv_k});
    case kEpiConvF32:
      return run(EpiConv<float>{reinterpret_cast<float *>(ep.act), ep.out_f32, ep.ld_out,
                                ep.conv_state, ep.conv_w, ep.conv_b, ep.conv_col0, ep.conv_n,
                                ep.conv_k});
    case kEpiBiasResid: return run(EpiBiasResid{ep.out_f32, ep.ld_out, ep.bias});
    case kEpiGeglu:
      return run(EpiGeglu<T>{reinterpret_cast<T *>(ep.act), ep.ld_act, ep.bias, ep.bias2});
    case kEpiRgIn:
      return run(EpiRgIn<T>{reinterpret_cast<T *>(ep.act), reinterpret_cast<T *>(ep.act2),
                            ep.out_f32, ep.ld_out, ep.width, ep.conv_k, ep.bias, ep.bias2,
                            ep.conv_state, ep.conv_w, ep.conv_b});
    case kEpiRglru:
      return run(EpiRglru<T>{reinterpret_cast<const T *>(ep.rg_x), ep.bias, ep.bias2, ep.lam,
                             ep.width, ep.group_n, ep.group_k, ep.out_f32, ep.out2, ep.row_seq,
                             ep.cu, ep.rg_fresh, ep.rg_state,
                             reinterpret_cast<const T *>(ep.rg_gy), reinterpret_cast<T *>(ep.act)});
  }
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_repack(int dtype, const RepackSrc &src, int n, int k, int perm, int head_dim,
                         int ffn_dim, void *wt, hipStream_t s, int src_dtype, int *err) {
  if (src_dtype < 0) src_dtype = dtype;
  const size_t chunks = (size_t)n * k * elem_bytes(dtype) / 16;
  const int blocks = (int)std::min<size_t>((chunks + 255) / 256, 65536);
  uint8_t *w = reinterpret_cast<uint8_t *>(wt);
  if (dtype == kF32 && src_dtype == kF32)
    LL_LAUNCH((k_repack<float>), dim3(blocks), dim3(256), 0, s, src, n, k, perm, head_dim, ffn_dim, w, err);
  else if (dtype == kBF16 && src_dtype == kBF16)
    LL_LAUNCH((k_repack<bf16>), dim3(blocks), dim3(256), 0, s, src, n, k, perm, head_dim, ffn_dim, w, err);
  else if (dtype == kF16 && src_dtype == kF16)
    LL_LAUNCH((k_repack<f16>), dim3(blocks), dim3(256), 0, s, src, n, k, perm, head_dim, ffn_dim, w, err);
  else if (dtype == kF16 && src_dtype == kBF16)
    LL_LAUNCH((k_repack<bf16, f16>), dim3(blocks), dim3(256), 0, s, src, n, k, perm, head_dim, ffn_dim, w, err);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_gemm_tiled(int dtype, const void *a, int lda, const void *wt, int m, int n,
                             int k, const EpiParams &ep, hipStream_t s, float *ws,
                             size_t ws_bytes, int tile) {
  if (m <= 0) return hipSuccess;
  if (tile < kTileAuto || tile > kTileMid) return hipErrorInvalidValue;
  if (dtype == kF32)
    return dispatch_epi<float, true>(a, lda, nullptr, wt, m, n, k, ep, s, ws, ws_bytes, nullptr,
                                     nullptr, tile);
  if (dtype == kF16)
    return dispatch_epi<f16, true>(a, lda, nullptr, wt, m, n, k, ep, s, ws, ws_bytes, nullptr,
                                   nullptr, tile);
  return dispatch_epi<bf16, true>(a, lda, nullptr, wt, m, n, k, ep, s, ws, ws_bytes, nullptr,
                                  nullptr, tile);
}

hipError_t launch_gemm_skinny(int dtype, const void *a, int lda, const NormIn *norm,
                              const void *wt, int m, int n, int k, const EpiParams &ep,
                              hipStream_t s, float *ws, size_t ws_bytes,
                              const PostNorm *post, bool *post_done, int ksplit) {
  if (post_done) *post_done = false;
  if (m <= 0) return hipSuccess;
  if (post && (!post->gain || !post->out)) return hipErrorInvalidValue;
  if (ksplit != 1 && ksplit != 2) return hipErrorInvalidValue;
  if (dtype == kF32)
    return dispatch_epi<float, false>(a, lda, norm, wt, m, n, k, ep, s, ws, ws_bytes, post,
                                      post_done, kTileAuto, ksplit);
  if (dtype == kF16)
    return dispatch_epi<f16, false>(a, lda, norm, wt, m, n, k, ep, s, ws, ws_bytes, post,
                                    post_done, kTileAuto, ksplit);
  return dispatch_epi<bf16, false>(a, lda, norm, wt, m, n, k, ep, s, ws, ws_bytes, post,
                                   post_done, kTileAuto, ksplit);
}

SplitKPlan prefill_splitk_plan(size_t elem, int m, int n, int k) {
  SplitKPlan p;
  const int tk = elem == 4 ? 16 : 32;
  if (m <= 0 || n % 128 != 0 || k % (2 * tk) != 0) return p;
  // Shapes that the 256-column kernels take are not split.
  if (n % 256 == 0 && ((m + 127) / 128) * (n / 256) >= kBigGemmMinTiles) return p;
  const int tiles = ((m + 63) / 64) * (n / 128);
  if (tiles >= kPrefillSplitMinTiles) return p;
  const int kt = k / tk;
  const int s0 = std::min({kPrefillSplitMax, (kPrefillSplitBlocks + tiles - 1) / tiles, kt / 4});
  if (s0 < 2) return p;
  p.kts = ((kt + s0 - 1) / s0 + 1) / 2 * 2;  // k-tiles per split, even
  p.nsplit = (kt + p.kts - 1) / p.kts;
  if (p.nsplit < 2) return SplitKPlan{};
  p.ws_bytes = (size_t)p.nsplit * m * n * sizeof(float);
  return p;
}

SplitKPlan splitk_plan(size_t elem, int m, int n, int k) {
  SplitKPlan p;
  const int tk = elem == 4 ? 16 : 32;
  if (m <= 16 || n % 128 != 0 || k % tk != 0) return p;
  const int kb_n = k / tk, groups = n / 128;
  // As few K slices as still give every CU a block: each slice's fp32 partials are written and
  // read again by the reduction, so fewer, longer slices (up to 64 k-tiles, a 128 KiB A slice
  // in LDS) move fewer bytes.  Take the longest compiled slice (8, 16, .., 64 k-tiles) that
  // still gives kSplitKBlocks blocks, preferring one that divides K evenly (an uneven last
  // slice leaves its blocks idle early).
  int kts = 8, best_even = 0;
  for (int t = 8; t <= kSplitKMaxTiles; t += 8) {
    const int ns = (kb_n + t - 1) / t;
    if ((long)ns * groups < kSplitKBlocks) break;
    kts = t;
    if (kb_n % t == 0) best_even = t;
  }
  if (best_even) kts = best_even;
  p.kts = kts;
  p.nsplit = (kb_n + kts - 1) / kts;
  p.ws_bytes = (size_t)p.nsplit * m * n * sizeof(float);
  return p;
}

}  // namespace ll
