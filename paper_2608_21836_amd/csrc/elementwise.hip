// Row-wise kernels of the decoder: embedding gather, RMSNorm, the final argmax reduction of
// the LM head and the prefill metadata builder.
#include <algorithm>

#include "device_common.h"
#include "kernels.h"

namespace ll {
namespace {

// x[m, :] = E[tokens[m], :] in fp32.  An id outside [0, vocab) sets flag bit 0 and reads row 0.
template <typename T>
__global__ __launch_bounds__(256) void k_embed(const int *__restrict__ tokens,
                                               const T *__restrict__ table, int vocab, int d,
                                               float *__restrict__ x, int *err,
                                               float scale) {
  const int m = blockIdx.x;
  int t = tokens[m];
  if (t < 0 || t >= vocab) {
    if (threadIdx.x == 0 && err) atomicOr(err, 1);
    t = 0;
  }
  const T *src = table + (size_t)t * d;
  float *dst = x + (size_t)m * d;
  for (int i = threadIdx.x; i < d; i += blockDim.x) dst[i] = to_f32(src[i]) * scale;
}

// y[r, :] = x[src, :] / sqrt(mean(x[src, :]^2) + eps) * gain, src = rowmap ? rowmap[r] : r.
template <typename T>
__global__ __launch_bounds__(256) void k_rmsnorm(const float *__restrict__ x, int ldx,
                                                 const int *__restrict__ rowmap, int d,
                                                 const T *__restrict__ gain, float eps,
                                                 T *__restrict__ y, int ldy) {
  const int r = blockIdx.x;
  const int src = rowmap ? rowmap[r] : r;
  const float4 *xr = reinterpret_cast<const float4 *>(x + (size_t)src * ldx);
  const int d4 = d >> 2;
  float ss = 0.f;
  for (int i = threadIdx.x; i < d4; i += 256) {
    const float4 v = xr[i];
    ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  }
  __shared__ float part[4];
  ss = wave_sum(ss);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = ss;
  __syncthreads();
  const float tot = part[0] + part[1] + part[2] + part[3];
  const float scale = 1.0f / sqrtf(tot / (float)d + eps);
  T *yr = y + (size_t)r * ldy;
  for (int i = threadIdx.x; i < d4; i += 256) {
    const float4 v = xr[i];
    yr[4 * i + 0] = from_f32<T>(v.x * scale * to_f32(gain[4 * i + 0]));
    yr[4 * i + 1] = from_f32<T>(v.y * scale * to_f32(gain[4 * i + 1]));
    yr[4 * i + 2] = from_f32<T>(v.z * scale * to_f32(gain[4 * i + 2]));
    yr[4 * i + 3] = from_f32<T>(v.w * scale * to_f32(gain[4 * i + 3]));
  }
}

__device__ __forceinline__ void better(float &bv, int &bi, float ov, int oi) {
  if (ov > bv || (ov == bv && oi < bi)) {
    bv = ov;
    bi = oi;
  }
}

// next[r] = column of the largest partial (lowest column on ties); lens_inc[r] += 1 if given.
// One block of 1024 threads per row; each thread requests 8 partials at a time, so a
// 256000-entry vocabulary (8000 partials) is one round of loads.
constexpr int kArgThreads = 1024, kArgBatch = 8;
__global__ __launch_bounds__(kArgThreads) void k_argmax_reduce(const float *__restrict__ pval,
                                                               const int *__restrict__ pidx,
                                                               int n_parts, int *__restrict__ next,
                                                               int *lens_inc) {
  const int r = blockIdx.x;
  const float *pv = pval + (size_t)r * n_parts;
  const int *pi = pidx + (size_t)r * n_parts;
  float bv = -INFINITY;
  int bi = 0x7fffffff;
  for (int i0 = threadIdx.x; i0 < n_parts; i0 += kArgThreads * kArgBatch) {
    float v[kArgBatch];
    int ix[kArgBatch];
#pragma unroll
    for (int q = 0; q < kArgBatch; ++q) {
      const int i = i0 + q * kArgThreads;
      v[q] = i < n_parts ? pv[i] : -INFINITY;
      ix[q] = i < n_parts ? pi[i] : 0x7fffffff;
    }
#pragma unroll
    for (int q = 0; q < kArgBatch; ++q) better(bv, bi, v[q], ix[q]);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float ov = __shfl_xor(bv, o);
    const int oi = __shfl_xor(bi, o);
    better(bv, bi, ov, oi);
  }
  constexpr int NWV = kArgThreads / 64;
  __shared__ float sv[NWV];
  __shared__ int si[NWV];
  if ((threadIdx.x & 63) == 0) {
    sv[threadIdx.x >> 6] = bv;
    si[threadIdx.x >> 6] = bi;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < NWV; ++w) better(bv, bi, sv[w], si[w]);
    next[r] = bi;
    if (lens_inc) lens_inc[r] += 1;
  }
}

__global__ __launch_bounds__(256) void k_prefill_meta(PrefillMeta pm, int total, int qtile, int *cu,
                                                      int *row_seq, int *row_pos, int *last_row,
                                                      int *lens_dev, int *kstart, int2 *qtiles,
                                                      int4 *sched, int sched_qt, int n_sched,
                                                      int hkv) {
  const int m = blockIdx.x * blockDim.x + threadIdx.x;
  if (sched && m < n_sched) {
    // entry m of the grouped-query work list: sequences in order, then KV heads, then query
    // tiles from the last one
    int b = 0, base = 0;
    for (;;) {
      const int nq = (pm.lens[b] + sched_qt - 1) / sched_qt;
      if (m < base + nq * hkv || b == pm.batch - 1) {
        const int r = m - base, kvh = r / nq, j = r - kvh * nq;
        sched[m] = make_int4(b, nq - 1 - j, kvh, 0);
        break;
      }
      base += nq * hkv;
      ++b;
    }
  }
  if (m < total) {
    int b = 0, first = 0;
    while (b < pm.batch - 1 && m >= first + pm.lens[b]) first += pm.lens[b++];
    row_seq[m] = b;
    row_pos[m] = pm.start[b] + m - first;
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    int acc = 0, maxk = 0;
    for (int b = 0; b < pm.batch; ++b) {
      cu[b] = acc;
      acc += pm.lens[b];
      last_row[b] = acc - 1;
      lens_dev[b] = pm.start[b] + pm.lens[b];
      if (kstart) kstart[b] = pm.start[b];
      maxk = max(maxk, pm.start[b] / qtile + (pm.lens[b] + qtile - 1) / qtile);
    }
    cu[pm.batch] = acc;
    // Longest causal work first: query tile t of sequence b attends to about
    // start[b] + (t + 1) * qtile keys, i.e. kk = start[b] / qtile + t key tiles of its size;
    // each (b, t) appears once, at kk = start[b] / qtile + t.
    int n = 0;
    for (int kk = maxk - 1; kk >= 0; --kk)
      for (int b = 0; b < pm.batch; ++b) {
        const int t = kk - pm.start[b] / qtile;
        if (t >= 0 && t * qtile < pm.lens[b]) qtiles[n++] = make_int2(b, t);
      }
  }
}

// MFMA-only loop for calibration: every wave runs iters rounds of 8 independent
// v_mfma_f32_16x16x32_bf16 on register operands (no memory traffic in the loop) and writes one
// float so that the work is kept.
// The eight chains use different B operands and start values, so that none can be folded
// into another.
__global__ __launch_bounds__(256) void k_mfma_loop(int iters, float *__restrict__ out) {
  bf16x8 a, b0, b1, b2, b3, b4, b5, b6, b7;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const float x = 0.5f - 0.001f * e;
    a[e] = static_cast<bf16>(1.0f + 0.001f * (threadIdx.x & 7));
    b0[e] = static_cast<bf16>(x);
    b1[e] = static_cast<bf16>(x - 0.01f);
    b2[e] = static_cast<bf16>(x - 0.02f);
    b3[e] = static_cast<bf16>(x - 0.03f);
    b4[e] = static_cast<bf16>(x - 0.04f);
    b5[e] = static_cast<bf16>(x - 0.05f);
    b6[e] = static_cast<bf16>(x - 0.06f);
    b7[e] = static_cast<bf16>(x - 0.07f);
  }
  f32x4 c0 = {0.f, 0.f, 0.f, 0.f}, c1 = c0, c2 = c0, c3 = c0, c4 = c0, c5 = c0, c6 = c0,
        c7 = c0;
  // in-place accumulation written out, so that no register copies enter the loop
#define LL_MFMA_STEP(C, B) \
  asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+a"(C) : "v"(a), "v"(B))
  for (int it = 0; it < iters; ++it) {
    LL_MFMA_STEP(c0, b0);
    LL_MFMA_STEP(c1, b1);
    LL_MFMA_STEP(c2, b2);
    LL_MFMA_STEP(c3, b3);
    LL_MFMA_STEP(c4, b4);
    LL_MFMA_STEP(c5, b5);
    LL_MFMA_STEP(c6, b6);
    LL_MFMA_STEP(c7, b7);
  }
#undef LL_MFMA_STEP
  const f32x4 sum = c0 + c1 + c2 + c3 + c4 + c5 + c6 + c7;
  const float t = sum[0] + sum[1] + sum[2] + sum[3];
  if ((threadIdx.x & 63) == 0) out[blockIdx.x * 4 + (threadIdx.x >> 6)] = t;
}

// Element-wise bf16 -> fp16 (exact for magnitudes in [2^-17, 65504]; beyond 65504 the value
// becomes inf and bit 1 of *err is set).
__global__ __launch_bounds__(256) void k_bf16_to_f16(const bf16 *__restrict__ src,
                                                     f16 *__restrict__ dst, size_t n, int *err) {
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (size_t)gridDim.x * 256) {
    const float v = static_cast<float>(src[i]);
    if (fabsf(v) > 65504.f && !__builtin_isnan(v) && err) atomicOr(err, 2);
    dst[i] = static_cast<f16>(v);
  }
}

}  // namespace

hipError_t launch_embed(int dtype, const int *tokens, int ntok, const void *table, int vocab,
                        int d, float *x, int *err, hipStream_t s, float scale) {
  if (ntok <= 0) return hipSuccess;
  if (dtype == kF32)
    LL_LAUNCH(k_embed<float>, dim3(ntok), dim3(256), 0, s, tokens,
                       reinterpret_cast<const float *>(table), vocab, d, x, err, scale);
  else if (dtype == kF16)
    LL_LAUNCH(k_embed<f16>, dim3(ntok), dim3(256), 0, s, tokens,
                       reinterpret_cast<const f16 *>(table), vocab, d, x, err, scale);
  else
    LL_LAUNCH(k_embed<bf16>, dim3(ntok), dim3(256), 0, s, tokens,
                       reinterpret_cast<const bf16 *>(table), vocab, d, x, err, scale);
  return hipGetLastError();
}

hipError_t launch_rmsnorm(int dtype, const float *x, int ldx, const int *rowmap, int rows, int d,
                          const void *gain, float eps, void *y, int ldy, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (dtype == kF32)
    LL_LAUNCH(k_rmsnorm<float>, dim3(rows), dim3(256), 0, s, x, ldx, rowmap, d,
                       reinterpret_cast<const float *>(gain), eps, reinterpret_cast<float *>(y),
                       ldy);
  else if (dtype == kF16)
    LL_LAUNCH(k_rmsnorm<f16>, dim3(rows), dim3(256), 0, s, x, ldx, rowmap, d,
                       reinterpret_cast<const f16 *>(gain), eps, reinterpret_cast<f16 *>(y),
                       ldy);
  else
    LL_LAUNCH(k_rmsnorm<bf16>, dim3(rows), dim3(256), 0, s, x, ldx, rowmap, d,
                       reinterpret_cast<const bf16 *>(gain), eps, reinterpret_cast<bf16 *>(y),
                       ldy);
  return hipGetLastError();
}

hipError_t launch_bf16_to_f16(const void *src, void *dst, size_t n, int *err, hipStream_t s) {
  if (n == 0) return hipSuccess;
  if (!src || !dst) return hipErrorInvalidValue;
  const int blocks = (int)std::min<size_t>((n + 255) / 256, 65536);
  LL_LAUNCH(k_bf16_to_f16, dim3(blocks), dim3(256), 0, s, reinterpret_cast<const bf16 *>(src),
            reinterpret_cast<f16 *>(dst), n, err);
  return hipGetLastError();
}

hipError_t launch_argmax_reduce(const float *pval, const int *pidx, int rows, int n_parts,
                                int *next, int *lens_inc, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (!pval || !pidx || !next) return hipErrorInvalidValue;
  LL_LAUNCH(k_argmax_reduce, dim3(rows), dim3(kArgThreads), 0, s, pval, pidx, n_parts, next,
            lens_inc);
  return hipGetLastError();
}

hipError_t launch_prefill_meta(const PrefillMeta &pm, int total, int qtile, int *cu,
                               int *row_seq, int *row_pos, int *last_row, int *lens_dev,
                               int *kstart, int2 *qtiles, hipStream_t s, int4 *sched,
                               const AttnSched *as, int hkv) {
  if (qtile <= 0 || pm.batch < 1 || pm.batch > 256) return hipErrorInvalidValue;
  const int n_sched = sched && as ? as->n_entries : 0;
  if (sched && (!as || as->qtile <= 0 || hkv < 1)) return hipErrorInvalidValue;
  const int blocks = std::max(1, (std::max(total, n_sched) + 255) / 256);
  LL_LAUNCH(k_prefill_meta, dim3(blocks), dim3(256), 0, s, pm, total, qtile, cu, row_seq,
            row_pos, last_row, lens_dev, kstart, qtiles, n_sched ? sched : nullptr,
            n_sched ? as->qtile : 1, n_sched, std::max(hkv, 1));
  return hipGetLastError();
}

// Calibration: a read-only stream over n4 float4 in which block b reads its own contiguous
// range [b per, (b + 1) per) (per = ceil(n4 / blocks)), eight non-temporal 16-byte loads in
// flight per thread; each block writes the sum of what it read to out[block].  (Contiguous
// ranges per block stream measurably faster than a grid-stride walk over the same bytes.)
__global__ __launch_bounds__(256) void k_read_stream(const f32x4 *__restrict__ src, long n4,
                                                     float *__restrict__ out) {
  constexpr int U = 8;
  const long per = (n4 + gridDim.x - 1) / gridDim.x;
  const long lo = min((long)blockIdx.x * per, n4), hi = min(lo + per, n4);
  float acc = 0.f;
  long i = lo + threadIdx.x;
  for (; i + (U - 1) * 256 < hi; i += U * 256) {
    f32x4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = __builtin_nontemporal_load(src + i + u * 256);
#pragma unroll
    for (int u = 0; u < U; ++u) acc += (v[u][0] + v[u][1]) + (v[u][2] + v[u][3]);
  }
  for (; i < hi; i += 256) {
    const f32x4 v = __builtin_nontemporal_load(src + i);
    acc += (v[0] + v[1]) + (v[2] + v[3]);
  }
  __shared__ float s_w[4];
  acc = wave_sum(acc);
  if ((threadIdx.x & 63) == 0) s_w[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) out[blockIdx.x] = (s_w[0] + s_w[1]) + (s_w[2] + s_w[3]);
}

hipError_t launch_read_stream(const float *src, long n, int blocks, float *out, hipStream_t s) {
  if (n < 0 || n % 4 || blocks < 1 || !out || (n && !src)) return hipErrorInvalidValue;
  LL_LAUNCH(k_read_stream, dim3(blocks), dim3(256), 0, s, reinterpret_cast<const f32x4 *>(src),
            n / 4, out);
  return hipGetLastError();
}

hipError_t launch_mfma_loop(int blocks, int iters, float *out, hipStream_t s) {
  if (blocks < 1 || iters < 1 || !out) return hipErrorInvalidValue;
  LL_LAUNCH(k_mfma_loop, dim3(blocks), dim3(256), 0, s, iters, out);
  return hipGetLastError();
}

}  // namespace ll
