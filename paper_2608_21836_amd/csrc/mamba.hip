// Kernels of the selective state-space (Mamba) mixer on gfx950: prefill metadata, the causal
// depthwise convolution + SiLU, the chunked selective scan (three passes) and small load-time
// transposes.  The in / x / out projections and the LM head run on the GEMM kernels.
//
// The paper's Mamba-family cases (appendix "Deployment Kernel Families", Table A.4) keep the
// SSM state in registers across the scan and load each step's B and C once for all channels;
// here one lane owns one channel and its N = 16 states, and a step's (dt_low | B | C) row is
// the same for every lane of the block, so it is read through the scalar cache.
#include <hip/hip_runtime.h>

#include "device_common.h"
#include "kernels.h"

namespace ll {
namespace {

constexpr int kNS = 16;  // SSM state size the scan kernels are built for

__device__ __forceinline__ float softplus_f(float x) {
  return x > 20.f ? x : log1pf(expf(x));
}

// One block of 256 threads: offsets and chunk list from the per-sequence lengths.
__global__ __launch_bounds__(256) void k_mamba_meta(MambaMeta mm, int total, int chunk_len,
                                                    int *__restrict__ cu,
                                                    int *__restrict__ row_seq,
                                                    int *__restrict__ last_row,
                                                    int4 *__restrict__ chunks,
                                                    int *__restrict__ seq_chunk0) {
  __shared__ int s_cu[257], s_ch[257];
  const int tid = threadIdx.x, B = mm.batch;
  if (tid == 0) {
    int o = 0, oc = 0;
    for (int b = 0; b < B; ++b) {
      s_cu[b] = o;
      s_ch[b] = oc;
      o += mm.lens[b];
      oc += (mm.lens[b] + chunk_len - 1) / chunk_len;
    }
    s_cu[B] = o;
    s_ch[B] = oc;
  }
  __syncthreads();
  for (int b = tid; b <= B; b += blockDim.x) {
    cu[b] = s_cu[b];
    seq_chunk0[b] = s_ch[b];
    if (b < B) {
      last_row[b] = s_cu[b + 1] - 1;
      const int len = mm.lens[b], n = s_ch[b + 1] - s_ch[b];
      for (int k = 0; k < n; ++k) {
        const int r0 = k * chunk_len;
        chunks[s_ch[b] + k] =
            make_int4(b, s_cu[b] + r0, min(chunk_len, len - r0), k == n - 1 ? kChunkLast : 0);
      }
    }
  }
  for (int t = tid; t < total; t += blockDim.x) {
    int lo = 0, hi = B - 1;  // last sequence whose first row is <= t
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (s_cu[mid] <= t) lo = mid;
      else hi = mid - 1;
    }
    row_seq[t] = lo;
  }
}

template <typename T>
__global__ __launch_bounds__(256) void k_mamba_conv(const float *__restrict__ xz, int ldxz,
                                                    const int *__restrict__ row_seq,
                                                    const int *__restrict__ cu,
                                                    const float *__restrict__ conv, int fresh,
                                                    const float *__restrict__ w,
                                                    const float *__restrict__ b, int rows,
                                                    int di, int K, T *__restrict__ u) {
  const long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (long)rows * di) return;
  const int r = (int)(idx / di), c = (int)(idx - (long)r * di);
  const int seq = row_seq ? row_seq[r] : r;
  const int i = cu ? r - cu[seq] : 0;  // index among the sequence's rows of this call
  float acc = b[c];
  for (int k = 0; k < K; ++k) {
    const int q = i - (K - 1) + k;  // < 0: from the conv state
    float v;
    if (q >= 0) v = xz[(size_t)(r - i + q) * ldxz + c];
    else v = fresh ? 0.f : conv[((size_t)seq * (K - 1) + (K - 1) + q) * di + c];
    acc = fmaf(w[c * K + k], v, acc);
  }
  u[(size_t)r * di + c] = from_f32<T>(silu_f(acc));
}

// Passes 1 (kOut = false) and 3 (kOut = true) of the scan; one wave per (channel block, chunk).
template <typename T, bool kOut>
__global__ __launch_bounds__(kScanChannels) void k_scan(
    ScanArgs p, const float *__restrict__ xdbl, const T *__restrict__ u,
    const float *__restrict__ xz, T *__restrict__ y, float *__restrict__ hloc) {
  extern __shared__ float s_w[];  // [R][64] dt projection rows of this block's channels
  const int j = blockIdx.y;
  const int4 ch = p.chunks ? p.chunks[j] : make_int4(j, j, 1, kChunkLast);
  if (!kOut && (ch.w & kChunkLast)) return;  // a sequence's last chunk needs no end state
  const int lane = threadIdx.x, di = p.di, R = p.R;
  const int c = blockIdx.x * kScanChannels + lane;
  for (int r = 0; r < R; ++r) s_w[r * kScanChannels + lane] = p.dtwT[(size_t)r * di + c];
  __syncthreads();
  float a2[kNS], h[kNS];
#pragma unroll
  for (int n = 0; n < kNS; ++n) {
    a2[n] = p.A2[(size_t)n * di + c];
    h[n] = 0.f;
  }
  if (kOut && p.carry == 1) {
#pragma unroll
    for (int n = 0; n < kNS; ++n) h[n] = p.ssm[((size_t)ch.x * kNS + n) * di + c];
  } else if (kOut && p.carry == 2) {
#pragma unroll
    for (int n = 0; n < kNS; ++n) h[n] = hloc[((size_t)j * kNS + n) * di + c];
  }
  const float bias = p.dt_b[c];
  const float Dc = kOut ? p.D[c] : 0.f;
  float dsum = 0.f;
  for (int t = ch.y; t < ch.y + ch.z; ++t) {
    const float *xr = xdbl + (size_t)t * p.ldx;  // same row for the whole wave
    float acc = bias;
    for (int r = 0; r < R; ++r) acc = fmaf(s_w[r * kScanChannels + lane], xr[r], acc);
    const float dt = softplus_f(acc);
    const float uv = to_f32(u[(size_t)t * di + c]);
    const float du = dt * uv;
    const float *Bt = xr + R, *Ct = xr + R + kNS;
    float yv = 0.f;
#pragma unroll
    for (int n = 0; n < kNS; ++n) {
      h[n] = fmaf(exp2f(dt * a2[n]), h[n], du * Bt[n]);
      if (kOut) yv = fmaf(h[n], Ct[n], yv);
    }
    if (kOut) {
      yv = fmaf(Dc, uv, yv);
      y[(size_t)t * di + c] = from_f32<T>(yv * silu_f(xz[(size_t)t * p.ldxz + di + c]));
    } else {
      dsum += dt;
    }
  }
  if (!kOut) {
#pragma unroll
    for (int n = 0; n < kNS; ++n) hloc[((size_t)j * kNS + n) * di + c] = h[n];
    p.dtsum[(size_t)j * di + c] = dsum;
    return;
  }
  if (!(ch.w & kChunkLast)) return;
  // End of the sequence's rows in this call: write its SSM state and the last K-1 conv inputs
  // (the old conv state followed by this call's x rows).
  const int seq = ch.x;
#pragma unroll
  for (int n = 0; n < kNS; ++n) p.ssm[((size_t)seq * kNS + n) * di + c] = h[n];
  const int K1 = p.K - 1;
  const int t0 = p.cu ? p.cu[seq] : seq;
  const int len = p.cu ? p.cu[seq + 1] - t0 : 1;
  float nv[3];
#pragma unroll
  for (int q = 0; q < 3; ++q) {
    if (q >= K1) break;
    const int pos = len + q;  // index into (old state ++ new rows)
    nv[q] = pos < K1 ? (p.fresh ? 0.f : p.conv[((size_t)seq * K1 + pos) * di + c])
                     : xz[(size_t)(t0 + pos - K1) * p.ldxz + c];
  }
#pragma unroll
  for (int q = 0; q < 3; ++q) {
    if (q >= K1) break;
    p.conv[((size_t)seq * K1 + q) * di + c] = nv[q];
  }
}

// Pass 2: per (sequence, channel), chain the chunk end states into each chunk's incoming
// state (written over hloc) starting from the SSM state (zero when fresh).
__global__ __launch_bounds__(kScanChannels) void k_scan_carry(ScanArgs p) {
  const int b = blockIdx.y, di = p.di;
  const int c = blockIdx.x * kScanChannels + threadIdx.x;
  float a2[kNS], H[kNS];
#pragma unroll
  for (int n = 0; n < kNS; ++n) {
    a2[n] = p.A2[(size_t)n * di + c];
    H[n] = p.fresh ? 0.f : p.ssm[((size_t)b * kNS + n) * di + c];
  }
  const int j0 = p.seq_chunk0[b], j1 = p.seq_chunk0[b + 1];
  for (int j = j0; j < j1; ++j) {
    float *hp = p.hloc + (size_t)j * kNS * di + c;
    if (j == j1 - 1) {
#pragma unroll
      for (int n = 0; n < kNS; ++n) hp[(size_t)n * di] = H[n];
      break;
    }
    const float S = p.dtsum[(size_t)j * di + c];
#pragma unroll
    for (int n = 0; n < kNS; ++n) {
      const float hl = hp[(size_t)n * di];
      hp[(size_t)n * di] = H[n];
      H[n] = fmaf(exp2f(a2[n] * S), H[n], hl);
    }
  }
}

__global__ __launch_bounds__(256) void k_transpose_f32(const float *__restrict__ src, int rows,
                                                       int cols, float *__restrict__ dst,
                                                       int neg_exp, float scale) {
  const long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (long)rows * cols) return;
  const int i = (int)(idx / cols), j = (int)(idx - (long)i * cols);
  float v = src[idx];
  if (neg_exp) v = -expf(v);
  dst[(size_t)j * rows + i] = v * scale;
}

template <typename T>
hipError_t scan_launch(bool out, const ScanArgs &a, int n_chunks, hipStream_t s) {
  const dim3 grid(a.di / kScanChannels, n_chunks);
  const size_t lds = (size_t)a.R * kScanChannels * sizeof(float);
  const float *xd = a.xdbl;
  const T *u = reinterpret_cast<const T *>(a.u);
  T *y = reinterpret_cast<T *>(a.y);
  if (out)
    LL_LAUNCH((k_scan<T, true>), grid, dim3(kScanChannels), lds, s, a, xd, u, a.xz, y, a.hloc);
  else
    LL_LAUNCH((k_scan<T, false>), grid, dim3(kScanChannels), lds, s, a, xd, u, a.xz, y, a.hloc);
  return hipGetLastError();
}

bool scan_args_ok(const ScanArgs &a) {
  return a.xdbl && a.u && a.xz && a.dtwT && a.dt_b && a.A2 && a.D && a.ssm && a.conv && a.y &&
         a.N == kNS && a.K >= 1 && a.K <= 4 && a.R >= 1 && a.R <= 256 && a.di > 0 &&
         a.di % kScanChannels == 0 && a.ldx >= a.R + 2 * kNS && a.ldxz >= 2 * a.di;
}

}  // namespace

int mamba_chunk_len(int total, int di) {
  const long waves_per_row = di / kScanChannels;
  long len = (total * waves_per_row + kScanTargetWaves - 1) / kScanTargetWaves;
  len = (len + kScanMinChunk - 1) / kScanMinChunk * kScanMinChunk;
  return (int)std::max<long>(len, kScanMinChunk);
}

int mamba_max_chunks(int max_total, int max_batch, int di) {
  // sum_b ceil(len_b / L) <= total / L + batch, with L >= 16 and L >= total * (di/64) / 2048
  const long a = (max_total + kScanMinChunk - 1) / kScanMinChunk;
  const long b = (long)kScanTargetWaves / std::max(1, di / kScanChannels) + 1;
  return (int)(std::min(a, b) + max_batch);
}

hipError_t launch_mamba_meta(const MambaMeta &mm, int total, int chunk_len, int *cu,
                             int *row_seq, int *last_row, int4 *chunks, int *seq_chunk0,
                             hipStream_t s) {
  if (mm.batch < 1 || mm.batch > 256 || chunk_len < 1) return hipErrorInvalidValue;
  LL_LAUNCH(k_mamba_meta, dim3(1), dim3(256), 0, s, mm, total, chunk_len, cu, row_seq, last_row,
            chunks, seq_chunk0);
  return hipGetLastError();
}

hipError_t launch_mamba_conv(int dtype, const float *xz, int ldxz, const int *row_seq,
                             const int *cu, const float *conv_state, int fresh, const float *w,
                             const float *b, int rows, int di, int K, void *u, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (!xz || !w || !b || !u || K < 1 || K > 4 || (!fresh && !conv_state) ||
      ((row_seq == nullptr) != (cu == nullptr)))
    return hipErrorInvalidValue;
  const long n = (long)rows * di;
  const dim3 grid((unsigned)((n + 255) / 256));
  if (dtype == kF32)
    LL_LAUNCH(k_mamba_conv<float>, grid, dim3(256), 0, s, xz, ldxz, row_seq, cu, conv_state,
              fresh, w, b, rows, di, K, reinterpret_cast<float *>(u));
  else
    LL_LAUNCH(k_mamba_conv<bf16>, grid, dim3(256), 0, s, xz, ldxz, row_seq, cu, conv_state,
              fresh, w, b, rows, di, K, reinterpret_cast<bf16 *>(u));
  return hipGetLastError();
}

hipError_t launch_scan_chunks(int dtype, const ScanArgs &a, int n_chunks, hipStream_t s) {
  if (n_chunks <= 0) return hipSuccess;
  if (!scan_args_ok(a) || !a.chunks || !a.hloc || !a.dtsum) return hipErrorInvalidValue;
  return dtype == kF32 ? scan_launch<float>(false, a, n_chunks, s)
                       : scan_launch<bf16>(false, a, n_chunks, s);
}

hipError_t launch_scan_carry(const ScanArgs &a, int batch, hipStream_t s) {
  if (batch <= 0) return hipSuccess;
  if (!scan_args_ok(a) || !a.seq_chunk0 || !a.hloc || !a.dtsum) return hipErrorInvalidValue;
  LL_LAUNCH(k_scan_carry, dim3(a.di / kScanChannels, batch), dim3(kScanChannels), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_scan_out(int dtype, const ScanArgs &a, int n_chunks, hipStream_t s) {
  if (n_chunks <= 0) return hipSuccess;
  if (!scan_args_ok(a) || (a.chunks && !a.cu) || (a.carry == 2 && !a.hloc) || a.carry < 0 ||
      a.carry > 2 || (a.carry == 0 && !a.fresh))
    return hipErrorInvalidValue;
  return dtype == kF32 ? scan_launch<float>(true, a, n_chunks, s)
                       : scan_launch<bf16>(true, a, n_chunks, s);
}

hipError_t launch_transpose_f32(const float *src, int rows, int cols, float *dst, int neg_exp,
                                float scale, hipStream_t s) {
  const long n = (long)rows * cols;
  if (n <= 0) return hipSuccess;
  LL_LAUNCH(k_transpose_f32, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, src, rows, cols,
            dst, neg_exp, scale);
  return hipGetLastError();
}

}  // namespace ll
