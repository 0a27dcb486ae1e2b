// Kernels of the RG-LRU recurrent block on gfx950 that are not GEMM epilogues: the load-time
// parameter preparation and the two passes of the prefill scan.
//
// The paper's recurrent case (appendix "Deployment Kernel Families", Table A.4) fuses the
// gates, the recurrent-gate derivation, reset handling, the input normalisation and the scan,
// carrying the state through the sequence inside the kernel and writing the final state once.
// Here the gate GEMM's epilogue already produces, per (token, channel), the decay a_t and the
// normalised input g_t (a_t = 0 at a sequence's first token: the reset), so the prefill scan is
// the linear recurrence h_t = a_t h_{t-1} + g_t.  Its time axis is cut into chunks so that a
// single sequence fills the GPU: pass 1 runs every chunk but each sequence's last one from zero
// and keeps (prod a, h_end); pass 3 chains the earlier chunks' pairs of its sequence into its
// incoming state, rescans, writes h_t * gelu(y_t) and, at a sequence's last chunk, the final
// recurrent state and conv state.  One thread owns one channel of one chunk; every load and
// store of a time step is a contiguous row segment over channels.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "device_common.h"
#include "kernels.h"

namespace ll {
namespace {

constexpr int kRgThreads = 256;
constexpr int kRgStage = 16;

template <typename T>
__global__ __launch_bounds__(256) void k_rg_prep(const T *__restrict__ wt,
                                                 const T *__restrict__ wc, int d,
                                                 const float *__restrict__ lam, int W, float c,
                                                 T *__restrict__ gt, T *__restrict__ gc,
                                                 float *__restrict__ lam_out) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i < d) {
    gt[i] = from_f32<T>(1.0f + to_f32(wt[i]));
    gc[i] = from_f32<T>(1.0f + to_f32(wc[i]));
  }
  if (lam && i < W) lam_out[i] = -c * softplus_f(lam[i]);
}

__global__ __launch_bounds__(256) void k_softcap(float *__restrict__ x, long n, float cap) {
  const long i = (long)blockIdx.x * 256 + threadIdx.x;
  if (i < n) x[i] = cap * tanhf(x[i] / cap);
}

__global__ __launch_bounds__(kRgThreads) void k_rg_scan_chunks(RgScanArgs p) {
  const int c = blockIdx.x * kRgThreads + threadIdx.x;
  const int j = blockIdx.y;
  const int4 ch = p.chunks[j];
  if ((ch.w & kChunkLast) || c >= p.W) return;
  const size_t W = p.W;
  float h = 0.f, P = 1.f;
  const int tend = ch.y + ch.z;
  for (int t0 = ch.y; t0 < tend; t0 += kRgStage) {
    float av[kRgStage], gv[kRgStage];
#pragma unroll
    for (int i = 0; i < kRgStage; ++i) {
      const bool ok = t0 + i < tend;
      av[i] = ok ? p.a[(size_t)(t0 + i) * W + c] : 1.f;
      gv[i] = ok ? p.g[(size_t)(t0 + i) * W + c] : 0.f;
    }
#pragma unroll
    for (int i = 0; i < kRgStage; ++i) {
      h = fmaf(av[i], h, gv[i]);
      P *= av[i];
    }
  }
  p.hend[(size_t)j * W + c] = h;
  p.aprod[(size_t)j * W + c] = P;
}

template <typename T>
__global__ __launch_bounds__(kRgThreads) void k_rg_scan_out(RgScanArgs p) {
  const int c = blockIdx.x * kRgThreads + threadIdx.x;
  const int j = blockIdx.y;
  const int4 ch = p.chunks[j];
  if (c >= p.W) return;
  const size_t W = p.W;
  const int seq = ch.x;
  float h = p.fresh ? 0.f : p.state[(size_t)seq * W + c];
  for (int k = p.seq_chunk0[seq]; k < j; ++k)
    h = fmaf(p.aprod[(size_t)k * W + c], h, p.hend[(size_t)k * W + c]);
  const T *gy = reinterpret_cast<const T *>(p.gy);
  T *out = reinterpret_cast<T *>(p.out);
  const int tend = ch.y + ch.z;
  for (int t0 = ch.y; t0 < tend; t0 += kRgStage) {
    float av[kRgStage], gv[kRgStage], yv[kRgStage];
#pragma unroll
    for (int i = 0; i < kRgStage; ++i) {
      const bool ok = t0 + i < tend;
      const size_t o = (size_t)(ok ? t0 + i : t0) * W + c;
      av[i] = ok ? p.a[o] : 1.f;
      gv[i] = ok ? p.g[o] : 0.f;
      yv[i] = ok ? to_f32(gy[o]) : 0.f;
    }
#pragma unroll
    for (int i = 0; i < kRgStage; ++i) {
      h = fmaf(av[i], h, gv[i]);
      if (t0 + i < tend) out[(size_t)(t0 + i) * W + c] = from_f32<T>(h * yv[i]);
    }
  }
  if (!(ch.w & kChunkLast)) return;
  p.state[(size_t)seq * W + c] = h;
  // the sequence's last K-1 conv inputs: old conv state followed by this call's rows
  const int K1 = p.K - 1;
  const int t0s = p.cu[seq], len = p.cu[seq + 1] - t0s;
  float nv[3];
#pragma unroll
  for (int q = 0; q < 3; ++q) {
    if (q >= K1) continue;
    const int pos = len + q;
    nv[q] = pos < K1 ? (p.fresh ? 0.f : p.conv[((size_t)seq * K1 + pos) * W + c])
                     : p.raw[(size_t)(t0s + pos - K1) * p.ld_raw + c];
  }
#pragma unroll
  for (int q = 0; q < 3; ++q)
    if (q < K1) p.conv[((size_t)seq * K1 + q) * W + c] = nv[q];
}

bool rg_args_ok(const RgScanArgs &a) {
  return a.a && a.g && a.gy && a.out && a.state && a.chunks && a.seq_chunk0 && a.cu && a.conv &&
         a.raw && a.W > 0 && a.K >= 1 && a.K <= 4 && a.ld_raw >= a.W;
}

}  // namespace

int rg_chunk_len(int max_len) {
  const int per = (max_len + kRgMaxChunksPerSeq - 1) / kRgMaxChunksPerSeq;
  return std::max(kRgStage, (per + kRgStage - 1) / kRgStage * kRgStage);
}

hipError_t launch_rg_prep(int dtype, const void *norm_t, const void *norm_c, int d,
                          const float *lam, int W, float c, void *gain_t, void *gain_c,
                          float *lam_out, hipStream_t s) {
  if (!norm_t || !norm_c || !gain_t || !gain_c || (lam && !lam_out) || d < 1 || W < 0)
    return hipErrorInvalidValue;
  const dim3 grid((std::max(d, W) + 255) / 256);
  if (dtype == kF32)
    LL_LAUNCH(k_rg_prep<float>, grid, dim3(256), 0, s, reinterpret_cast<const float *>(norm_t),
              reinterpret_cast<const float *>(norm_c), d, lam, W, c,
              reinterpret_cast<float *>(gain_t), reinterpret_cast<float *>(gain_c), lam_out);
  else
    LL_LAUNCH(k_rg_prep<bf16>, grid, dim3(256), 0, s, reinterpret_cast<const bf16 *>(norm_t),
              reinterpret_cast<const bf16 *>(norm_c), d, lam, W, c,
              reinterpret_cast<bf16 *>(gain_t), reinterpret_cast<bf16 *>(gain_c), lam_out);
  return hipGetLastError();
}

hipError_t launch_softcap(float *x, long n, float cap, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (!x || !(cap > 0.f)) return hipErrorInvalidValue;
  LL_LAUNCH(k_softcap, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, x, n, cap);
  return hipGetLastError();
}

hipError_t launch_rg_scan_chunks(const RgScanArgs &a, int n_chunks, hipStream_t s) {
  if (n_chunks <= 0) return hipSuccess;
  if (!rg_args_ok(a) || !a.hend || !a.aprod) return hipErrorInvalidValue;
  LL_LAUNCH(k_rg_scan_chunks, dim3((a.W + kRgThreads - 1) / kRgThreads, n_chunks),
            dim3(kRgThreads), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_rg_scan_out(int dtype, const RgScanArgs &a, int n_chunks, hipStream_t s) {
  if (n_chunks <= 0) return hipSuccess;
  if (!rg_args_ok(a) || !a.hend || !a.aprod) return hipErrorInvalidValue;
  const dim3 grid((a.W + kRgThreads - 1) / kRgThreads, n_chunks);
  if (dtype == kF32) LL_LAUNCH(k_rg_scan_out<float>, grid, dim3(kRgThreads), 0, s, a);
  else LL_LAUNCH(k_rg_scan_out<bf16>, grid, dim3(kRgThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace ll
