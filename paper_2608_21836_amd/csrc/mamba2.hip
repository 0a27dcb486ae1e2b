// Kernels of the Mamba2 mixer on gfx950: the chunked scan over heads (passes 1 and 3, the
// carry pass) with the state tile of a head in registers.  The conv + SiLU, the projections,
// the gated RMSNorm (an RMSNorm of g = y * silu(z)) and the LM head run on the shared kernels.
//
// The paper's Mamba2 case (appendix "Deployment Kernel Families", Table A.4) loads the compact
// B and C vectors once per time step and shares them across heads, with the state tile kept in
// registers across the scan.  Here a block covers 16 rows of one head's [P][N] state (16 lanes
// per row, N / 16 states per lane); a stage of 16 steps of B, C, x, dt is staged in LDS in one
// round of loads and read as broadcasts (every row of the block reads the same B and C words).
#include <hip/hip_runtime.h>

#include "device_common.h"
#include "kernels.h"

namespace ll {
namespace {

constexpr int kM2Stage = 16;
constexpr int kM2Threads = 256;

template <bool kOut, int NPT>
__global__ __launch_bounds__(kM2Threads) void k_m2_scan(M2ScanArgs p) {
  constexpr int N = 16 * NPT;
  __shared__ __attribute__((aligned(16))) float s_B[kM2Stage][N];
  __shared__ __attribute__((aligned(16))) float s_C[kM2Stage][N];
  __shared__ float s_x[kM2Stage][kM2Rows];
  __shared__ float s_dt[kM2Stage], s_dec[kM2Stage];
  const int j = blockIdx.y;
  const int4 ch = p.chunks ? p.chunks[j] : make_int4(j, j, 1, kChunkLast);
  if (!kOut && (ch.w & kChunkLast)) return;  // a sequence's last chunk needs no end state
  const int tid = threadIdx.x, pr = tid >> 4, nq = tid & 15;
  const int PB = p.P / kM2Rows;
  const int h = blockIdx.x / PB, pb = blockIdx.x - h * PB;
  const int row = pb * kM2Rows + pr;                 // row of the head's state tile
  const int grp = h / (p.H / p.G);
  const int di = p.di, GN = p.G * N;
  const size_t tile = (size_t)p.P * N;               // one head's state
  const float a2 = p.A2[h], bias = p.dt_b[h], Dh = kOut ? p.D[h] : 0.f;
  // incoming state: none (zero), the sequence's SSM state (carry 1) or the chunk's slot of hloc
  // (carry 2), as one base pointer and two strides
  const float *init = nullptr;
  size_t init_seq = 0, init_chunk = 0;
  if (kOut && p.carry == 1) {
    init = p.ssm;
    init_seq = (size_t)p.H * tile;
  } else if (kOut && p.carry == 2) {
    init = p.hloc;
    init_chunk = (size_t)p.H * tile;
  }
  float st[NPT];
  {
    const float *sp = init ? init + (size_t)ch.x * init_seq + (size_t)j * init_chunk +
                                 (size_t)h * tile + (size_t)row * N + nq
                           : nullptr;
#pragma unroll
    for (int k = 0; k < NPT; ++k) st[k] = sp ? sp[16 * k] : 0.f;
  }
  float dsum = 0.f;
  const int tend = ch.y + ch.z;
  for (int t0 = ch.y; t0 < tend; t0 += kM2Stage) {
    const int nt = min(kM2Stage, tend - t0);
    __syncthreads();  // the previous stage has been read
    {
      // B and C rows of the stage: 2 * 16 * N floats, float4 each, all in flight
      constexpr int V4 = 2 * kM2Stage * N / 4 / kM2Threads;  // float4 per thread
      float4 v[V4];
#pragma unroll
      for (int q = 0; q < V4; ++q) {
        const int e = (q * kM2Threads + tid) * 4;       // element of [2][16][N]
        const int which = e / (kM2Stage * N), rem = e - which * (kM2Stage * N);
        const int r = rem / N, n = rem - r * N;
        v[q] = r < nt ? *reinterpret_cast<const float4 *>(
                            p.xbc + (size_t)(t0 + r) * p.conv_n + di + which * GN + grp * N + n)
                      : make_float4(0.f, 0.f, 0.f, 0.f);
      }
      const float xv = pr < nt ? p.xbc[(size_t)(t0 + pr) * p.conv_n + h * p.P + pb * kM2Rows + nq]
                               : 0.f;
      float dtr = 0.f;
      if (tid < nt) dtr = p.zxd[(size_t)(t0 + tid) * p.ldz + p.dt_col + h];
#pragma unroll
      for (int q = 0; q < V4; ++q) {
        const int e = (q * kM2Threads + tid) * 4;
        const int which = e / (kM2Stage * N), rem = e - which * (kM2Stage * N);
        const int r = rem / N, n = rem - r * N;
        *reinterpret_cast<float4 *>(which ? &s_C[r][n] : &s_B[r][n]) = v[q];
      }
      s_x[pr][nq] = xv;  // s_x[step][row]: thread (pr, nq) loads step pr, row nq
      if (tid < kM2Stage) {
        const float dt = softplus_f(dtr + bias);
        s_dt[tid] = dt;
        s_dec[tid] = exp2_fast(dt * a2);
      }
    }
    float zv[kM2Stage];
#pragma unroll
    for (int i = 0; i < kM2Stage; ++i)
      zv[i] = (kOut && nq == 0 && i < nt) ? p.zxd[(size_t)(t0 + i) * p.ldz + h * p.P + row] : 0.f;
    __syncthreads();
#pragma unroll
    for (int i = 0; i < kM2Stage; ++i) {
      if (i < nt) {
        const float dt = s_dt[i], dec = s_dec[i];
        const float xv = s_x[i][pr];
        const float dtx = dt * xv;
        float ys = 0.f;
#pragma unroll
        for (int k = 0; k < NPT; ++k) {
          st[k] = fmaf(dec, st[k], dtx * s_B[i][nq + 16 * k]);
          if (kOut) ys = fmaf(s_C[i][nq + 16 * k], st[k], ys);
        }
        if (kOut) {
          ys = group_sum<16>(ys);
          if (nq == 0)
            p.g[(size_t)(t0 + i) * di + h * p.P + row] = fmaf(Dh, xv, ys) * silu_fast(zv[i]);
        } else {
          dsum += dt;
        }
      }
    }
  }
  if (!kOut) {
    float *hp = p.hloc + ((size_t)j * p.H + h) * tile + (size_t)row * N + nq;
#pragma unroll
    for (int k = 0; k < NPT; ++k) hp[16 * k] = st[k];
    if (pb == 0 && tid == 0) p.dtsum[(size_t)j * p.H + h] = dsum;
    return;
  }
  if (!(ch.w & kChunkLast)) return;
  const int seq = ch.x;
  float *sp = p.ssm + ((size_t)seq * p.H + h) * tile + (size_t)row * N + nq;
#pragma unroll
  for (int k = 0; k < NPT; ++k) sp[16 * k] = st[k];
  if (!p.update_conv) return;
  // The sequence's last K-1 conv inputs (old conv state followed by this call's rows), spread
  // over the threads of the sequence's last-chunk blocks.
  const int K1 = p.K - 1;
  const int t0s = p.cu[seq], len = p.cu[seq + 1] - t0s;
  for (int cc = blockIdx.x * kM2Threads + tid; cc < p.conv_n; cc += gridDim.x * kM2Threads) {
    float nv[3];
#pragma unroll
    for (int q = 0; q < 3; ++q) {
      if (q >= K1) continue;
      const int pos = len + q;
      nv[q] = pos < K1 ? (p.fresh ? 0.f : p.conv[((size_t)seq * K1 + pos) * p.conv_n + cc])
                       : p.zxd[(size_t)(t0s + pos - K1) * p.ldz + p.conv_col + cc];
    }
#pragma unroll
    for (int q = 0; q < 3; ++q)
      if (q < K1) p.conv[((size_t)seq * K1 + q) * p.conv_n + cc] = nv[q];
  }
}

// Pass 2: per (sequence, head, row, state) element, chain the chunk end states into each
// chunk's incoming state (written over hloc), from the SSM state (zero when fresh).
constexpr int kM2CarryStage = 16;

__global__ __launch_bounds__(256) void k_m2_carry(M2ScanArgs p) {
  const size_t tile = (size_t)p.P * p.N;
  const size_t e = (size_t)blockIdx.x * 256 + threadIdx.x;  // element of [H][P][N]
  if (e >= tile * p.H) return;
  const int b = blockIdx.y;
  const int h = (int)(e / tile);
  const float a2 = p.A2[h];
  float H = p.fresh ? 0.f : p.ssm[(size_t)b * p.H * tile + e];
  const int j0 = p.seq_chunk0[b], j1 = p.seq_chunk0[b + 1];
  const size_t jstride = tile * p.H;
  for (int jb = j0; jb < j1; jb += kM2CarryStage) {
    float hl[kM2CarryStage], S[kM2CarryStage];
#pragma unroll
    for (int i = 0; i < kM2CarryStage; ++i) {
      const int jj = jb + i;
      const bool ok = jj < j1 - 1;
      hl[i] = ok ? p.hloc[(size_t)jj * jstride + e] : 0.f;
      S[i] = ok ? p.dtsum[(size_t)jj * p.H + h] : 0.f;
    }
#pragma unroll
    for (int i = 0; i < kM2CarryStage; ++i) {
      const int jj = jb + i;
      if (jj < j1) {
        p.hloc[(size_t)jj * jstride + e] = H;
        H = fmaf(exp2_fast(a2 * S[i]), H, hl[i]);
      }
    }
  }
}

// ------------------------------------------------------------------------------------------
// Prefill scan of 16-bit models as matrix products (the chunked state-space-duality form of
// the same recurrence), on v_mfma_f32_16x16x32_f16 with fp32 accumulation.  One block of 4
// waves per (head h, chunk of Q <= 64 steps).  With dA_t = dt_t A (log2 units) and
// c_t = dA_{t0} + .. + dA_t, the recurrence h_t = 2^dA_t h_{t-1} + dt_t x_t B_t^T gives
//   h_t = 2^c_t h_init + sum_{s <= t} 2^(c_t - c_s) dt_s x_s B_s^T,
//   y_t = C_t h_t^T = 2^c_t (C_t h_init^T) + sum_{s <= t} (C_t . B_s) 2^(c_t - c_s) dt_s x_s,
// i.e. Y = diag(2^c) C Hinit^T + (S o L) X with S = C B^T and L[t][s] = 2^(c_t - c_s) dt_s
// (s <= t, else 0), and the chunk's end state h_end = 2^c_last h_init + X^T diag(w) B with
// w_s = dt_s 2^(c_last - c_s).  Pass 1 (kOut false) writes h_end from a zero state for every
// chunk but a sequence's last; pass 3 writes g = (y + D x) silu(z) for every chunk and, at a
// sequence's last chunk, the SSM state and the conv state.
// Operands are staged in LDS as fp16 ([t][n] rows of C and B; x, w B and the masked decayed
// scores transposed where the product needs the contraction index contiguous); every row is
// padded by 8 elements so that the 16 rows of a fragment read fall in distinct bank groups.
// ------------------------------------------------------------------------------------------

// LDS layout (fp16 elements).  Pass 3: C and B rows, x transposed, the masked decayed scores and
// the incoming state; the transposed w B of the end state reuses the space of the last two once
// the outputs are done.  Pass 1: w B and x, both transposed.
__device__ __forceinline__ void store4_f16(_Float16 *d, float4 v) {
  d[0] = (_Float16)v.x;
  d[1] = (_Float16)v.y;
  d[2] = (_Float16)v.z;
  d[3] = (_Float16)v.w;
}

template <bool kOut, int N, int P>
struct SsdLds {
  static constexpr int LDN = N + 8, LDQ = kM2SsdChunk + 8;  // padded rows
  static constexpr int C = 0;                               // [Q][LDN]
  static constexpr int B = kOut ? C + kM2SsdChunk * LDN : 0;  // [Q][LDN]
  static constexpr int XT = kOut ? B + kM2SsdChunk * LDN : 0;  // [P][LDQ]
  static constexpr int M = XT + P * LDQ;                      // [Q][LDQ]
  static constexpr int HI = M + kM2SsdChunk * LDQ;            // [P][LDN]
  static constexpr int BT = M;                                // [N][LDQ]
  static constexpr int TOTAL =
      kOut ? (HI + P * LDN > BT + N * LDQ ? HI + P * LDN : BT + N * LDQ) : BT + N * LDQ;
};

template <bool kOut, int N, int P>
__global__ __launch_bounds__(256) void k_m2_ssd(M2ScanArgs p) {
  constexpr int Q = kM2SsdChunk;
  using Lds = SsdLds<kOut, N, P>;
  constexpr int LDN = Lds::LDN, LDQ = Lds::LDQ;
  static_assert(P % 16 == 0 && N % 32 == 0, "16-row output tiles, 32-wide contraction steps");
  __shared__ __attribute__((aligned(16))) _Float16 sm[Lds::TOTAL];
  __shared__ float s_c[Q], s_dt[Q];
  _Float16 *const sC = sm + Lds::C, *const sB = sm + Lds::B, *const sBT = sm + Lds::BT;
  _Float16 *const sXT = sm + Lds::XT, *const sM = sm + Lds::M, *const sH = sm + Lds::HI;

  const int j = blockIdx.y, h = blockIdx.x;
  const int4 ch = p.chunks[j];
  const bool last = ch.w & kChunkLast;
  if (!kOut && last) return;  // a sequence's last chunk needs no end state
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r16 = lane & 15, kq = lane >> 4;
  const int t0 = ch.y, nt = ch.z;
  const int grp = h / (p.H / p.G);
  const int di = p.di, GN = p.G * N;
  const float a2 = p.A2[h], bias = p.dt_b[h];
  const size_t tile = (size_t)P * N;
  const float *init = nullptr;  // incoming state (fp32): the SSM state or the carried one
  if (kOut && p.carry == 1) init = p.ssm + ((size_t)ch.x * p.H + h) * tile;
  if (kOut && p.carry == 2) init = p.hloc + ((size_t)j * p.H + h) * tile;
  const float *xbc = p.xbc + (size_t)t0 * p.conv_n;

  // dt and the cumulative dt of the chunk (steps past its end: dt = 0), as an inclusive scan
  // over the lanes of wave 0 (lane t = step t)
  static_assert(Q == 64, "one step per lane of a wave");
  if (wave == 0) {
    const float dtv = lane < nt ? softplus_f(p.zxd[(size_t)(t0 + lane) * p.ldz + p.dt_col + h] + bias) : 0.f;
    float c = dtv;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const float u = __shfl_up(c, o, 64);
      if (lane >= o) c += u;
    }
    s_dt[lane] = dtv;
    s_c[lane] = c;
    if (!kOut && lane == 63) p.dtsum[(size_t)j * p.H + h] = c;
  }
  // Operands in fp16; rows past the chunk are zero.  Every thread requests all of its loads
  // before its first LDS store, so the global latencies overlap instead of adding up.
  constexpr int NV = N / 4, PV = P / 4;
  constexpr int NBC = Q * NV / 256, NH = P * NV / 256, NX = Q * PV / 256;
  static_assert(Q * NV % 256 == 0 && P * NV % 256 == 0 && Q * PV % 256 == 0, "whole rounds");
  {
    float4 xv[NX];
#pragma unroll
    for (int k = 0; k < NX; ++k) {
      const int i = tid + 256 * k, t = i / PV, q = 4 * (i % PV);
      xv[k] = t < nt ? *reinterpret_cast<const float4 *>(xbc + (size_t)t * p.conv_n + h * P + q)
                     : make_float4(0.f, 0.f, 0.f, 0.f);
    }
    if (kOut) {
      float4 bv[NBC], cv[NBC];
#pragma unroll
      for (int k = 0; k < NBC; ++k) {
        const int i = tid + 256 * k, t = i / NV, n = 4 * (i % NV);
        const float *row = xbc + (size_t)t * p.conv_n + di + grp * N + n;
        bv[k] = t < nt ? *reinterpret_cast<const float4 *>(row) : make_float4(0.f, 0.f, 0.f, 0.f);
        cv[k] = t < nt ? *reinterpret_cast<const float4 *>(row + GN) : make_float4(0.f, 0.f, 0.f, 0.f);
      }
#pragma unroll
      for (int k = 0; k < NBC; ++k) {
        const int i = tid + 256 * k, t = i / NV, n = 4 * (i % NV);
        store4_f16(sB + t * LDN + n, bv[k]);
        store4_f16(sC + t * LDN + n, cv[k]);
      }
      if (init) {
        float4 hv[NH];
#pragma unroll
        for (int k = 0; k < NH; ++k) {
          const int i = tid + 256 * k, q = i / NV, n = 4 * (i % NV);
          hv[k] = *reinterpret_cast<const float4 *>(init + (size_t)q * N + n);
        }
#pragma unroll
        for (int k = 0; k < NH; ++k) {
          const int i = tid + 256 * k, q = i / NV, n = 4 * (i % NV);
          store4_f16(sH + q * LDN + n, hv[k]);
        }
      }
    }
#pragma unroll
    for (int k = 0; k < NX; ++k) {
      const int i = tid + 256 * k, t = i / PV, q = 4 * (i % PV);
      sXT[(q + 0) * LDQ + t] = (_Float16)xv[k].x;
      sXT[(q + 1) * LDQ + t] = (_Float16)xv[k].y;
      sXT[(q + 2) * LDQ + t] = (_Float16)xv[k].z;
      sXT[(q + 3) * LDQ + t] = (_Float16)xv[k].w;
    }
  }
  __syncthreads();
  const float c_last = s_c[Q - 1];

  if (kOut) {
    const int tw = 16 * wave;  // the wave's 16 rows t
    // S = C B^T (tiles of s up to the diagonal), masked and decayed into
    // M[t][s] = S[t][s] 2^(A (c_t - c_s)) dt_s for s <= t
    for (int jt = 0; jt < Q / 16; ++jt) {
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
      if (jt <= wave) {
#pragma unroll
        for (int kk = 0; kk < N / 32; ++kk) {
          const f16x8 a = *reinterpret_cast<const f16x8 *>(sC + (tw + r16) * LDN + 32 * kk + 8 * kq);
          const f16x8 b = *reinterpret_cast<const f16x8 *>(sB + (16 * jt + r16) * LDN + 32 * kk + 8 * kq);
          acc = mma_chunk(a, b, acc);
        }
      }
      const int sc = 16 * jt + r16;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int t = tw + 4 * kq + i;
        const float m = sc <= t ? acc[i] * exp2_fast(a2 * (s_c[t] - s_c[sc])) * s_dt[sc] : 0.f;
        sM[t * LDQ + sc] = (_Float16)m;
      }
    }
    __syncthreads();
    // Y = 2^(A c_t) (C Hinit^T) + M X, then g = (y + D x) silu(z)
    f32x4 y[P / 16];
#pragma unroll
    for (int jp = 0; jp < P / 16; ++jp) y[jp] = f32x4{0.f, 0.f, 0.f, 0.f};
    if (init) {
#pragma unroll
      for (int kk = 0; kk < N / 32; ++kk) {
        const f16x8 a = *reinterpret_cast<const f16x8 *>(sC + (tw + r16) * LDN + 32 * kk + 8 * kq);
#pragma unroll
        for (int jp = 0; jp < P / 16; ++jp) {
          const f16x8 b = *reinterpret_cast<const f16x8 *>(sH + (16 * jp + r16) * LDN + 32 * kk + 8 * kq);
          y[jp] = mma_chunk(a, b, y[jp]);
        }
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float e = exp2_fast(a2 * s_c[tw + 4 * kq + i]);
#pragma unroll
        for (int jp = 0; jp < P / 16; ++jp) y[jp][i] *= e;
      }
    }
#pragma unroll
    for (int kk = 0; kk < Q / 32; ++kk) {
      const f16x8 a = *reinterpret_cast<const f16x8 *>(sM + (tw + r16) * LDQ + 32 * kk + 8 * kq);
#pragma unroll
      for (int jp = 0; jp < P / 16; ++jp) {
        const f16x8 b = *reinterpret_cast<const f16x8 *>(sXT + (16 * jp + r16) * LDQ + 32 * kk + 8 * kq);
        y[jp] = mma_chunk(a, b, y[jp]);
      }
    }
    const float Dh = p.D[h];
    float xo[4][P / 16], zo[4][P / 16];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const size_t row = (size_t)(t0 + min(tw + 4 * kq + i, nt - 1));
#pragma unroll
      for (int jp = 0; jp < P / 16; ++jp) {
        const int col = h * P + 16 * jp + r16;
        xo[i][jp] = p.xbc[row * p.conv_n + col];
        zo[i][jp] = p.zxd[row * p.ldz + col];
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int t = tw + 4 * kq + i;
      if (t < nt) {
        const size_t row = (size_t)(t0 + t);
#pragma unroll
        for (int jp = 0; jp < P / 16; ++jp)
          p.g[row * di + h * P + 16 * jp + r16] = fmaf(Dh, xo[i][jp], y[jp][i]) * silu_fast(zo[i][jp]);
      }
    }
    if (!last) return;
    __syncthreads();  // M and Hinit are read; their space takes w B
  }

  // h_end = 2^(A c_last) h_init + X^T diag(w) B, w_s = dt_s 2^(A (c_last - c_s)): w B staged
  // transposed from the fp32 rows, then 16 x 16 tiles of [P][N] over the waves
  {
    float4 bv[NBC];
#pragma unroll
    for (int k = 0; k < NBC; ++k) {
      const int i = tid + 256 * k, t = i / NV, n = 4 * (i % NV);
      bv[k] = t < nt ? *reinterpret_cast<const float4 *>(xbc + (size_t)t * p.conv_n + di + grp * N + n)
                     : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int k = 0; k < NBC; ++k) {
      const int i = tid + 256 * k, t = i / NV, n = 4 * (i % NV);
      const float w = s_dt[t] * exp2_fast(a2 * (c_last - s_c[t]));
      sBT[(n + 0) * LDQ + t] = (_Float16)(bv[k].x * w);
      sBT[(n + 1) * LDQ + t] = (_Float16)(bv[k].y * w);
      sBT[(n + 2) * LDQ + t] = (_Float16)(bv[k].z * w);
      sBT[(n + 3) * LDQ + t] = (_Float16)(bv[k].w * w);
    }
  }
  __syncthreads();
  float *dst = kOut ? p.ssm + ((size_t)ch.x * p.H + h) * tile : p.hloc + ((size_t)j * p.H + h) * tile;
  const float e_last = exp2_fast(a2 * c_last);
  constexpr int TPW = (P / 16) * (N / 16) / 4;  // 16 x 16 tiles per wave
  static_assert((P / 16) * (N / 16) % 4 == 0, "tiles split evenly over the waves");
  float iv[TPW][4];
#pragma unroll
  for (int r = 0; r < TPW; ++r) {
    const int q = wave + 4 * r, tp = q / (N / 16), tn = q % (N / 16);
#pragma unroll
    for (int i = 0; i < 4; ++i)
      iv[r][i] = init ? init[(size_t)(16 * tp + 4 * kq + i) * N + 16 * tn + r16] : 0.f;
  }
#pragma unroll
  for (int r = 0; r < TPW; ++r) {
    const int q = wave + 4 * r, tp = q / (N / 16), tn = q % (N / 16);
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < Q / 32; ++kk) {
      const f16x8 a = *reinterpret_cast<const f16x8 *>(sXT + (16 * tp + r16) * LDQ + 32 * kk + 8 * kq);
      const f16x8 b = *reinterpret_cast<const f16x8 *>(sBT + (16 * tn + r16) * LDQ + 32 * kk + 8 * kq);
      acc = mma_chunk(a, b, acc);
    }
    const int n = 16 * tn + r16;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      dst[(size_t)(16 * tp + 4 * kq + i) * N + n] = fmaf(e_last, iv[r][i], acc[i]);
    }
  }
  if (!kOut || !p.update_conv) return;
  // The sequence's last K-1 conv inputs (old conv state followed by this call's rows), spread
  // over the threads of the sequence's last-chunk blocks.
  const int seq = ch.x, K1 = p.K - 1;
  const int t0s = p.cu[seq], len = p.cu[seq + 1] - t0s;
  for (int cc = blockIdx.x * 256 + tid; cc < p.conv_n; cc += gridDim.x * 256) {
    float nv[3];
#pragma unroll
    for (int q = 0; q < 3; ++q) {
      if (q >= K1) continue;
      const int pos = len + q;
      nv[q] = pos < K1 ? (p.fresh ? 0.f : p.conv[((size_t)seq * K1 + pos) * p.conv_n + cc])
                       : p.zxd[(size_t)(t0s + pos - K1) * p.ldz + p.conv_col + cc];
    }
#pragma unroll
    for (int q = 0; q < 3; ++q)
      if (q < K1) p.conv[((size_t)seq * K1 + q) * p.conv_n + cc] = nv[q];
  }
}

bool m2_args_ok(const M2ScanArgs &a) {
  return a.zxd && a.xbc && a.dt_b && a.A2 && a.D && a.ssm && a.g && a.H > 0 && a.G > 0 &&
         a.H % a.G == 0 && a.P > 0 && a.P % kM2Rows == 0 && a.di == a.H * a.P &&
         (a.N == 32 || a.N == 64 || a.N == 128 || a.N == 256) &&
         a.conv_n == a.di + 2 * a.G * a.N && a.dt_col >= 0 && a.ldz >= a.dt_col + a.H;
}

template <bool kOut, int P>
hipError_t ssd_launch_p(const M2ScanArgs &a, int n_chunks, hipStream_t s) {
  const dim3 grid(a.H, n_chunks);
  switch (a.N) {
    case 32: LL_LAUNCH((k_m2_ssd<kOut, 32, P>), grid, dim3(256), 0, s, a); break;
    case 64: LL_LAUNCH((k_m2_ssd<kOut, 64, P>), grid, dim3(256), 0, s, a); break;
    case 128: LL_LAUNCH((k_m2_ssd<kOut, 128, P>), grid, dim3(256), 0, s, a); break;
    case 256: LL_LAUNCH((k_m2_ssd<kOut, 256, P>), grid, dim3(256), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <bool kOut>
hipError_t m2_launch(const M2ScanArgs &a, int n_chunks, hipStream_t s) {
  if (a.mfma && a.chunks) {
    if (!mamba2_ssd_ok(a.P, a.N)) return hipErrorInvalidValue;
    return a.P == 32 ? ssd_launch_p<kOut, 32>(a, n_chunks, s) : ssd_launch_p<kOut, 64>(a, n_chunks, s);
  }
  const dim3 grid(a.H * (a.P / kM2Rows), n_chunks);
  switch (a.N) {
    case 32: LL_LAUNCH((k_m2_scan<kOut, 2>), grid, dim3(kM2Threads), 0, s, a); break;
    case 64: LL_LAUNCH((k_m2_scan<kOut, 4>), grid, dim3(kM2Threads), 0, s, a); break;
    case 128: LL_LAUNCH((k_m2_scan<kOut, 8>), grid, dim3(kM2Threads), 0, s, a); break;
    case 256: LL_LAUNCH((k_m2_scan<kOut, 16>), grid, dim3(kM2Threads), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

bool mamba2_ssd_ok(int head_dim, int d_state) {
  return (head_dim == 32 || head_dim == 64) &&
         (d_state == 32 || d_state == 64 || d_state == 128 || d_state == 256);
}

int mamba2_chunk_len(int total, int n_heads, int head_dim) {
  const long blocks_per_chunk = (long)n_heads * (head_dim / kM2Rows);
  long len = (total * blocks_per_chunk + kM2TargetBlocks - 1) / kM2TargetBlocks;
  len = (len + kM2Stage - 1) / kM2Stage * kM2Stage;
  return (int)std::max<long>(len, kM2Stage);
}

int mamba2_max_chunks(int max_total, int max_batch, int n_heads, int head_dim) {
  const long a = (max_total + kM2Stage - 1) / kM2Stage;
  const long b = (long)kM2TargetBlocks / std::max(1, n_heads * (head_dim / kM2Rows)) + 1;
  return (int)(std::min(a, b) + max_batch);
}

hipError_t launch_m2_scan_chunks(const M2ScanArgs &a, int n_chunks, hipStream_t s) {
  if (n_chunks <= 0) return hipSuccess;
  if (!m2_args_ok(a) || !a.chunks || !a.hloc || !a.dtsum) return hipErrorInvalidValue;
  return m2_launch<false>(a, n_chunks, s);
}

hipError_t launch_m2_scan_carry(const M2ScanArgs &a, int batch, hipStream_t s) {
  if (batch <= 0) return hipSuccess;
  if (!m2_args_ok(a) || !a.seq_chunk0 || !a.hloc || !a.dtsum) return hipErrorInvalidValue;
  const size_t elems = (size_t)a.H * a.P * a.N;
  LL_LAUNCH(k_m2_carry, dim3((unsigned)((elems + 255) / 256), batch), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_m2_scan_out(const M2ScanArgs &a, int n_chunks, hipStream_t s) {
  if (n_chunks <= 0) return hipSuccess;
  if (!m2_args_ok(a) || (a.chunks && !a.cu) || (a.carry == 2 && !a.hloc) || a.carry < 0 ||
      a.carry > 2 || (a.carry == 0 && !a.fresh) ||
      (a.update_conv && (!a.conv || !a.cu || a.K < 1 || a.K > 4 || a.conv_col < 0)))
    return hipErrorInvalidValue;
  return m2_launch<true>(a, n_chunks, s);
}

}  // namespace ll
