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
                                                    int di, int K, int act, T *__restrict__ u) {
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
  u[(size_t)r * di + c] = from_f32<T>(act ? silu_f(acc) : acc);
}

// Passes 1 (kOut = false) and 3 (kOut = true) of the scan; one wave per (channel block, chunk).
// The chunk is walked in stages of kScanStage steps: a stage's (dt_low | B | C) rows go to LDS,
// re-laid as [dt_low zero-padded to R16 = 16 NR | B | C] so every step reads its row as float4s
// (all in flight at once, the same words for every lane), and its u (and z) values go to
// registers, in one round of loads; the steps then run from there.  The dt projection of the
// lane's channel (R16 rows, zero beyond R) sits in registers.
constexpr int kScanStage = 16;
constexpr int kScanMaxNR = 10;  // dt rank up to 160

template <typename T, bool kOut, int NR>
__global__ __launch_bounds__(kScanChannels) void k_scan(
    ScanArgs p, const float *__restrict__ xdbl, const T *__restrict__ u,
    const float *__restrict__ xz, T *__restrict__ y, float *__restrict__ hloc) {
  constexpr int R16 = 16 * NR, XS = R16 + 2 * kNS, XS4 = XS / 4;
  __shared__ __attribute__((aligned(16))) float s_r[kScanStage][XS];
  const int j = blockIdx.y;
  const int4 ch = p.chunks ? p.chunks[j] : make_int4(j, j, 1, kChunkLast);
  if (!kOut && (ch.w & kChunkLast)) return;  // a sequence's last chunk needs no end state
  const int lane = threadIdx.x, di = p.di, R = p.R;
  const int c = blockIdx.x * kScanChannels + lane;
  float wreg[R16];
#pragma unroll
  for (int r = 0; r < R16; ++r) wreg[r] = p.dtwT[(size_t)r * di + c];
  float a2[kNS], h[kNS];
#pragma unroll
  for (int n = 0; n < kNS; ++n) {
    a2[n] = p.A2[(size_t)n * di + c];
    h[n] = 0.f;
  }
  if (kOut && p.carry == 1) {
    const float4 *sp = reinterpret_cast<const float4 *>(p.ssm + ((size_t)ch.x * di + c) * kNS);
#pragma unroll
    for (int q = 0; q < kNS / 4; ++q) {
      const float4 v = sp[q];
      h[4 * q] = v.x;
      h[4 * q + 1] = v.y;
      h[4 * q + 2] = v.z;
      h[4 * q + 3] = v.w;
    }
  } else if (kOut && p.carry == 2) {
#pragma unroll
    for (int n = 0; n < kNS; ++n) h[n] = hloc[((size_t)j * kNS + n) * di + c];
  }
  const float bias = p.dt_b[c];
  const float Dc = kOut ? p.D[c] : 0.f;
  float dsum = 0.f;
  const int tend = ch.y + ch.z;
  // source column of padded column col: dt_low (col < R), zero (R <= col < R16), B | C after
  constexpr int kCols = (XS + kScanChannels - 1) / kScanChannels;
  for (int t0 = ch.y; t0 < tend; t0 += kScanStage) {
    const int nt = min(kScanStage, tend - t0);
    __syncthreads();  // the previous stage's rows have been read
    {
      float v[kScanStage][kCols];
#pragma unroll
      for (int r = 0; r < kScanStage; ++r)
#pragma unroll
        for (int q = 0; q < kCols; ++q) {
          const int col = lane + q * kScanChannels;
          const int src = col < R16 ? col : col - R16 + R;
          v[r][q] = (r < nt && col < XS && (col < R || col >= R16))
                        ? xdbl[(size_t)(t0 + r) * p.ldx + src] : 0.f;
        }
#pragma unroll
      for (int r = 0; r < kScanStage; ++r)
#pragma unroll
        for (int q = 0; q < kCols; ++q) {
          const int col = lane + q * kScanChannels;
          if (col < XS) s_r[r][col] = v[r][q];
        }
    }
    float uv[kScanStage], zv[kScanStage];
#pragma unroll
    for (int i = 0; i < kScanStage; ++i) {
      uv[i] = i < nt ? to_f32(u[(size_t)(t0 + i) * di + c]) : 0.f;
      zv[i] = (kOut && i < nt) ? xz[(size_t)(t0 + i) * p.ldxz + di + c] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < kScanStage; ++i) {
      if (i < nt) {
        float xr[XS];
        const float4 *x4 = reinterpret_cast<const float4 *>(s_r[i]);
#pragma unroll
        for (int q = 0; q < XS4; ++q) {
          const float4 t4 = x4[q];
          xr[4 * q] = t4.x;
          xr[4 * q + 1] = t4.y;
          xr[4 * q + 2] = t4.z;
          xr[4 * q + 3] = t4.w;
        }
        float acc = bias;
#pragma unroll
        for (int r = 0; r < R16; ++r) acc = fmaf(wreg[r], xr[r], acc);
        const float dt = softplus_f(acc);
        const float du = dt * uv[i];
        float yv = 0.f;
#pragma unroll
        for (int n = 0; n < kNS; ++n) {
          h[n] = fmaf(exp2_fast(dt * a2[n]), h[n], du * xr[R16 + n]);
          if (kOut) yv = fmaf(h[n], xr[R16 + kNS + n], yv);
        }
        if (kOut) {
          yv = fmaf(Dc, uv[i], yv);
          y[(size_t)(t0 + i) * di + c] = from_f32<T>(yv * silu_fast(zv[i]));
        } else {
          dsum += dt;
        }
      }
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
  float4 *sp = reinterpret_cast<float4 *>(p.ssm + ((size_t)seq * di + c) * kNS);
#pragma unroll
  for (int q = 0; q < kNS / 4; ++q) sp[q] = make_float4(h[4 * q], h[4 * q + 1], h[4 * q + 2], h[4 * q + 3]);
  const int K1 = p.K - 1;
  const int t0 = p.cu ? p.cu[seq] : seq;
  const int len = p.cu ? p.cu[seq + 1] - t0 : 1;
  float nv[3];
#pragma unroll
  for (int q = 0; q < 3; ++q) {
    if (q >= K1) continue;
    const int pos = len + q;  // index into (old state ++ new rows)
    nv[q] = pos < K1 ? (p.fresh ? 0.f : p.conv[((size_t)seq * K1 + pos) * di + c])
                     : xz[(size_t)(t0 + pos - K1) * p.ldxz + c];
  }
#pragma unroll
  for (int q = 0; q < 3; ++q)
    if (q < K1) p.conv[((size_t)seq * K1 + q) * di + c] = nv[q];
}

// Pass 2: per (sequence, channel, state), chain the chunk end states into each chunk's incoming
// state (written over hloc), starting from the SSM state (zero when fresh).  Grid (di / 64,
// N, batch); the chunk values are read kCarryStage at a time, all loads in flight together.
constexpr int kCarryStage = 16;

__global__ __launch_bounds__(kScanChannels) void k_scan_carry(ScanArgs p) {
  const int n = blockIdx.y, b = blockIdx.z, di = p.di;
  const int c = blockIdx.x * kScanChannels + threadIdx.x;
  const float a2 = p.A2[(size_t)n * di + c];
  float H = p.fresh ? 0.f : p.ssm[((size_t)b * di + c) * kNS + n];
  const int j0 = p.seq_chunk0[b], j1 = p.seq_chunk0[b + 1];
  for (int jb = j0; jb < j1; jb += kCarryStage) {
    float hl[kCarryStage], S[kCarryStage];
#pragma unroll
    for (int i = 0; i < kCarryStage; ++i) {
      const int j = jb + i;
      const bool ok = j < j1 - 1;  // the last chunk has no end state
      hl[i] = ok ? p.hloc[((size_t)j * kNS + n) * di + c] : 0.f;
      S[i] = ok ? p.dtsum[(size_t)j * di + c] : 0.f;
    }
#pragma unroll
    for (int i = 0; i < kCarryStage; ++i) {
      const int j = jb + i;
      if (j < j1) {
        p.hloc[((size_t)j * kNS + n) * di + c] = H;
        H = fmaf(exp2_fast(a2 * S[i]), H, hl[i]);
      }
    }
  }
}

// Fused decode step; grid (di / 32), 512 threads (8 waves).  x_proj runs on MFMA from the
// repacked (zero-padded) x_proj tiles: each wave takes a range of k-tiles for all NT output
// tiles of 16, issues up to 32 weight tiles and their activation fragments in one round, and
// leaves its partial sums in LDS; the 8 partials are then added per output.  Everything the
// state update reads is loaded at the start, so its latency overlaps the x_proj phase.
constexpr int kSsmThreads = 512;
constexpr int kSsmWaves = kSsmThreads / 64;
constexpr int kSsmChannels = kSsmThreads / 16;  // channels per block (16 lanes each)
constexpr int kSsmPairs = 32;                   // weight tiles per wave per round
constexpr int kOutPre = 6;                      // out_proj tiles per wave requested up front

template <typename T, int NT>
__global__ __launch_bounds__(kSsmThreads) void k_ssm_decode(SsmDecodeArgs p) {
  using F = typename Frag<T>::type;
  constexpr int EPL = Frag<T>::EPL, TK = 4 * EPL, KR = kSsmPairs / NT;
  constexpr int XP = NT * 16;  // padded x_proj outputs
  __shared__ float s_part[kSsmWaves][kSsmDecodeMaxRows][XP];
  __shared__ float s_x[kSsmDecodeMaxRows][XP];
  __shared__ __attribute__((aligned(16))) T s_y[kSsmDecodeMaxRows][kSsmChannels];
  const int rows = p.rows, di = p.di, R = p.R, X = R + 2 * kNS;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // state-update operands of this thread: channel c, state n
  const int n = tid & 15;
  const int c = blockIdx.x * kSsmChannels + (tid >> 4);
  const T *u = reinterpret_cast<const T *>(p.u);
  float hs[kSsmDecodeMaxRows], zs[kSsmDecodeMaxRows], us[kSsmDecodeMaxRows], wr[4];
#pragma unroll
  for (int b = 0; b < kSsmDecodeMaxRows; ++b) {
    hs[b] = b < rows ? p.ssm[((size_t)b * di + c) * kNS + n] : 0.f;
    zs[b] = b < rows ? p.z[(size_t)b * p.ldz + c] : 0.f;
    us[b] = b < rows ? to_f32(u[(size_t)b * di + c]) : 0.f;
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) wr[i] = n + 16 * i < R ? p.dtwT[(size_t)(n + 16 * i) * di + c] : 0.f;
  const float a2 = p.A2[(size_t)n * di + c], bias = p.dt_b[c], Dc = p.D[c];

  // out_proj weight tiles of this block's channels (fused out_proj): the first OP of this
  // wave's output tiles are requested now, the rest when used.
  constexpr int KTO = kSsmChannels / TK;  // k-tiles of this block's 32 channels (1 or 2)
  const uint8_t *wo = reinterpret_cast<const uint8_t *>(p.wout) + (size_t)lane * 16;
  const int nbo = p.d / 16, kbo_n = di / TK;
  constexpr int OP = sizeof(T) == 2 ? kOutPre : kOutPre / 3;  // fp32 tiles take 2 fragments
  F wop[OP][KTO];
  if (p.wout) {
#pragma unroll
    for (int i = 0; i < OP; ++i)
#pragma unroll
      for (int q = 0; q < KTO; ++q) {
        const int nb = wave + kSsmWaves * i;
        wop[i][q] = nb < nbo ? load_frag<F>(wo + ((size_t)nb * kbo_n + blockIdx.x * KTO + q) * 1024)
                             : frag_zero<F>();
      }
  }

  // x_proj partial sums over this wave's k-tiles: acc[t] = u rows x weight tile t.
  const int kb_n = di / TK;
  const int kb0 = wave * kb_n / kSsmWaves, kb1 = (wave + 1) * kb_n / kSsmWaves;
  const uint8_t *wt = reinterpret_cast<const uint8_t *>(p.wx) + (size_t)lane * 16;
  const int arow = lane & 15;
  const T *ap = u + (size_t)(arow < rows ? arow : 0) * di + (lane >> 4) * EPL;
  const F fz = frag_zero<F>();
  f32x4 acc[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int kr = kb0; kr < kb1; kr += KR) {
    F wf[KR][NT], af[KR];
#pragma unroll
    for (int q = 0; q < KR; ++q) {
      const int kb = kr + q;
      af[q] = (kb < kb1 && arow < rows) ? load_frag<F>(ap + (size_t)kb * TK) : fz;
#pragma unroll
      for (int t = 0; t < NT; ++t)
        wf[q][t] = kb < kb1 ? load_frag<F>(wt + ((size_t)t * kb_n + kb) * 1024) : fz;
    }
#pragma unroll
    for (int q = 0; q < KR; ++q)
#pragma unroll
      for (int t = 0; t < NT; ++t) acc[t] = mma_chunk(af[q], wf[q][t], acc[t]);
  }
  // lane l holds rows 4 (l / 16) + r of output column l % 16 of each tile; rows < 4 only
  if (lane < 16) {
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int r = 0; r < kSsmDecodeMaxRows; ++r) s_part[wave][r][t * 16 + lane] = acc[t][r];
  }
  __syncthreads();
  for (int i = tid; i < rows * XP; i += kSsmThreads) {
    const int b = i / XP, o = i % XP;
    float v = 0.f;
#pragma unroll
    for (int w = 0; w < kSsmWaves; ++w) v += s_part[w][b][o];
    s_x[b][o] = v;
  }
  __syncthreads();

  // State update: 16 lanes per channel, one state each.
  T *y = reinterpret_cast<T *>(p.y);
#pragma unroll
  for (int b = 0; b < kSsmDecodeMaxRows; ++b) {
    if (b >= rows) continue;
    const float *xr = s_x[b];
    float acc1 = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (n + 16 * i < R) acc1 = fmaf(wr[i], xr[n + 16 * i], acc1);
    for (int r = n + 64; r < R; r += 16) acc1 = fmaf(p.dtwT[(size_t)r * di + c], xr[r], acc1);
    acc1 = group_sum<16>(acc1);
    const float dt = softplus_f(acc1 + bias);
    const float h = fmaf(exp2_fast(dt * a2), hs[b], dt * us[b] * xr[R + n]);
    p.ssm[((size_t)b * di + c) * kNS + n] = h;
    const float ys = group_sum<16>(h * xr[R + kNS + n]);
    if (n == 0) {
      const T yv = from_f32<T>(fmaf(Dc, us[b], ys) * silu_fast(zs[b]));
      if (p.wout) s_y[b][tid >> 4] = yv;
      else y[(size_t)b * di + c] = yv;
    }
  }
  if (!p.wout) return;

  // out_proj of this block's 32 channels (one 32-wide k-range of the repacked out_proj) for
  // every output column, added to the residual rows with fp32 atomics (the order of the
  // blocks' additions is not fixed).
  __syncthreads();
  {
    F af[KTO];
#pragma unroll
    for (int q = 0; q < KTO; ++q)
      af[q] = arow < rows ? *reinterpret_cast<const F *>(&s_y[arow][q * TK + (lane >> 4) * EPL]) : fz;
    auto emit = [&](int nb, const f32x4 &o4) {
      if (lane < 16) {
#pragma unroll
        for (int r = 0; r < kSsmDecodeMaxRows; ++r)
          if (r < rows) unsafeAtomicAdd(p.x + (size_t)r * p.ldx + nb * 16 + lane, o4[r]);
      }
    };
#pragma unroll
    for (int i = 0; i < OP; ++i) {
      const int nb = wave + kSsmWaves * i;
      if (nb < nbo) {
        f32x4 o4 = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int q = 0; q < KTO; ++q) o4 = mma_chunk(af[q], wop[i][q], o4);
        emit(nb, o4);
      }
    }
    for (int nb = wave + kSsmWaves * OP; nb < nbo; nb += kSsmWaves) {
      f32x4 o4 = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int q = 0; q < KTO; ++q)
        o4 = mma_chunk(af[q], load_frag<F>(wo + ((size_t)nb * kbo_n + blockIdx.x * KTO + q) * 1024), o4);
      emit(nb, o4);
    }
  }
  (void)X;
}

// dst[j][i] = f(src[i][j]) for j < cols, and 0 for cols <= j < cols_pad.
__global__ __launch_bounds__(256) void k_transpose_f32(const float *__restrict__ src, int rows,
                                                       int cols, int cols_pad,
                                                       float *__restrict__ dst, int neg_exp,
                                                       float scale) {
  const long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (long)rows * cols_pad) return;
  const int i = (int)(idx / cols_pad), j = (int)(idx - (long)i * cols_pad);
  float v = 0.f;
  if (j < cols) {
    v = src[(size_t)i * cols + j];
    if (neg_exp) v = -expf(v);
    v *= scale;
  }
  dst[(size_t)j * rows + i] = v;
}

template <typename T, int NR>
hipError_t scan_launch_nr(bool out, const ScanArgs &a, int n_chunks, hipStream_t s) {
  const dim3 grid(a.di / kScanChannels, n_chunks);
  const float *xd = a.xdbl;
  const T *u = reinterpret_cast<const T *>(a.u);
  T *y = reinterpret_cast<T *>(a.y);
  if (out)
    LL_LAUNCH((k_scan<T, true, NR>), grid, dim3(kScanChannels), 0, s, a, xd, u, a.xz, y, a.hloc);
  else
    LL_LAUNCH((k_scan<T, false, NR>), grid, dim3(kScanChannels), 0, s, a, xd, u, a.xz, y, a.hloc);
  return hipGetLastError();
}

template <typename T>
hipError_t scan_launch(bool out, const ScanArgs &a, int n_chunks, hipStream_t s) {
  switch ((a.R + 15) / 16) {
    case 1: return scan_launch_nr<T, 1>(out, a, n_chunks, s);
    case 2: return scan_launch_nr<T, 2>(out, a, n_chunks, s);
    case 3: return scan_launch_nr<T, 3>(out, a, n_chunks, s);
    case 4: return scan_launch_nr<T, 4>(out, a, n_chunks, s);
    case 5: return scan_launch_nr<T, 5>(out, a, n_chunks, s);
    case 6: return scan_launch_nr<T, 6>(out, a, n_chunks, s);
    case 7: return scan_launch_nr<T, 7>(out, a, n_chunks, s);
    case 8: return scan_launch_nr<T, 8>(out, a, n_chunks, s);
    case 9: return scan_launch_nr<T, 9>(out, a, n_chunks, s);
    case 10: return scan_launch_nr<T, 10>(out, a, n_chunks, s);
  }
  return hipErrorInvalidValue;
}

bool scan_args_ok(const ScanArgs &a) {
  return a.xdbl && a.u && a.xz && a.dtwT && a.dt_b && a.A2 && a.D && a.ssm && a.conv && a.y &&
         a.N == kNS && a.K >= 1 && a.K <= 4 && a.R >= 1 && a.R <= 16 * kScanMaxNR && a.di > 0 &&
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
                             const float *b, int rows, int di, int K, void *u, hipStream_t s,
                             int act) {
  if (rows <= 0) return hipSuccess;
  if (!xz || !w || !b || !u || K < 1 || K > 4 || (!fresh && !conv_state) ||
      ((row_seq == nullptr) != (cu == nullptr)))
    return hipErrorInvalidValue;
  const long n = (long)rows * di;
  const dim3 grid((unsigned)((n + 255) / 256));
  if (dtype == kF32)
    LL_LAUNCH(k_mamba_conv<float>, grid, dim3(256), 0, s, xz, ldxz, row_seq, cu, conv_state,
              fresh, w, b, rows, di, K, act, reinterpret_cast<float *>(u));
  else
    LL_LAUNCH(k_mamba_conv<bf16>, grid, dim3(256), 0, s, xz, ldxz, row_seq, cu, conv_state,
              fresh, w, b, rows, di, K, act, reinterpret_cast<bf16 *>(u));
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
  LL_LAUNCH(k_scan_carry, dim3(a.di / kScanChannels, kNS, batch), dim3(kScanChannels), 0, s, a);
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

hipError_t launch_ssm_decode(int dtype, const SsmDecodeArgs &a, hipStream_t s) {
  if (a.rows <= 0) return hipSuccess;
  const int X = a.R + 2 * kNS;
  if (!a.u || !a.z || a.ldz < a.di || !a.wx || !a.dtwT || !a.dt_b || !a.A2 || !a.D || !a.ssm ||
      a.rows > kSsmDecodeMaxRows || a.N != kNS || a.R < 1 || X > kSsmDecodeMaxX || a.di <= 0 ||
      a.di % kScanChannels != 0)
    return hipErrorInvalidValue;
  if (a.wout ? (!a.x || a.d <= 0 || a.d % 16 != 0 || a.ldx < a.d) : !a.y)
    return hipErrorInvalidValue;
  const dim3 grid(a.di / kSsmChannels);
#define LL_SSM(NT)                                                                         \
  do {                                                                                     \
    if (dtype == kF32) LL_LAUNCH((k_ssm_decode<float, NT>), grid, dim3(kSsmThreads), 0, s, a); \
    else LL_LAUNCH((k_ssm_decode<bf16, NT>), grid, dim3(kSsmThreads), 0, s, a);              \
  } while (0)
  if (X <= 48) LL_SSM(3);
  else if (X <= 80) LL_SSM(5);
  else LL_SSM(8);
#undef LL_SSM
  return hipGetLastError();
}

hipError_t launch_transpose_f32(const float *src, int rows, int cols, int cols_pad, float *dst,
                                int neg_exp, float scale, hipStream_t s) {
  const long n = (long)rows * cols_pad;
  if (n <= 0) return hipSuccess;
  if (cols_pad < cols) return hipErrorInvalidValue;
  LL_LAUNCH(k_transpose_f32, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, src, rows, cols,
            cols_pad, dst, neg_exp, scale);
  return hipGetLastError();
}

}  // namespace ll
