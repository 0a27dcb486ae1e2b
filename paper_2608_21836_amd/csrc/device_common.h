// Device helpers shared by the gfx950 kernels: element types, 16-byte MFMA operand
// fragments, conversions and wave reductions.
#pragma once
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernels.h"

// Launch through the thread's LaunchTimer when one is installed, else a plain launch.
#define LL_LAUNCH(kernel, grid, block, shmem, stream, ...)                                    \
  do {                                                                                      \
    hipEvent_t ll_ev0_ = nullptr, ll_ev1_ = nullptr;                                        \
    if (::ll::g_launch_timer && ::ll::g_launch_timer->next(&ll_ev0_, &ll_ev1_))             \
      hipExtLaunchKernelGGL(kernel, grid, block, shmem, stream, ll_ev0_, ll_ev1_, 0,          \
                            __VA_ARGS__);                                                   \
    else                                                                                    \
      hipLaunchKernelGGL(kernel, grid, block, shmem, stream, __VA_ARGS__);                  \
  } while (0)

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16;
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(1))) void global_void_t;

// global_load_lds_dwordx4: lane l's 16 bytes from `src` (its own address) land at byte
// 16 l of the 1 KiB LDS tile; the wave's LDS base goes through M0, so `lds_tile` must be
// wave-uniform.  Completion is counted by vmcnt.
__device__ __forceinline__ void load_tile_to_lds(const void *src, void *lds_tile) {
  __builtin_amdgcn_global_load_lds((global_void_t *)src, (lds_void_t *)lds_tile, 16, 0, 0);
}

// One lane's 16-byte share of a 16-row MFMA operand tile.
//   bf16: 8 elements, the tile spans 32 along the contraction axis (v_mfma_f32_16x16x32_bf16)
//   fp32: 4 elements, the tile spans 16 along the contraction axis (4 x v_mfma_f32_16x16x4_f32)
// Lane l covers row (l % 16) and contraction indices EPL * (l / 16) + e, e < EPL.
template <typename T> struct Frag;
template <> struct Frag<bf16> {
  typedef bf16x8 type;
  static constexpr int EPL = 8;
};
template <> struct Frag<float> {
  typedef f32x4 type;
  static constexpr int EPL = 4;
};
//   fp16: as bf16 (v_mfma_f32_16x16x32_f16)
template <> struct Frag<f16> {
  typedef f16x8 type;
  static constexpr int EPL = 8;
};

// 16x16 output tile += A-fragment x B-fragment over one 16-byte-per-lane chunk.
// Output layout: lane l holds rows 4*(l/16) + r (r < 4) of column l % 16.
__device__ __forceinline__ f32x4 mma_chunk(const bf16x8 &a, const bf16x8 &b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mma_chunk(const f16x8 &a, const f16x8 &b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mma_chunk(const f32x4 &a, const f32x4 &b, f32x4 c) {
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[0], b[0], c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[1], b[1], c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[2], b[2], c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[3], b[3], c, 0, 0, 0);
  return c;
}

// 32x32 output tile += A x B over 16 contraction indices (v_mfma_f32_32x32x16_bf16).
// A lane l: row l % 32, contraction 8 (l / 32) + e; B lane l: column l % 32, same contraction
// indices.  Output: lane l holds column l % 32, rows 8 (i / 4) + 4 (l / 32) + i % 4, i < 16.
__device__ __forceinline__ f32x16 mma32(const bf16x8 &a, const bf16x8 &b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x16 mma32(const f16x8 &a, const f16x8 &b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16 x) { return static_cast<float>(x); }
__device__ __forceinline__ float to_f32(f16 x) { return static_cast<float>(x); }

template <typename T> __device__ __forceinline__ T from_f32(float x);
template <> __device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <> __device__ __forceinline__ bf16 from_f32<bf16>(float x) { return static_cast<bf16>(x); }
template <> __device__ __forceinline__ f16 from_f32<f16>(float x) { return static_cast<f16>(x); }

template <typename F> __device__ __forceinline__ F frag_zero() {
  F z;
#pragma unroll
  for (int i = 0; i < (int)(sizeof(F) / sizeof(z[0])); ++i) z[i] = 0;
  return z;
}

template <typename F> __device__ __forceinline__ F load_frag(const void *p) {
  return *reinterpret_cast<const F *>(p);
}

// Streaming (read-once) 16-byte load that should not displace reused data in the caches.
template <typename F> __device__ __forceinline__ F load_frag_stream(const void *p) {
  return __builtin_nontemporal_load(reinterpret_cast<const F *>(p));
}

// Cross-lane sums on the DPP / swizzle paths (no LDS-crossbar permutes).
//   dpp_add<CTRL>(v): v + v from the lane the DPP control selects (all lanes enabled)
template <int CTRL> __device__ __forceinline__ float dpp_add(float v) {
  const int o = __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xf, 0xf, false);
  return v + __builtin_bit_cast(float, o);
}
constexpr int kDppXor1 = 0xB1;        // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4E;        // quad_perm [2,3,0,1]
constexpr int kDppHalfMirror = 0x141; // lane i <-> 7 - i within 8 (pairs the two quads)
constexpr int kDppMirror = 0x140;     // lane i <-> 15 - i within 16 (pairs the two halves)
constexpr int kDppRor8 = 0x128;       // lane i <- (i + 8) mod 16 within 16
__device__ __forceinline__ float swizzle_xor16_add(float v) {
  // bit-mask swizzle over 32 lanes: and 0x1f, or 0, xor 0x10
  const int o = __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, v), (0x10 << 10) | 0x1f);
  return v + __builtin_bit_cast(float, o);
}
// Sum over aligned groups of W lanes (W = 8, 16 or 32); every lane of a group gets the sum.
template <int W> __device__ __forceinline__ float group_sum(float v) {
  static_assert(W == 8 || W == 16 || W == 32, "group of 8, 16 or 32 lanes");
  v = dpp_add<kDppXor1>(v);
  v = dpp_add<kDppXor2>(v);
  v = dpp_add<kDppHalfMirror>(v);
  if constexpr (W >= 16) v = dpp_add<kDppMirror>(v);
  if constexpr (W >= 32) v = swizzle_xor16_add(v);
  return v;
}
// Sum over the lanes of one 32-lane half that share (lane % W), W = 8, 16 or 32; every such
// lane gets the sum.
template <int W> __device__ __forceinline__ float stride_sum32(float v) {
  static_assert(W == 8 || W == 16 || W == 32, "stride of 8, 16 or 32 lanes");
  if constexpr (W <= 8) v = dpp_add<kDppRor8>(v);
  if constexpr (W <= 16) v = swizzle_xor16_add(v);
  return v;
}

template <int CTRL> __device__ __forceinline__ float dpp_max(float v) {
  const int o = __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xf, 0xf, false);
  return fmaxf(v, __builtin_bit_cast(float, o));
}
__device__ __forceinline__ float lane_read(float v, int lane) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), lane));
}
// Whole-wave sum / maximum (every lane active): DPP and swizzle within each 32-lane half, then
// the two halves' results read from lanes 0 and 32.
__device__ __forceinline__ float wave_sum(float v) {
  v = group_sum<32>(v);
  return lane_read(v, 0) + lane_read(v, 32);
}
__device__ __forceinline__ float wave_max(float v) {
  v = dpp_max<kDppXor1>(v);
  v = dpp_max<kDppXor2>(v);
  v = dpp_max<kDppHalfMirror>(v);
  v = dpp_max<kDppMirror>(v);
  const int o = __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, v), (0x10 << 10) | 0x1f);
  v = fmaxf(v, __builtin_bit_cast(float, o));
  return fmaxf(lane_read(v, 0), lane_read(v, 32));
}

__device__ __forceinline__ float silu_f(float z) { return z / (1.0f + __expf(-z)); }

constexpr float kLog2e = 1.4426950408889634f;

// softplus(x) = max(x, 0) + log1p(exp(-|x|)), with log1p(e) = log(1 + e) * e / ((1 + e) - 1)
// (exact rounding compensation of 1 + e; e itself when 1 + e rounds to 1).
__device__ __forceinline__ float softplus_f(float x) {
  const float e = __expf(-fabsf(x));
  const float u = 1.f + e;
  const float l = u == 1.f ? e : __logf(u) * __fdividef(e, u - 1.f);
  return fmaxf(x, 0.f) + l;
}
// 2^x with the hardware instruction (results below the normal range flush to zero).
__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float silu_fast(float z) { return __fdividef(z, 1.f + __expf(-z)); }
__device__ __forceinline__ float sigmoid_f(float z) { return 1.0f / (1.0f + __expf(-z)); }
// tanh-approximated GELU, x/2 (1 + tanh(y)) with y = sqrt(2/pi) (x + 0.044715 x^3), written
// as x * sigmoid(2 y) (the same function: 1 + tanh(y) = 2 sigmoid(2 y)).
__device__ __forceinline__ float gelu_tanh_f(float x) {
  const float y2 = 1.5957691216057308f * fmaf(0.044715f * x, x * x, x);
  return x / (1.0f + __expf(-y2));
}

// Merge of split-K attention partials, in split order: sum_s w_s o_s / sum_s w_s l_s, where
// w_s = 2^(m_s - max_s m_s) (log-sum-exp rescaling of each split's unnormalised output o_s and
// sum l_s).  `po` points at split 0's output element, `stride` floats between splits; w and l
// usually sit in LDS.
// The same merge for at most MAXS splits in one pass, all loads issued up front: `ml` holds
// (m_s, l_s) pairs; slots past ns load split ns - 1 again and get weight 0.  Used where the
// split count is small, so the merge costs one memory round trip.
template <int MAXS>
__device__ __forceinline__ float merge_splits_direct(const float *ml, const float *po,
                                                     size_t stride, int ns) {
  float m[MAXS], l[MAXS], o[MAXS];
#pragma unroll
  for (int sp = 0; sp < MAXS; ++sp) {
    const int s = min(sp, ns - 1);
    m[sp] = ml[2 * s];
    l[sp] = ml[2 * s + 1];
    o[sp] = po[s * stride];
  }
  float mx = -INFINITY;
#pragma unroll
  for (int sp = 0; sp < MAXS; ++sp) mx = fmaxf(mx, m[sp]);
  float num = 0.f, den = 0.f;
#pragma unroll
  for (int sp = 0; sp < MAXS; ++sp) {
    const float w = sp < ns ? exp2f(m[sp] - mx) : 0.f;
    num += w * o[sp];
    den += w * l[sp];
  }
  return num / den;
}

__device__ __forceinline__ float merge_splits(const float *po, size_t stride, const float *w,
                                              const float *l, int ns) {
  float num = 0.f, den = 0.f;
#pragma unroll 8
  for (int sp = 0; sp < ns; ++sp) {
    num += w[sp] * po[sp * stride];
    den += w[sp] * l[sp];
  }
  return num / den;
}
