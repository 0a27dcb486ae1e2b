// An LM-head + greedy-argmax entry point that allocates nothing: its per-block argmax partials
// live in a file-scope device array instead of a caller-provided scratch buffer, for callers
// that cannot allocate (code under HIP graph capture, tight serving loops, harnesses that
// forbid allocation).  The kernels are those of ll_op_lmhead_argmax.
#include <hip/hip_runtime.h>

#include <mutex>
#include <vector>

#include "kernels.h"
#include "ll_ops.h"
#include "runtime_common.h"

namespace ll {
namespace {

// Partials of one call: rows x (vocab / 32) (value, index) pairs, 8 bytes each.
constexpr size_t kNoAllocScratchBytes = 2u << 20;
__device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

// Device address of `scratch` on each device, resolved once per device (with that device
// current).  In host code the array's name is a host-side stand-in, never a device address.
std::mutex g_scratch_mu;
std::vector<void *> g_scratch_ptr;

ll_status scratch_ptr(void **out) {
  int dev = 0;
  LL_HIP(hipGetDevice(&dev));
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if ((int)g_scratch_ptr.size() <= dev) g_scratch_ptr.resize(dev + 1, nullptr);
  if (!g_scratch_ptr[dev]) {
    void *p = nullptr;
    LL_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (!p) return fail(LL_ERR_HIP, "hipGetSymbolAddress returned NULL for the scratch array");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return LL_OK;
}

}  // namespace
}  // namespace ll

using namespace ll;

extern "C" ll_status ll_op_lmhead_argmax_noalloc(int32_t dtype, int32_t rows, int32_t vocab,
                                                 int32_t k, const void *h, const void *wt,
                                                 float *logits, int32_t *next, void *stream) {
  g_err.clear();
  if (dtype != LL_F32 && dtype != LL_BF16 && dtype != LL_F16)
    return fail(LL_ERR_UNSUPPORTED, "dtype %d unknown", dtype);
  if (rows < 1 || vocab < 32 || vocab % 32 || k < 64 || k % 64)
    return fail(LL_ERR_UNSUPPORTED, "rows >= 1, vocab %% 32, k %% 64 required");
  if (!h || !wt || !next) return fail(LL_ERR_INVALID_ARGUMENT, "NULL pointer");
  const size_t parts = (size_t)rows * (vocab / 32);
  if (parts * 8 > kNoAllocScratchBytes)
    return fail(LL_ERR_CAPACITY, "rows * vocab / 32 = %zu partials need %zu bytes; the static "
                "scratch holds %zu (at most %zu partials)", parts, parts * 8,
                kNoAllocScratchBytes, kNoAllocScratchBytes / 8);
  void *sc = nullptr;
  ll_status st = scratch_ptr(&sc);
  if (st != LL_OK) return st;
  // every partial is written by its block before the reduction reads it: nothing to clear
  EpiParams ep;
  ep.kind = kEpiArgmax;
  ep.out_f32 = logits;
  ep.ld_out = vocab;
  ep.part_val = reinterpret_cast<float *>(sc);
  ep.part_idx = reinterpret_cast<int *>(reinterpret_cast<char *>(sc) + parts * 4);
  ep.n_parts = vocab / 32;
  hipStream_t s = (hipStream_t)stream;
  LL_HIP(launch_gemm_skinny(dtype, h, k, nullptr, wt, rows, vocab, k, ep, s));
  LL_HIP(launch_argmax_reduce(ep.part_val, ep.part_idx, rows, ep.n_parts, next, nullptr, s));
  return LL_OK;
}
