// Host-side helpers shared by the C-ABI translation units: thread-local error text, status
// helpers, workspace alignment and the per-launch timer behind the kernel-timing calls.
#pragma once
#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdio>
#include <string>
#include <vector>

#include "kernels.h"
#include "ll.h"

namespace ll {

// Text of the last failure on this thread (ll_last_error).
extern thread_local std::string g_err;

inline ll_status fail(ll_status st, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

#define LL_HIP(expr)                                                                  \
  do {                                                                                \
    hipError_t e_ = (expr);                                                           \
    if (e_ != hipSuccess)                                                             \
      return ::ll::fail(LL_ERR_HIP, "%s failed: %s", #expr, hipGetErrorString(e_));   \
  } while (0)

constexpr size_t kAlign = 256;
// Gap after every workspace region of the decoder's layout that no kernel writes (a write past
// a region's end lands there, where a guard check sees it).
constexpr size_t kGuardBytes = 256;
inline size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// Operand type of a decoder's kernels: the storage dtype, or fp16 for bf16 weights with
// f16_compute (converted at load).
inline int compute_dtype(const ll_config &c) {
  return c.dtype == LL_BF16 && c.f16_compute ? kF16 : c.dtype;
}

inline ll_status check_ws(const void *p) {
  if (!p) return fail(LL_ERR_WORKSPACE, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(p) % kAlign)
    return fail(LL_ERR_WORKSPACE, "workspace not %zu-byte aligned", kAlign);
  return LL_OK;
}

// Collects (phase, kernel class, start, stop) for every launch while installed.  A launcher's
// follow-up kernel (split-K reduction, attention combine) is counted under `sec_to` when the
// current class is `sec_from`, else under the current class.
struct Timer : LaunchTimer {
  struct Rec {
    int phase, cls;
    hipEvent_t a, b;
  };
  std::vector<hipEvent_t> pool;
  std::vector<Rec> recs;
  int phase = 0, cls = 0;
  int sec_from = -1, sec_to = -1;
  Timer(int from = -1, int to = -1) : sec_from(from), sec_to(to) {}
  bool next(hipEvent_t *a, hipEvent_t *b) override {
    while (pool.size() < 2 * recs.size() + 2) {
      hipEvent_t e;
      if (hipEventCreate(&e) != hipSuccess) return false;
      pool.push_back(e);
    }
    *a = pool[2 * recs.size()];
    *b = pool[2 * recs.size() + 1];
    recs.push_back({phase, cls, *a, *b});
    return true;
  }
  void secondary() override {
    if (cls == sec_from) cls = sec_to;
  }
  ~Timer() override {
    for (auto e : pool) (void)hipEventDestroy(e);
  }
  // Sum the recorded launches into counts / ms [2 * n_classes] (phase-major) and forget them.
  ll_status drain(hipStream_t s, int n_classes, int32_t *counts, double *ms) {
    LL_HIP(hipStreamSynchronize(s));
    for (const auto &r : recs) {
      float t = 0.f;
      LL_HIP(hipEventElapsedTime(&t, r.a, r.b));
      counts[r.phase * n_classes + r.cls] += 1;
      ms[r.phase * n_classes + r.cls] += t;
    }
    recs.clear();
    return LL_OK;
  }
};

// Installs a model's timer on this thread for the duration of one ll_* call.
struct TimerScope {
  LaunchTimer *saved;
  TimerScope(Timer *t, int phase) : saved(g_launch_timer) {
    if (t) t->phase = phase;
    g_launch_timer = t;
  }
  ~TimerScope() { g_launch_timer = saved; }
};

}  // namespace ll
