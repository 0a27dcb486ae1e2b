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

// Host state of the state-space models (Mamba, Mamba2, RG-LRU) and the C-ABI calls that only
// touch it: the caller's workspace and stream, the sequences held, implementation options, the
// decode-graph cache and the per-launch timer.  Each model's handle derives from it and adds
// its configuration, workspace layout and kernels.
struct StateModel {
  struct Graph {
    const void *in;
    void *out;
    void *logits;
    int batch;
    hipGraphExec_t exec;
  };
  const char *reset_call;  // the model's reset entry point, named in error messages
  bool fused_option;       // LL_OPT_DECODE_FUSED applies to this model
  char *ws = nullptr;
  hipStream_t stream = nullptr;
  hipStream_t cap_stream = nullptr;
  int batch = 0;
  std::vector<int> lens;
  int opt[LL_OPT_COUNT] = {1, 1, 1, 0, 0, 0};
  std::vector<Graph> graphs;
  Timer *timer = nullptr;

  StateModel(const char *reset, bool fused) : reset_call(reset), fused_option(fused) {
    opt[LL_OPT_DECODE_FUSED] = fused ? 1 : 0;
  }
  StateModel(const StateModel &) = delete;
  StateModel &operator=(const StateModel &) = delete;
  ~StateModel() {
    drop_graphs();
    if (cap_stream) (void)hipStreamDestroy(cap_stream);
    delete timer;
  }
  void mark(int cls) const {
    if (timer) timer->cls = cls;
  }
  template <typename P = void> P *at(size_t off) const { return reinterpret_cast<P *>(ws + off); }
  void drop_graphs() {
    for (auto &g : graphs) (void)hipGraphExecDestroy(g.exec);
    graphs.clear();
  }

  ll_status reset() {
    batch = 0;
    lens.clear();
    return LL_OK;
  }
  ll_status seq_lengths(int32_t *out, int32_t cap, int32_t *n) const {
    if (!n || (cap > 0 && !out)) return fail(LL_ERR_INVALID_ARGUMENT, "NULL argument");
    *n = batch;
    for (int b = 0; b < batch && b < cap; ++b) out[b] = lens[b];
    return LL_OK;
  }
  bool option_applies(int32_t option) const {
    return option != LL_OPT_ATTN_DECODE_CHUNK && (option != LL_OPT_DECODE_FUSED || fused_option);
  }
  ll_status set_option(int32_t option, int32_t value) {
    if (option < 0 || option >= LL_OPT_COUNT) return fail(LL_ERR_INVALID_ARGUMENT, "unknown option %d", option);
    if (!option_applies(option))
      return fail(LL_ERR_UNSUPPORTED, "option %d does not apply to this model", option);
    switch (option) {
      case LL_OPT_DECODE_GRAPH:
      case LL_OPT_PREFILL_SPLITK:
        if (value != 0 && value != 1) return fail(LL_ERR_INVALID_ARGUMENT, "option %d takes 0 or 1", option);
        break;
      case LL_OPT_DECODE_SPLITK:
        if (value < 0 || value > 2) return fail(LL_ERR_INVALID_ARGUMENT, "decode split-K 0, 1 or 2");
        break;
      case LL_OPT_PREFILL_TILE:
        if (value < 0 || value > 3) return fail(LL_ERR_INVALID_ARGUMENT, "prefill tile 0..3");
        break;
      case LL_OPT_DECODE_FUSED:
        if (value < 0 || value > 2) return fail(LL_ERR_INVALID_ARGUMENT, "option %d takes 0, 1 or 2", option);
        break;
    }
    if (opt[option] != value) drop_graphs();
    opt[option] = value;
    return LL_OK;
  }
  ll_status get_option(int32_t option, int32_t *value) const {
    if (!value) return fail(LL_ERR_INVALID_ARGUMENT, "NULL argument");
    if (option < 0 || option >= LL_OPT_COUNT) return fail(LL_ERR_INVALID_ARGUMENT, "unknown option %d", option);
    if (!option_applies(option))
      return fail(LL_ERR_UNSUPPORTED, "option %d does not apply to this model", option);
    *value = opt[option];
    return LL_OK;
  }
  // Synchronises the stream and copies the device flags (an int32 at workspace offset err_off).
  ll_status device_flags(size_t err_off, int32_t *flags) {
    if (!flags) return fail(LL_ERR_INVALID_ARGUMENT, "NULL argument");
    LL_HIP(hipStreamSynchronize(stream));
    LL_HIP(hipMemcpy(flags, at(err_off), 4, hipMemcpyDeviceToHost));
    return LL_OK;
  }
  ll_status set_kernel_timing(int32_t enable) {
    if (enable && !timer) timer = new Timer();
    if (!enable && timer) {
      (void)hipStreamSynchronize(stream);
      delete timer;
      timer = nullptr;
    }
    return LL_OK;
  }
  ll_status kernel_timing_read(int n_classes, int32_t *counts, double *ms) {
    if (!counts || !ms) return fail(LL_ERR_INVALID_ARGUMENT, "NULL argument");
    for (int i = 0; i < 2 * n_classes; ++i) {
      counts[i] = 0;
      ms[i] = 0.0;
    }
    if (!timer) return fail(LL_ERR_STATE, "kernel timing is not enabled");
    return timer->drain(stream, n_classes, counts, ms);
  }
  // A prefill of n sequences with host lengths lens_host: on a held state it is a further
  // chunk of the same sequences.  The prompt tokens in all go to *total.
  ll_status check_prefill(int32_t n, const int32_t *lens_host, int max_batch, int max_tokens,
                          long *total) const {
    if (n < 1) return fail(LL_ERR_INVALID_ARGUMENT, "batch %d < 1", n);
    if (n > max_batch) return fail(LL_ERR_CAPACITY, "batch %d > max_batch %d", n, max_batch);
    if (batch != 0 && n != batch)
      return fail(LL_ERR_STATE, "prefill of %d sequences on state of %d (a further chunk extends "
                  "the same sequences; %s starts new ones)", n, batch, reset_call);
    long t = 0;
    for (int b = 0; b < n; ++b) {
      if (lens_host[b] < 1) return fail(LL_ERR_INVALID_ARGUMENT, "seq_lens[%d] = %d < 1", b, lens_host[b]);
      t += lens_host[b];
    }
    if (t > max_tokens)
      return fail(LL_ERR_CAPACITY, "%ld prompt tokens > max_prefill_tokens %d", t, max_tokens);
    *total = t;
    return LL_OK;
  }
  void commit_prefill(int32_t n, const int32_t *lens_host) {
    if (batch != 0) {
      for (int b = 0; b < n; ++b) lens[b] += lens_host[b];
    } else {
      batch = n;
      lens.assign(lens_host, lens_host + n);
    }
  }
  // One decode step of the held sequences: replayed from the graph cache (captured on a
  // model-owned stream the first time these buffers are used) or launched directly, with the
  // timer on or the graph option off.  enqueue(stream) issues the step's kernels.
  template <typename Enqueue>
  ll_status decode(const int32_t *in, int32_t *out, float *logits, Enqueue &&enqueue) {
    if (batch == 0) return fail(LL_ERR_STATE, "decode before prefill");
    TimerScope scope(timer, 1);
    if (opt[LL_OPT_DECODE_GRAPH] && !timer) {
      hipGraphExec_t exec = nullptr;
      for (auto &g : graphs)
        if (g.in == in && g.out == out && g.logits == logits && g.batch == batch) exec = g.exec;
      if (!exec) {
        if (!cap_stream) LL_HIP(hipStreamCreateWithFlags(&cap_stream, hipStreamNonBlocking));
        LL_HIP(hipStreamBeginCapture(cap_stream, hipStreamCaptureModeThreadLocal));
        ll_status st = enqueue(cap_stream);
        hipGraph_t graph = nullptr;
        hipError_t ec = hipStreamEndCapture(cap_stream, &graph);
        if (st != LL_OK) {
          if (graph) (void)hipGraphDestroy(graph);
          return st;
        }
        if (ec != hipSuccess) return fail(LL_ERR_HIP, "hipStreamEndCapture: %s", hipGetErrorString(ec));
        ec = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
        (void)hipGraphDestroy(graph);
        if (ec != hipSuccess) return fail(LL_ERR_HIP, "hipGraphInstantiate: %s", hipGetErrorString(ec));
        if (graphs.size() >= 8) {
          (void)hipGraphExecDestroy(graphs.front().exec);
          graphs.erase(graphs.begin());
        }
        graphs.push_back({in, out, logits, batch, exec});
      }
      LL_HIP(hipGraphLaunch(exec, stream));
    } else {
      ll_status st = enqueue(stream);
      if (st != LL_OK) return st;
    }
    for (auto &l : lens) ++l;
    return LL_OK;
  }
};

}  // namespace ll
