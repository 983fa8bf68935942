// C ABI of the pcmoe library: argument validation (before any HIP call), workspace sizing,
// error reporting and the optional per-kernel event timing. Kernels live in the other files.
#include "pcmoe_internal.h"

#include <atomic>
#include <mutex>
#include <string>
#include <vector>
#include <map>
#include <cstdio>
#include <cstring>
#include <cstdarg>
#include <cmath>

using namespace pcmoe;

namespace {

thread_local std::string g_last_error;

moe_status fail(moe_status s, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
moe_status fail(moe_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return s;
}

moe_status hip_status(hipError_t e, const char* where) {
  if (e == hipSuccess) return MOE_OK;
  return fail(MOE_ERR_HIP, "%s: %s", where, hipGetErrorString(e));
}

moe_status check_desc(const moe_desc* d) {
  if (!d) return fail(MOE_ERR_INVALID_ARGUMENT, "desc is NULL");
  if (d->dtype != MOE_F32 && d->dtype != MOE_BF16) return fail(MOE_ERR_INVALID_ARGUMENT, "dtype %d", d->dtype);
  if (d->T < 1 || d->d_model < 1 || d->d_ff < 1 || d->n_experts < 1)
    return fail(MOE_ERR_INVALID_ARGUMENT, "non-positive shape T=%d d=%d f=%d E=%d", d->T, d->d_model, d->d_ff,
                d->n_experts);
  if (d->top_k < 1 || d->top_k > d->n_experts)
    return fail(MOE_ERR_INVALID_ARGUMENT, "top_k=%d outside [1, E=%d]", d->top_k, d->n_experts);
  if (d->local_count < 0 || d->local_begin < 0 || d->local_begin + d->local_count > d->n_experts)
    return fail(MOE_ERR_INVALID_ARGUMENT, "hosted range [%d, %d+%d) outside [0, %d)", d->local_begin,
                d->local_begin, d->local_count, d->n_experts);
  if (d->n_shared < 0) return fail(MOE_ERR_INVALID_ARGUMENT, "n_shared=%d < 0", d->n_shared);
  // A party hosts at least one routed expert: the dispatch, the combine and the grouped GEMMs all read the
  // per-expert offsets that moe_permute produces for the hosted range.
  if (d->local_count < 1)
    return fail(MOE_ERR_INVALID_ARGUMENT, "local_count=%d: at least one hosted routed expert", d->local_count);
  if (d->renormalize != 0 && d->renormalize != 1)
    return fail(MOE_ERR_INVALID_ARGUMENT, "renormalize must be 0 or 1");
  if (d->top_k > 8) return fail(MOE_ERR_UNSUPPORTED, "top_k=%d > 8", d->top_k);
  if (d->n_experts > 256) return fail(MOE_ERR_UNSUPPORTED, "n_experts=%d > 256", d->n_experts);
  if (d->local_count + d->n_shared > 511)
    return fail(MOE_ERR_UNSUPPORTED, "local_count + n_shared = %d > 511", d->local_count + d->n_shared);
  if (d->d_model % 128 || d->d_ff % 128)
    return fail(MOE_ERR_UNSUPPORTED, "d_model=%d and d_ff=%d must be multiples of 128", d->d_model, d->d_ff);
  const int64_t R = rows_total(*d);
  if (R * (int64_t)(2 * d->d_ff) >= (int64_t)1 << 40 || R >= ((int64_t)1 << 31) / 2)
    return fail(MOE_ERR_UNSUPPORTED, "row space of %lld rows is too large", (long long)R);
  if ((int64_t)d->T * d->top_k >= ((int64_t)1 << 31) - 1024)
    return fail(MOE_ERR_UNSUPPORTED, "T*k too large for int32 slot indices");
  // The grouped GEMMs address one group's operand rows and one expert's weight matrix through 32-bit buffer
  // ranges and 32-bit lane offsets. A group holds at most T rows (a token selects an expert once; a shared
  // expert takes every token), and its widest row is max(d_model, 2 d_ff) elements (x / dY rows, or the
  // G|U and dG|dU rows). A tile's lanes address up to one 256-row tile past the last row of a group (the
  // rows of a group's last m-tile, the K rows of a weight gradient's last K-tile) or of a weight matrix (the
  // last n-tile): those offsets, too, stay below 2^31.
  const int64_t es = d->dtype == MOE_BF16 ? 2 : 4;
  const int64_t row_bytes = (int64_t)(d->d_model > 2 * d->d_ff ? d->d_model : 2 * d->d_ff) * es;
  if (((int64_t)d->T + 256) * row_bytes >= ((int64_t)1 << 31))
    return fail(MOE_ERR_UNSUPPORTED, "T=%d (+ 256) rows of %lld bytes exceed the 2 GiB extent of one operand group",
                d->T, (long long)row_bytes);
  const int64_t wmax = d->d_ff > d->d_model ? d->d_ff : d->d_model;
  if ((wmax + 256) * wmax * es >= ((int64_t)1 << 31))
    return fail(MOE_ERR_UNSUPPORTED, "one expert's %d x %d weight matrix (+ 256 rows) exceeds 2 GiB", d->d_ff,
                d->d_model);
  return MOE_OK;
}

// Every buffer is read and written in 16-byte vectors.
#define NEED(p)                                                                         \
  do {                                                                                  \
    if (!(p)) return fail(MOE_ERR_INVALID_ARGUMENT, #p " is NULL");                     \
    if ((uintptr_t)(p) & 15) return fail(MOE_ERR_INVALID_ARGUMENT, #p " is not 16-byte aligned"); \
  } while (0)

#define NEED_WS(have, need)                                                                                   \
  do {                                                                                                        \
    size_t need_ = (need);                                                                                    \
    if ((have) < need_)                                                                                       \
      return fail(MOE_ERR_WORKSPACE_TOO_SMALL, "workspace of %zu bytes, %zu needed", (size_t)(have), need_); \
    if (need_ && !ws) return fail(MOE_ERR_INVALID_ARGUMENT, "ws is NULL");                                    \
    if ((uintptr_t)ws & 255) return fail(MOE_ERR_INVALID_ARGUMENT, "ws is not 256-byte aligned");             \
  } while (0)

// ------------------------------------------------------------------ per-kernel timing
// The library's one global besides the thread-local error string: a measurement aid, off by default. Its event
// pool and record table are created by moe_kernel_timing(1) (the only call that creates anything); the layer calls
// then take events from the pool and append to the preallocated table, so they never allocate, timing on or off.
// When the pool is spent, further launches go unrecorded (counted in `dropped`).
constexpr size_t kTimingPairs = 4096;  // event pairs in the pool: launches recorded between two enables
struct TimingState {
  std::mutex mu;
  std::atomic<bool> on{false};  // read without the lock on every launch (the common case: timing off)
  std::string only;  // record only launches with this name (empty: all)
  struct Rec {
    const char* name;  // a launcher's string literal
    hipEvent_t a, b;
  };
  std::vector<Rec> recs;         // capacity kTimingPairs, reserved once
  std::vector<hipEvent_t> pool;  // 2 * kTimingPairs events, created once
  size_t used = 0;               // pairs handed out since the last enable
  size_t dropped = 0;
};
TimingState& timing() {
  static TimingState* t = new TimingState();
  return *t;
}

}  // namespace

namespace pcmoe {
KernelTimer::KernelTimer(const char* n, hipStream_t s) : name(n), stream(s), slot(nullptr) {
  TimingState& ts = timing();
  if (!ts.on.load(std::memory_order_acquire)) return;
  std::lock_guard<std::mutex> lk(ts.mu);
  if (!ts.on.load(std::memory_order_relaxed)) return;
  if (!ts.only.empty() && ts.only != n) return;
  if (ts.used >= kTimingPairs || 2 * ts.used + 1 >= ts.pool.size()) {
    ++ts.dropped;
    return;
  }
  hipEvent_t a = ts.pool[2 * ts.used], b = ts.pool[2 * ts.used + 1];
  ++ts.used;
  (void)hipEventRecord(a, s);
  ts.recs.push_back({n, a, b});  // within the reserved capacity
  slot = (void*)(uintptr_t)ts.recs.size();
}
KernelTimer::~KernelTimer() {
  if (!slot) return;
  TimingState& ts = timing();
  std::lock_guard<std::mutex> lk(ts.mu);
  size_t i = (size_t)(uintptr_t)slot - 1;
  if (i < ts.recs.size()) (void)hipEventRecord(ts.recs[i].b, stream);
}
}  // namespace pcmoe

extern "C" {

const char* moe_status_string(moe_status s) {
  switch (s) {
    case MOE_OK: return "MOE_OK";
    case MOE_ERR_INVALID_ARGUMENT: return "MOE_ERR_INVALID_ARGUMENT";
    case MOE_ERR_UNSUPPORTED: return "MOE_ERR_UNSUPPORTED";
    case MOE_ERR_WORKSPACE_TOO_SMALL: return "MOE_ERR_WORKSPACE_TOO_SMALL";
    case MOE_ERR_HIP: return "MOE_ERR_HIP";
  }
  return "MOE_ERR_UNKNOWN";
}

const char* moe_last_error(void) { return g_last_error.c_str(); }

size_t moe_workspace_size(const moe_desc* d, int which) {
  if (check_desc(d) != MOE_OK) return 0;
  switch (which) {
    case MOE_WS_PERMUTE: return permute_ws_bytes(*d);
    case MOE_WS_FFN_SAVED: return ffn_saved_bytes(*d);
    case MOE_WS_FFN_FWD: return ffn_fwd_ws_bytes(*d);
    case MOE_WS_FFN_BWD: return ffn_bwd_ws_bytes(*d);
    case MOE_WS_ROUTE_BWD: return route_bwd_ws_bytes(*d);
  }
  return 0;
}

moe_status moe_route(const moe_desc* d, const void* x, const void* w_router, const float* logit_bias,
                     int32_t bias_groups, float* logits, int32_t* topk_idx, float* topk_w, hipStream_t stream) {
  moe_status st = check_desc(d);
  if (st) return st;
  NEED(x); NEED(w_router); NEED(logits); NEED(topk_idx); NEED(topk_w);
  if (logit_bias && ((uintptr_t)logit_bias & 3)) return fail(MOE_ERR_INVALID_ARGUMENT, "logit_bias misaligned");
  if (logit_bias && (bias_groups < 1 || d->T % bias_groups))
    return fail(MOE_ERR_INVALID_ARGUMENT, "bias_groups=%d must divide T=%d", bias_groups, d->T);
  return hip_status(launch_route_fwd(*d, x, w_router, logit_bias, logit_bias ? bias_groups : 1, logits, topk_idx,
                                     topk_w, stream),
                    "moe_route");
}

moe_status moe_permute(const moe_desc* d, const int32_t* topk_idx, const void* x, int32_t* counts, int32_t* offsets,
                       int32_t* row_to_slot, int32_t* slot_to_row, void* x_perm, void* ws, size_t ws_bytes,
                       hipStream_t stream) {
  moe_status st = check_desc(d);
  if (st) return st;
  NEED(topk_idx); NEED(x); NEED(counts); NEED(offsets); NEED(row_to_slot); NEED(slot_to_row); NEED(x_perm);
  NEED_WS(ws_bytes, permute_ws_bytes(*d));
  return hip_status(launch_permute(*d, topk_idx, x, counts, offsets, row_to_slot, slot_to_row, x_perm, ws, stream),
                    "moe_permute");
}

moe_status moe_permute_noalloc(const moe_desc* d, const int32_t* topk_idx, const void* x, int32_t* counts,
                               int32_t* offsets, int32_t* row_to_slot, int32_t* slot_to_row, void* x_perm,
                               hipStream_t stream) {
  moe_status st = check_desc(d);
  if (st) return st;
  NEED(topk_idx); NEED(x); NEED(counts); NEED(offsets); NEED(row_to_slot); NEED(slot_to_row); NEED(x_perm);
  const size_t need = permute_ws_bytes(*d);
  if (need > permute_noalloc_capacity())
    return fail(MOE_ERR_UNSUPPORTED, "moe_permute_noalloc: %zu bytes of scratch needed, its fixed scratch holds %zu",
                need, permute_noalloc_capacity());
  void* ws = nullptr;
  if (hipError_t e = permute_noalloc_scratch(&ws); e != hipSuccess) return hip_status(e, "moe_permute_noalloc");
  return hip_status(launch_permute(*d, topk_idx, x, counts, offsets, row_to_slot, slot_to_row, x_perm, ws, stream),
                    "moe_permute_noalloc");
}

moe_status moe_expert_ffn_fwd(const moe_desc* d, const void* x, const void* x_perm, const int32_t* offsets,
                              const void* w_gate, const void* w_up, const void* w_down, void* y_perm, void* saved,
                              void* ws, size_t ws_bytes, hipStream_t stream) {
  moe_status st = check_desc(d);
  if (st) return st;
  if (d->n_shared > 0) NEED(x);
  NEED(x_perm); NEED(offsets);
  NEED(w_gate); NEED(w_up); NEED(w_down); NEED(y_perm); NEED(saved);
  NEED_WS(ws_bytes, ffn_fwd_ws_bytes(*d));
  return hip_status(launch_ffn_fwd(*d, x, x_perm, offsets, w_gate, w_up, w_down, y_perm, saved, ws, stream),
                    "moe_expert_ffn_fwd");
}

moe_status moe_combine(const moe_desc* d, const void* y_perm, const int32_t* slot_to_row, const float* topk_w,
                       void* y, hipStream_t stream) {
  moe_status st = check_desc(d);
  if (st) return st;
  NEED(y_perm); NEED(slot_to_row); NEED(topk_w); NEED(y);
  return hip_status(launch_combine(*d, y_perm, slot_to_row, topk_w, y, stream), "moe_combine");
}

moe_status moe_combine_bwd(const moe_desc* d, const void* dy, const void* y_perm, const int32_t* slot_to_row,
                           const float* topk_w, void* dy_perm, float* dgate, hipStream_t stream) {
  moe_status st = check_desc(d);
  if (st) return st;
  NEED(dy); NEED(y_perm); NEED(slot_to_row); NEED(topk_w); NEED(dy_perm); NEED(dgate);
  return hip_status(launch_combine_bwd(*d, dy, y_perm, slot_to_row, topk_w, dy_perm, dgate, stream),
                    "moe_combine_bwd");
}

moe_status moe_expert_ffn_bwd(const moe_desc* d, const void* x, const void* x_perm, const void* dy,
                              const void* dy_perm, const int32_t* offsets, const void* w_gate, const void* w_up,
                              const void* w_down, const void* saved, void* dx_perm, void* dw_gate, void* dw_up,
                              void* dw_down, void* ws, size_t ws_bytes, hipStream_t stream) {
  moe_status st = check_desc(d);
  if (st) return st;
  if (d->n_shared > 0) { NEED(x); NEED(dy); }
  NEED(x_perm); NEED(dy_perm); NEED(offsets);
  NEED(w_gate); NEED(w_up); NEED(w_down); NEED(saved); NEED(dx_perm); NEED(dw_gate); NEED(dw_up); NEED(dw_down);
  NEED_WS(ws_bytes, ffn_bwd_ws_bytes(*d));
  return hip_status(launch_ffn_bwd(*d, x, x_perm, dy, dy_perm, offsets, w_gate, w_up, w_down, saved, dx_perm,
                                   dw_gate, dw_up, dw_down, ws, stream),
                    "moe_expert_ffn_bwd");
}

moe_status moe_route_bwd(const moe_desc* d, const void* x, const float* logits, const int32_t* topk_idx,
                         const float* topk_w, const float* dgate, float* dlogits, float* dw_router, void* ws,
                         size_t ws_bytes, hipStream_t stream) {
  moe_status st = check_desc(d);
  if (st) return st;
  if (d->local_begin != 0 || d->local_count != d->n_experts)
    return fail(MOE_ERR_INVALID_ARGUMENT,
                "moe_route_bwd needs every expert's dgate (local range must be [0, E)); a party shard leaves the "
                "router gradient to the data owner");
  NEED(x); NEED(topk_idx); NEED(topk_w); NEED(dgate); NEED(dlogits); NEED(dw_router);
  if (!d->renormalize) NEED(logits);
  NEED_WS(ws_bytes, route_bwd_ws_bytes(*d));
  return hip_status(launch_route_bwd(*d, x, logits, topk_idx, topk_w, dgate, dlogits, dw_router, ws, stream),
                    "moe_route_bwd");
}

moe_status moe_permute_bwd(const moe_desc* d, const void* dx_perm, const int32_t* slot_to_row, const float* dlogits,
                           const void* w_router, void* dx, hipStream_t stream) {
  moe_status st = check_desc(d);
  if (st) return st;
  NEED(dx_perm); NEED(slot_to_row); NEED(dx);
  if (dlogits) NEED(w_router);
  return hip_status(launch_permute_bwd(*d, dx_perm, slot_to_row, dlogits, w_router, dx, stream), "moe_permute_bwd");
}

moe_status moe_expert_update(const moe_desc* d, const moe_opt* opt, void* w_gate, void* w_up, void* w_down,
                             const void* dw_gate, const void* dw_up, const void* dw_down, float* master, float* m,
                             float* v, hipStream_t stream) {
  moe_status st = check_desc(d);
  if (st) return st;
  if (!opt) return fail(MOE_ERR_INVALID_ARGUMENT, "opt is NULL");
  if (opt->kind != MOE_OPT_SGD && opt->kind != MOE_OPT_ADAMW)
    return fail(MOE_ERR_INVALID_ARGUMENT, "optimiser kind %d", opt->kind);
  if (!(opt->lr > 0.f) || !std::isfinite(opt->lr)) return fail(MOE_ERR_INVALID_ARGUMENT, "lr must be > 0");
  if (!(opt->weight_decay >= 0.f) || !std::isfinite(opt->weight_decay))
    return fail(MOE_ERR_INVALID_ARGUMENT, "weight_decay must be >= 0");
  NEED(w_gate); NEED(w_up); NEED(w_down); NEED(dw_gate); NEED(dw_up); NEED(dw_down);
  if (master) NEED(master);
  const int64_t params = (int64_t)(d->local_count + d->n_shared) * d->d_ff * d->d_model;
  if (params / 8 * 3 / 256 >= ((int64_t)1 << 31) - 1)
    return fail(MOE_ERR_UNSUPPORTED, "%lld parameters per weight tensor are too many", (long long)params);
  if (opt->kind == MOE_OPT_ADAMW) {
    if (!(opt->beta1 >= 0.f && opt->beta1 < 1.f) || !(opt->beta2 >= 0.f && opt->beta2 < 1.f))
      return fail(MOE_ERR_INVALID_ARGUMENT, "beta1, beta2 must lie in [0, 1)");
    if (!(opt->eps > 0.f) || !std::isfinite(opt->eps)) return fail(MOE_ERR_INVALID_ARGUMENT, "eps must be > 0");
    if (opt->step < 1) return fail(MOE_ERR_INVALID_ARGUMENT, "step must be >= 1");
    NEED(m); NEED(v);
  }
  return hip_status(launch_expert_update(*d, *opt, w_gate, w_up, w_down, dw_gate, dw_up, dw_down, master, m, v,
                                         stream),
                    "moe_expert_update");
}

moe_status moe_kernel_timing(int enable) {
  TimingState& ts = timing();
  std::lock_guard<std::mutex> lk(ts.mu);
  if (enable && ts.pool.size() < 2 * kTimingPairs) {
    ts.recs.reserve(kTimingPairs);
    while (ts.pool.size() < 2 * kTimingPairs) {
      hipEvent_t e = nullptr;
      if (hipError_t err = hipEventCreate(&e); err != hipSuccess) {
        ts.on.store(false, std::memory_order_release);
        return hip_status(err, "moe_kernel_timing");
      }
      ts.pool.push_back(e);
    }
  }
  ts.recs.clear();
  ts.used = 0;
  ts.dropped = 0;
  ts.on.store(enable != 0, std::memory_order_release);
  return MOE_OK;
}

moe_status moe_kernel_timing_select(const char* kernel_name) {
  TimingState& ts = timing();
  std::lock_guard<std::mutex> lk(ts.mu);
  ts.only = kernel_name ? kernel_name : "";
  return MOE_OK;
}

size_t moe_kernel_timing_report(char* buf, size_t n) {
  TimingState& ts = timing();
  std::lock_guard<std::mutex> lk(ts.mu);
  std::map<std::string, std::pair<long, double>> agg;
  std::vector<std::string> order;
  if (ts.dropped) {
    order.push_back("(unrecorded)");
    agg["(unrecorded)"] = {(long)ts.dropped, 0.0};
  }
  for (auto& r : ts.recs) {
    float ms = 0.f;
    if (hipEventSynchronize(r.b) != hipSuccess || hipEventElapsedTime(&ms, r.a, r.b) != hipSuccess) continue;
    auto it = agg.find(r.name);
    if (it == agg.end()) {
      order.push_back(r.name);
      agg[r.name] = {1, (double)ms};
    } else {
      it->second.first += 1;
      it->second.second += ms;
    }
  }
  std::string out;
  for (auto& nm : order) {
    char line[256];
    snprintf(line, sizeof(line), "%s %ld %.6f\n", nm.c_str(), agg[nm].first, agg[nm].second);
    out += line;
  }
  if (buf && n) {
    size_t m = out.size() < n - 1 ? out.size() : n - 1;
    memcpy(buf, out.data(), m);
    buf[m] = 0;
  }
  return out.size() + 1;
}

}  // extern "C"
