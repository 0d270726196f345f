// C ABI of libreflex: host-side validation, workspace carving and launch order.
// Every check happens before the first launch; nothing here allocates, frees or
// synchronises.
#include <algorithm>
#include <cmath>
#include <cstring>

#include <initializer_list>
#include <mutex>
#include <vector>

#include "common.h"

using namespace rfx;

#define RFX_TRY_INNER(expr)           \
  do {                                \
    const int rc_ = (expr);           \
    if (rc_ != REFLEX_OK) return rc_; \
  } while (0)

namespace {

constexpr int kVersion = 100;

// Pointers the kernels access with 16-byte vectors (bf16 matrices, the fp32 router
// weight, the workspace) must be 16-byte aligned; every other pointer only needs the
// natural alignment of its element type.
bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

int check_ptr(const void* p, size_t a = 16) {
  if (p == nullptr) return REFLEX_ERR_NULL;
  return aligned(p, a) ? REFLEX_OK : REFLEX_ERR_SHAPE;
}

int check_opt_ptr(const void* p, size_t a = 16) {
  return (p == nullptr || aligned(p, a)) ? REFLEX_OK : REFLEX_ERR_SHAPE;
}

int check_ptrs(std::initializer_list<const void*> ps, size_t a) {
  for (const void* p : ps) RFX_TRY_INNER(check_ptr(p, a));
  return REFLEX_OK;
}

#define RFX_TRY(expr)                 \
  do {                                \
    const int rc_ = (expr);           \
    if (rc_ != REFLEX_OK) return rc_; \
  } while (0)

bool valid_T(int T) { return T >= 0 && T <= REFLEX_MAX_TOKENS; }
bool valid_E(int E) { return E >= 1 && E <= REFLEX_MAX_EXPERTS; }
bool valid_d(int d) { return d >= REFLEX_D_MULTIPLE && d <= REFLEX_MAX_DIM && d % REFLEX_D_MULTIPLE == 0; }
bool valid_f(int f) { return f >= REFLEX_F_MULTIPLE && f <= REFLEX_MAX_DIM && f % REFLEX_F_MULTIPLE == 0; }
bool valid_kmax(int k_max, int E) { return k_max >= 0 && k_max <= REFLEX_MAX_K && k_max <= E; }

int check_params(const reflex_alloc_params* p) {
  if (p == nullptr) return REFLEX_ERR_NULL;
  const float fs[5] = {p->q, p->theta, p->w_cf, p->v_ref, p->tau};
  for (float v : fs)
    if (!std::isfinite(v)) return REFLEX_ERR_PARAM;
  if (p->k_min < 0 || p->k_min > p->k_max || p->k_max > REFLEX_MAX_K) return REFLEX_ERR_PARAM;
  if (p->k_base < 0 || p->delta_role < 0 || p->delta_cur < 0) return REFLEX_ERR_PARAM;
  if (p->k_base > 1024 || p->delta_role > 1024 || p->delta_cur > 1024) return REFLEX_ERR_PARAM;
  if (!(p->q > 0.0f && p->q <= 0.5f) || !(p->tau > 0.0f) || !(p->w_cf > 0.0f)) return REFLEX_ERR_PARAM;
  if (p->signal < REFLEX_SIGNAL_FPS || p->signal > REFLEX_SIGNAL_UNCERTAINTY) return REFLEX_ERR_PARAM;
  return REFLEX_OK;
}

// Fused-path workspace carve-up; every region 256-byte aligned.
// Threshold of a score-derived count rule: p in (0, 1] for Top-p, tau in [0, 1).
int check_rule(int rule, float threshold) {
  if (!std::isfinite(threshold)) return REFLEX_ERR_PARAM;
  if (rule == REFLEX_RULE_TOP_P) return threshold > 0.0f && threshold <= 1.0f ? REFLEX_OK : REFLEX_ERR_PARAM;
  if (rule == REFLEX_RULE_THRESHOLD)
    return threshold >= 0.0f && threshold < 1.0f ? REFLEX_OK : REFLEX_ERR_PARAM;
  return REFLEX_ERR_PARAM;
}

// A second stream per device for work of the forward that reads nothing the routing
// computes (the shared expert): non-blocking (no implicit ordering with the legacy
// default stream), default priority, created on first use and kept for the life of the
// process.  NULL if it cannot be created (the work then stays on the caller's stream).
hipStream_t side_stream() {
  static std::mutex mu;
  static hipStream_t streams[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return nullptr;
  std::lock_guard<std::mutex> g(mu);
  if (streams[dev] == nullptr) {
    hipStream_t st = nullptr;
    if (hipStreamCreateWithFlags(&st, hipStreamNonBlocking) != hipSuccess) return nullptr;
    streams[dev] = st;
  }
  return streams[dev];
}

// Fork and join events of the shared-expert side stream.  Each forward borrows one
// pair from a per-device pool for the duration of the host call and returns it at
// exit: a wait enqueued on a stream waits for the event's record as of the wait call,
// so a later re-record by another forward cannot affect it, and concurrent callers
// never hold the same pair.  Events are created only when the pool of a device is
// empty (at most one pair per concurrent caller) and kept for the life of the process.
struct EventPair {
  hipEvent_t fork = nullptr, join = nullptr;
};

class EventPool {
 public:
  bool take(int dev, EventPair& out) {
    {
      std::lock_guard<std::mutex> g(mu_);
      std::vector<EventPair>& v = free_[dev];
      if (!v.empty()) {
        out = v.back();
        v.pop_back();
        return true;
      }
    }
    EventPair e;
    if (hipEventCreateWithFlags(&e.fork, hipEventDisableTiming) != hipSuccess) return false;
    if (hipEventCreateWithFlags(&e.join, hipEventDisableTiming) != hipSuccess) {
      (void)hipEventDestroy(e.fork);
      return false;
    }
    out = e;
    return true;
  }
  void give(int dev, const EventPair& e) {
    std::lock_guard<std::mutex> g(mu_);
    free_[dev].push_back(e);
  }

 private:
  std::mutex mu_;
  std::vector<EventPair> free_[64];
};

EventPool& event_pool() {
  static EventPool* pool = new EventPool();   // never destroyed: outlives every caller
  return *pool;
}

// The shared expert's fork off the caller's stream `s` onto the side stream, as a
// scope guard.  Once fork() has succeeded, every exit from the forward (success or
// error) leaves `s` ordered after all work enqueued on the side stream by this call:
// join() does it on the normal path; on an early error return the destructor records
// the join and makes `s` wait on it (or, should even that fail, waits on the host for
// the side stream), so the caller may free or reuse the workspace once `s` is done.
class SideFork {
 public:
  explicit SideFork(hipStream_t s) : s_(s) {}
  SideFork(const SideFork&) = delete;
  SideFork& operator=(const SideFork&) = delete;

  // true: `side()` now runs after everything enqueued on `s` so far
  bool fork() {
    side_ = side_stream();
    if (side_ == nullptr || hipGetDevice(&dev_) != hipSuccess || dev_ < 0 || dev_ >= 64) return false;
    if (!event_pool().take(dev_, ev_)) return false;
    have_ev_ = true;
    if (hipEventRecord(ev_.fork, s_) != hipSuccess || hipStreamWaitEvent(side_, ev_.fork, 0) != hipSuccess)
      return false;     // nothing reached the side stream, or it waits on a recorded fork
    forked_ = true;
    return true;
  }
  hipStream_t side() const { return side_; }
  bool forked() const { return forked_; }

  int join() {
    if (!forked_ || joined_) return REFLEX_OK;
    joined_ = true;
    if (hipEventRecord(ev_.join, side_) != hipSuccess || hipStreamWaitEvent(s_, ev_.join, 0) != hipSuccess) {
      (void)hipStreamSynchronize(side_);
      return REFLEX_ERR_LAUNCH;
    }
    return REFLEX_OK;
  }

  ~SideFork() {
    (void)join();
    if (have_ev_) event_pool().give(dev_, ev_);
  }

 private:
  hipStream_t s_;
  hipStream_t side_ = nullptr;
  int dev_ = -1;
  EventPair ev_;
  bool have_ev_ = false, forked_ = false, joined_ = false;
};

struct Layout {
  size_t logits, k, done, pair_offsets, pair_expert, pair_weight, expert_offsets, sorted_token,
      pair_to_sorted, perm, route_hist, swiglu, y, shared_act, shared_y, total;
};

bool make_layout(int T, int E, int d, int f, int fs, int kcap, Layout& L) {
  if (!valid_T(T) || !valid_E(E) || !valid_d(d) || !valid_f(f)) return false;
  if (fs != 0 && !valid_f(fs)) return false;
  if (!valid_kmax(kcap, E)) return false;
  const size_t cap = static_cast<size_t>(T) * kcap;
  if (cap > static_cast<size_t>(INT32_MAX)) return false;
  size_t o = 0;
  auto take = [&](size_t bytes) {
    const size_t at = o;
    o += align_up(bytes);
    return at;
  };
  // scores, or on the split-K router paths their per-slice partials
  const int parts = std::max(front_fits(T, d) ? front_slices(d) : 1, router_slices(T, d, E));
  L.logits = take(sizeof(float) * static_cast<size_t>(T) * E * parts);
  L.k = take(sizeof(int32_t) * static_cast<size_t>(T));
  L.done = take(sizeof(int32_t));
  L.pair_offsets = take(sizeof(int32_t) * (static_cast<size_t>(T) + 1));
  L.pair_expert = take(sizeof(int32_t) * cap);
  L.pair_weight = take(sizeof(float) * cap);
  L.expert_offsets = take(sizeof(int32_t) * (E + 1));
  L.sorted_token = take(sizeof(int32_t) * cap);
  L.pair_to_sorted = take(sizeof(int32_t) * cap);
  L.perm = take(permute_ws_bytes(static_cast<int>(cap), E));
  L.route_hist = take(route_fused_sorts(T, E) || route_block_sorts(T, E) ? route_hist_bytes(T, E) : 0);
  L.swiglu = take(swiglu_ws_bytes(static_cast<int>(cap), E, f));
  L.y = take(sizeof(uint16_t) * cap * d);
  L.shared_act = fs ? take(swiglu_dense_ws_bytes(T, fs)) : o;
  L.shared_y = fs ? take(sizeof(uint16_t) * static_cast<size_t>(T) * d) : o;
  L.total = o;
  return true;
}

}  // namespace

extern "C" {

int reflex_version(void) { return kVersion; }

const char* reflex_status_string(int status) {
  switch (status) {
    case REFLEX_OK: return "ok";
    case REFLEX_ERR_NULL: return "null pointer";
    case REFLEX_ERR_SHAPE: return "unsupported shape or misaligned pointer";
    case REFLEX_ERR_PARAM: return "invalid hyper-parameter";
    case REFLEX_ERR_WORKSPACE: return "workspace or pair capacity too small";
    case REFLEX_ERR_LAUNCH: return "HIP launch error";
    case REFLEX_ERR_UNSUPPORTED: return "unsupported request";
    default: return "unknown status";
  }
}

size_t reflex_sizeof_alloc_params(void) { return sizeof(reflex_alloc_params); }

int reflex_alloc_preset(int preset, int k_min, int k_max, float w_cf, reflex_alloc_params* out) {
  if (out == nullptr) return REFLEX_ERR_NULL;
  if (preset < REFLEX_PRESET_FULL || preset > REFLEX_PRESET_UNCERTAINTY_ONLY) return REFLEX_ERR_PARAM;
  reflex_alloc_params p;
  p.k_base = 8;          // Section 5.1
  p.delta_role = 4;
  p.delta_cur = 2;
  p.k_min = k_min;
  p.k_max = k_max;
  p.q = 0.25f;
  p.theta = 0.9f;
  p.w_cf = w_cf;
  p.v_ref = 0.01f;
  p.tau = 0.05f;
  p.signal = REFLEX_SIGNAL_FPS;
  switch (preset) {
    case REFLEX_PRESET_RRB_ONLY: p.delta_cur = 0; break;
    case REFLEX_PRESET_FGER_ONLY: p.delta_role = 0; break;
    case REFLEX_PRESET_FRONTIER_ONLY: p.signal = REFLEX_SIGNAL_FRONTIER; break;
    case REFLEX_PRESET_PROGRESS_ONLY: p.signal = REFLEX_SIGNAL_PROGRESS; break;
    case REFLEX_PRESET_CONFIDENCE_ONLY: p.signal = REFLEX_SIGNAL_CONFIDENCE; break;
    case REFLEX_PRESET_UNCERTAINTY_ONLY: p.signal = REFLEX_SIGNAL_UNCERTAINTY; break;
    default: break;
  }
  RFX_TRY(check_params(&p));
  *out = p;
  return REFLEX_OK;
}
size_t reflex_sizeof_moe_args(void) { return sizeof(reflex_moe_args); }

size_t reflex_workspace_size(int T, int E, int d, int f, int f_shared, int k_max) {
  Layout L;
  return make_layout(T, E, d, f, f_shared, k_max, L) ? L.total : 0;
}

size_t reflex_workspace_offset(int T, int E, int d, int f, int f_shared, int k_max, int field) {
  Layout L;
  if (!make_layout(T, E, d, f, f_shared, k_max, L)) return static_cast<size_t>(-1);
  switch (field) {
    case REFLEX_WS_PAIR_OFFSETS: return L.pair_offsets;
    case REFLEX_WS_PAIR_EXPERT: return L.pair_expert;
    case REFLEX_WS_PAIR_WEIGHT: return L.pair_weight;
    case REFLEX_WS_EXPERT_OFFSETS: return L.expert_offsets;
    case REFLEX_WS_SORTED_TOKEN: return L.sorted_token;
    case REFLEX_WS_PAIR_TO_SORTED: return L.pair_to_sorted;
    default: return static_cast<size_t>(-1);
  }
}

size_t reflex_permute_workspace_size(int pair_capacity, int E) {
  if (pair_capacity < 0 || !valid_E(E)) return 0;
  return permute_ws_bytes(pair_capacity, E);
}

size_t reflex_swiglu_workspace_size(int pair_capacity, int E, int f) {
  if (pair_capacity < 0 || !valid_E(E) || !valid_f(f)) return 0;
  return swiglu_ws_bytes(pair_capacity, E, f);
}

int reflex_router_logits(const uint16_t* h, const float* w_router, const float* bias,
                         float* logits, int T, int d, int E, void* stream) {
  RFX_TRY(check_ptrs({h, w_router}, 16));
  RFX_TRY(check_ptr(logits, 4));
  RFX_TRY(check_opt_ptr(bias, 4));
  if (!valid_T(T) || !valid_d(d) || !valid_E(E)) return REFLEX_ERR_SHAPE;
  if (T == 0) return REFLEX_OK;
  return launch_router(h, w_router, bias, logits, T, d, E, static_cast<hipStream_t>(stream));
}

int reflex_assign_budget(const int32_t* block_idx, const uint8_t* masked, const int8_t* hist_len,
                         const float* conf_prev1, const float* conf_prev2,
                         const int32_t* seq_offsets, const int32_t* active_block, int B, int T,
                         const reflex_alloc_params* params, int32_t* k_out, int32_t* pairs_out,
                         double* fps_out, void* stream) {
  RFX_TRY(check_ptrs({masked, hist_len}, 1));
  RFX_TRY(check_ptrs({block_idx, conf_prev1, conf_prev2, seq_offsets, active_block, k_out,
                      pairs_out}, 4));
  RFX_TRY(check_opt_ptr(fps_out, 8));
  RFX_TRY(check_params(params));
  if (!valid_T(T) || B < 0 || B > REFLEX_MAX_TOKENS || (T > 0 && B < 1)) return REFLEX_ERR_SHAPE;
  if (T == 0) return REFLEX_OK;
  return launch_budget(block_idx, masked, hist_len, conf_prev1, conf_prev2, seq_offsets,
                       active_block, B, T, *params, k_out, pairs_out, fps_out,
                       static_cast<hipStream_t>(stream));
}

int reflex_advance_state(const float* conf_t, const int32_t* block_idx, const int32_t* seq_offsets,
                         int B, int T, float theta, int min_commit, uint8_t* masked,
                         int8_t* hist_len, float* conf_prev1, float* conf_prev2,
                         int32_t* active_block, int32_t* remaining, void* stream) {
  RFX_TRY(check_ptrs({masked, hist_len}, 1));
  RFX_TRY(check_ptrs({conf_t, block_idx, seq_offsets, conf_prev1, conf_prev2, active_block}, 4));
  RFX_TRY(check_opt_ptr(remaining, 4));
  if (!valid_T(T) || B < 0 || B > REFLEX_MAX_TOKENS || (T > 0 && B < 1)) return REFLEX_ERR_SHAPE;
  if (!(theta > 0.0f && theta <= 1.0f) || (min_commit != 0 && min_commit != 1))
    return REFLEX_ERR_PARAM;
  if (B == 0) return REFLEX_OK;
  return launch_advance_state(conf_t, block_idx, seq_offsets, B, T, theta, min_commit, masked,
                              hist_len, conf_prev1, conf_prev2, active_block, remaining,
                              static_cast<hipStream_t>(stream));
}

int reflex_count_rule(const float* logits, int T, int E, int rule, float threshold, int k_min,
                      int k_max, int32_t* k_out, int32_t* pairs_out, void* stream) {
  RFX_TRY(check_ptrs({logits, k_out}, 4));
  RFX_TRY(check_opt_ptr(pairs_out, 4));
  RFX_TRY(check_rule(rule, threshold));
  if (!valid_T(T) || !valid_E(E) || !valid_kmax(k_max, E) || k_min < 0 || k_min > k_max)
    return REFLEX_ERR_SHAPE;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (T == 0) return pairs_out ? launch_fill_i32(pairs_out, 0, 1, s) : REFLEX_OK;
  return launch_count_rule(logits, T, E, rule, threshold, k_min, k_max, k_out, pairs_out, s);
}

int reflex_topk_variable(const float* logits, const int32_t* k, int T, int E, int k_max,
                         int norm_topk, int32_t* pair_offsets, int32_t* pair_expert,
                         float* pair_weight, int32_t pair_capacity, void* stream) {
  RFX_TRY(check_ptrs({logits, k, pair_offsets, pair_expert, pair_weight}, 4));
  if (!valid_T(T) || !valid_E(E) || !valid_kmax(k_max, E)) return REFLEX_ERR_SHAPE;
  if (norm_topk != 0 && norm_topk != 1) return REFLEX_ERR_PARAM;
  if (pair_capacity < 0 || static_cast<long long>(T) * k_max > pair_capacity) return REFLEX_ERR_WORKSPACE;
  if (T == 0) return REFLEX_OK;
  hipStream_t s = static_cast<hipStream_t>(stream);
  RFX_TRY(launch_count_scan(k, T, k_max, pair_offsets, nullptr, s));
  return launch_topk(logits, k, T, E, k_max, norm_topk, pair_offsets, pair_expert, pair_weight, s);
}

int reflex_permute(const int32_t* pair_offsets, const int32_t* pair_expert, const int32_t* pairs,
                   int T, int E, int32_t pair_capacity, int32_t* expert_offsets,
                   int32_t* sorted_token, int32_t* pair_to_sorted, void* ws, size_t ws_bytes,
                   void* stream) {
  RFX_TRY(check_ptrs({pair_offsets, pair_expert, pairs, expert_offsets, sorted_token,
                      pair_to_sorted}, 4));
  RFX_TRY(check_ptr(ws, 16));
  if (!valid_T(T) || !valid_E(E) || pair_capacity < 0) return REFLEX_ERR_SHAPE;
  if (ws_bytes < permute_ws_bytes(pair_capacity, E)) return REFLEX_ERR_WORKSPACE;
  if (T == 0) return REFLEX_OK;
  return launch_permute(pair_offsets, pair_expert, pairs, T, E, pair_capacity, expert_offsets,
                        sorted_token, pair_to_sorted, ws, nullptr, static_cast<hipStream_t>(stream));
}

int reflex_grouped_swiglu(const uint16_t* h, const int32_t* sorted_token,
                          const int32_t* expert_offsets, const uint16_t* w_gate,
                          const uint16_t* w_up, const uint16_t* w_down, int T, int E, int d,
                          int f, int32_t pair_capacity, uint16_t* y_sorted, void* ws,
                          size_t ws_bytes, void* stream) {
  RFX_TRY(check_ptrs({h, w_gate, w_up, w_down, y_sorted, ws}, 16));
  RFX_TRY(check_ptrs({sorted_token, expert_offsets}, 4));
  if (!valid_T(T) || !valid_E(E) || !valid_d(d) || !valid_f(f) || pair_capacity < 0)
    return REFLEX_ERR_SHAPE;
  if (ws_bytes < swiglu_ws_bytes(pair_capacity, E, f)) return REFLEX_ERR_WORKSPACE;
  if (T == 0 || pair_capacity == 0) return REFLEX_OK;
  return launch_swiglu_routed(h, sorted_token, expert_offsets, w_gate, w_up, w_down, T, E, d, f,
                              pair_capacity, y_sorted, ws, static_cast<hipStream_t>(stream));
}

int reflex_combine(const uint16_t* y_sorted, const int32_t* pair_offsets,
                   const int32_t* pair_to_sorted, const float* pair_weight,
                   const uint16_t* shared_y, int T, int d, int32_t pair_capacity, uint16_t* out,
                   void* stream) {
  RFX_TRY(check_ptrs({y_sorted, out}, 16));
  RFX_TRY(check_ptrs({pair_offsets, pair_to_sorted, pair_weight}, 4));
  RFX_TRY(check_opt_ptr(shared_y, 16));
  if (!valid_T(T) || !valid_d(d) || pair_capacity < 0) return REFLEX_ERR_SHAPE;
  if (T == 0) return REFLEX_OK;
  return launch_combine(y_sorted, pair_offsets, pair_to_sorted, pair_weight, shared_y, nullptr,
                        nullptr, T, d, pair_capacity, out, static_cast<hipStream_t>(stream));
}

static int moe_forward_impl(const reflex_moe_args* a, void* ws, size_t ws_bytes, void* stream,
                            void* const* ev, bool may_fork = true) {
  if (a == nullptr || ws == nullptr) return REFLEX_ERR_NULL;
  const int T = a->T, E = a->E, d = a->d, f = a->f, fs = a->f_shared;
  if (!valid_T(T) || !valid_E(E) || !valid_d(d) || !valid_f(f) || fs < 0 || (fs && !valid_f(fs)))
    return REFLEX_ERR_SHAPE;
  if (a->norm_topk != 0 && a->norm_topk != 1) return REFLEX_ERR_PARAM;
  RFX_TRY(check_ptrs({a->h, a->w_router, a->out, ws, a->w_gate, a->w_up, a->w_down}, 16));
  for (const void* p : {static_cast<const void*>(a->residual_a), static_cast<const void*>(a->residual_b)})
    RFX_TRY(check_opt_ptr(p, 16));
  for (const void* p : {static_cast<const void*>(a->router_bias), static_cast<const void*>(a->k_in),
                        static_cast<const void*>(a->k_out), static_cast<const void*>(a->pairs_out),
                        static_cast<const void*>(a->logits_out)})
    RFX_TRY(check_opt_ptr(p, 4));
  if (fs) RFX_TRY(check_ptrs({a->ws_gate, a->ws_up, a->ws_down}, 16));
  // pair capacity T * kcap: kcap = uniform_k when set (caller counts are then clamped
  // to it), else params.k_max
  int kcap;
  const bool by_rule = a->k_in == nullptr && a->uniform_k <= 0 && a->k_rule != REFLEX_RULE_BUDGET;
  const bool budget = a->k_in == nullptr && a->uniform_k <= 0 && !by_rule;
  if (by_rule) RFX_TRY(check_rule(a->k_rule, a->k_threshold));
  if (a->uniform_k > 0) {
    kcap = a->uniform_k;
  } else {
    RFX_TRY(check_params(&a->params));
    kcap = a->params.k_max;
  }
  if (!valid_kmax(kcap, E)) return REFLEX_ERR_SHAPE;
  if (budget) {
    RFX_TRY(check_ptrs({a->masked, a->hist_len}, 1));
    RFX_TRY(check_ptrs({a->block_idx, a->seq_offsets, a->active_block, a->conf_prev1,
                        a->conf_prev2}, 4));
    if (a->B < 0 || a->B > REFLEX_MAX_TOKENS || (T > 0 && a->B < 1)) return REFLEX_ERR_SHAPE;
  }
  Layout L;
  if (!make_layout(T, E, d, f, fs, kcap, L)) return REFLEX_ERR_SHAPE;
  if (ws_bytes < L.total) return REFLEX_ERR_WORKSPACE;
  if (T == 0) return REFLEX_OK;

  hipStream_t s = static_cast<hipStream_t>(stream);
  auto mark = [&](int i) {
    if (ev && hipEventRecord(static_cast<hipEvent_t>(ev[i]), s) != hipSuccess) return REFLEX_ERR_LAUNCH;
    return REFLEX_OK;
  };
  char* base = static_cast<char*>(ws);
  auto at = [&](size_t off) { return static_cast<void*>(base + off); };
  const int cap = T * kcap;
  float* logits = a->logits_out ? a->logits_out : static_cast<float*>(at(L.logits));
  int32_t* pair_offsets = static_cast<int32_t*>(at(L.pair_offsets));
  int32_t* pair_expert = static_cast<int32_t*>(at(L.pair_expert));
  float* pair_weight = static_cast<float*>(at(L.pair_weight));
  int32_t* expert_offsets = static_cast<int32_t*>(at(L.expert_offsets));
  int32_t* sorted_token = static_cast<int32_t*>(at(L.sorted_token));
  int32_t* pair_to_sorted = static_cast<int32_t*>(at(L.pair_to_sorted));
  uint16_t* y = static_cast<uint16_t*>(at(L.y));
  void* gws = at(L.swiglu);

  // how the pairs get sorted: inside the route launch (its completion counter is zeroed
  // by the router launch), by the block-sort launches, or by the permutation launches
  const bool fused_sort = route_fused_sorts(T, E), block_sort = route_block_sorts(T, E);
  int32_t* done = fused_sort ? static_cast<int32_t*>(at(L.done)) : nullptr;
  int32_t* route_hist =
      fused_sort || block_sort ? static_cast<int32_t*>(at(L.route_hist)) : nullptr;
  RFX_TRY(mark(0));
  // The shared expert reads only h: on the side stream it runs beside the routing
  // launches, which leave most CUs idle, and joins the caller's stream before the combine.
  // The stage-timed variant keeps it in line, so that its stage time is its own.
  uint16_t* shared_y_buf = fs ? static_cast<uint16_t*>(at(L.shared_y)) : nullptr;
  SideFork side(s);      // declared before any early return below: its exit joins
  if (fs && ev == nullptr && may_fork && side.fork())
    RFX_TRY(launch_swiglu_dense(a->h, a->ws_gate, a->ws_up, a->ws_down, T, d, fs, shared_y_buf,
                                at(L.shared_act), side.side()));
  const int32_t* k = a->k_in;
  // small layers: scores and counts in one launch (independent work side by side)
  const bool front = budget && front_fits(T, d);
  // score source of the route kernel: finished scores, or the front launch's partials
  const float* scores = logits;
  int n_parts = 1;
  const float* part_bias = nullptr;
  float* scores_out = nullptr;
  if (front) {
    int32_t* kb = a->k_out ? a->k_out : static_cast<int32_t*>(at(L.k));
    float* parts = static_cast<float*>(at(L.logits));
    RFX_TRY(launch_front(a->h, a->w_router, parts, T, d, E, a->block_idx, a->masked, a->hist_len,
                         a->conf_prev1, a->conf_prev2, a->seq_offsets, a->active_block, a->B,
                         a->params, kb, s, done));
    k = kb;
    scores = parts;
    n_parts = front_slices(d);
    part_bias = a->router_bias;
    scores_out = a->logits_out;
  } else {
    // partial scores for the route kernel to add, unless a count rule reads the scores
    const int ns = by_rule ? 1 : router_slices(T, d, E);
    if (ns > 1) {
      float* parts = static_cast<float*>(at(L.logits));
      RFX_TRY(launch_router(a->h, a->w_router, a->router_bias, parts, T, d, E, s, done, ns));
      scores = parts;
      n_parts = ns;
      part_bias = a->router_bias;
      scores_out = a->logits_out;
    } else {
      RFX_TRY(launch_router(a->h, a->w_router, a->router_bias, logits, T, d, E, s, done));
    }
  }
  RFX_TRY(mark(1));
  if (k == nullptr) {
    int32_t* kb = a->k_out ? a->k_out : static_cast<int32_t*>(at(L.k));
    if (a->uniform_k > 0) {
      RFX_TRY(launch_fill_i32(kb, a->uniform_k, T, s));
    } else if (by_rule) {
      RFX_TRY(launch_count_rule(logits, T, E, a->k_rule, a->k_threshold, a->params.k_min,
                                a->params.k_max, kb, nullptr, s));
    } else {
      RFX_TRY(launch_budget(a->block_idx, a->masked, a->hist_len, a->conf_prev1, a->conf_prev2,
                            a->seq_offsets, a->active_block, a->B, T, a->params, kb, nullptr,
                            nullptr, s));
    }
    k = kb;
  }
  RFX_TRY(mark(2));
  // pair offsets and TopK in one launch (P lives in pair_offsets[T]); for layers with
  // at most RF_HIST_MAX (token block, expert) counts the pairs are also sorted there,
  // otherwise by the permutation launches.  Either way the sort writes the GEMM tile
  // plan at the head of gws.
  RFX_TRY(launch_route_fused(scores, n_parts, static_cast<size_t>(T) * E, part_bias, scores_out, k,
                             T, E, kcap, a->norm_topk, pair_offsets, pair_expert,
                             pair_weight, a->pairs_out, done, route_hist,
                             expert_offsets, sorted_token, pair_to_sorted,
                             static_cast<int32_t*>(gws), s));
  RFX_TRY(mark(3));
  if (block_sort)
    RFX_TRY(launch_block_sort(pair_offsets, pair_expert, T, E, cap, route_hist, expert_offsets,
                              sorted_token, pair_to_sorted, static_cast<int32_t*>(gws), s));
  else if (!fused_sort)
    RFX_TRY(launch_permute(pair_offsets, pair_expert, pair_offsets + T, T, E, cap, expert_offsets,
                           sorted_token, pair_to_sorted, at(L.perm), static_cast<int32_t*>(gws), s));
  RFX_TRY(mark(4));
  RFX_TRY(launch_swiglu_up(a->h, sorted_token, expert_offsets, a->w_gate, a->w_up, T, E, d, f,
                           cap, gws, s));
  RFX_TRY(mark(5));
  RFX_TRY(launch_swiglu_down(expert_offsets, a->w_down, E, d, f, cap, y, gws, s));
  RFX_TRY(mark(6));
  const uint16_t* shared_y = nullptr;
  if (fs && side.forked()) {
    RFX_TRY(side.join());
    shared_y = shared_y_buf;
  } else if (fs) {
    uint16_t* sy = shared_y_buf;
    RFX_TRY(launch_swiglu_dense(a->h, a->ws_gate, a->ws_up, a->ws_down, T, d, fs, sy,
                                at(L.shared_act), s));
    shared_y = sy;
  }
  RFX_TRY(mark(7));
  RFX_TRY(launch_combine(y, pair_offsets, pair_to_sorted, pair_weight, shared_y, a->residual_a,
                         a->residual_b, T, d, cap, a->out, s));
  return mark(8);
}

int reflex_moe_forward(const reflex_moe_args* a, void* ws, size_t ws_bytes, void* stream) {
  return moe_forward_impl(a, ws, ws_bytes, stream, nullptr);
}

// The device scratch of reflex_moe_forward_noalloc: one copy per device, held from the
// library's load on that device until the process ends.  In host code `scratch` names
// a host-side stand-in, not device memory: its device address comes from
// hipGetSymbolAddress, per device, and only that address is ever passed on.
static __device__ __align__(256) unsigned char scratch[REFLEX_NOALLOC_SCRATCH_BYTES];

// Device address of `scratch` on the current device, looked up once per device (with
// that device current) and kept; NULL if the lookup fails.
static void* noalloc_scratch() {
  static std::mutex mu;
  static void* ptrs[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return nullptr;
  std::lock_guard<std::mutex> g(mu);
  if (ptrs[dev] == nullptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return nullptr;
    ptrs[dev] = p;
  }
  return ptrs[dev];
}

int reflex_moe_forward_noalloc(const reflex_moe_args* a, void* stream) {
  if (a == nullptr) return REFLEX_ERR_NULL;
  void* ws = noalloc_scratch();
  if (ws == nullptr) return REFLEX_ERR_LAUNCH;
  // the shared expert stays on `stream`: forking it would create a stream and events
  return moe_forward_impl(a, ws, REFLEX_NOALLOC_SCRATCH_BYTES, stream, nullptr, false);
}

int reflex_moe_forward_timed(const reflex_moe_args* a, void* ws, size_t ws_bytes, void* stream,
                             void* const* stage_events, int n_stage_events) {
  if (stage_events == nullptr) return REFLEX_ERR_NULL;
  if (n_stage_events != REFLEX_N_STAGE_EVENTS) return REFLEX_ERR_SHAPE;
  for (int i = 0; i < n_stage_events; ++i)
    if (stage_events[i] == nullptr) return REFLEX_ERR_NULL;
  return moe_forward_impl(a, ws, ws_bytes, stream, stage_events);
}

}  // extern "C"
