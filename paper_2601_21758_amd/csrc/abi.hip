// C ABI of the EWSJF scheduler core: argument checks on the host, then
// launches on the caller's stream.  Nothing here allocates device memory or
// synchronizes, except ewsjf_table_upload (a set-up call, documented).
#include <hip/hip_runtime.h>

#include <atomic>
#include <cfloat>
#include <cmath>
#include <cstddef>
#include <cstring>
#include <memory>
#include <mutex>

#include "ewsjf.h"
#include "ewsjf_launch.h"

namespace {

static_assert(offsetof(ewsjf_queue_table, lut) % 16 == 0, "routing lut must be 16-byte aligned");
static_assert(offsetof(ewsjf_queue_table, route) % 16 == 0, "routing map must be 16-byte aligned");
static_assert(sizeof(ewsjf_partition_params) == 40, "ABI layout");
static_assert(sizeof(ewsjf_cost) == 24, "ABI layout");

constexpr int kMaxDevices = 64;
std::atomic<int> g_arch_ok[kMaxDevices];  // 0 unknown, 1 gfx950, -1 other/no device

ewsjf_status check_device() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return EWSJF_ERR_DEVICE;
  if (dev >= kMaxDevices) return EWSJF_ERR_DEVICE;
  int st = g_arch_ok[dev].load(std::memory_order_relaxed);
  if (st == 0) {
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return EWSJF_ERR_DEVICE;
    st = std::strncmp(prop.gcnArchName, "gfx950", 6) == 0 ? 1 : -1;
    g_arch_ok[dev].store(st, std::memory_order_relaxed);
  }
  return st == 1 ? EWSJF_OK : EWSJF_ERR_DEVICE;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

// The kernels evaluate C_prefill and the reciprocal of (b + 1) C_prefill(b)
// in binary32: c0 must be a normal binary32 value and c1, c2 zero or normal,
// and (b + 1) C(b) must stay at most 1 / (2 FLT_MIN) up to the longest int32
// length (it grows with b), so that C is finite and nonzero and the
// reciprocal a normal number for every request.
bool f32_normal(double x) { return x >= (double)FLT_MIN && x <= (double)FLT_MAX; }
bool cost_ok(const ewsjf_cost* c) {
  if (!(f32_normal(c->c0) && (c->c1 == 0.0 || f32_normal(c->c1)) && (c->c2 == 0.0 || f32_normal(c->c2))))
    return false;
  const double b = 2147483647.0;
  return (b + 1.0) * (c->c0 + c->c1 * b + c->c2 * b * b) <= 0.5 / (double)FLT_MIN;
}

bool params_ok(const ewsjf_partition_params* p) {
  if (p->init_mode != EWSJF_INIT_EQUAL_WIDTH && p->init_mode != EWSJF_INIT_KMEANS3) return false;
  if (p->init_mode == EWSJF_INIT_EQUAL_WIDTH && (p->init_queues < 1 || p->init_queues > EWSJF_MAX_LEN)) return false;
  if (p->max_queues < 1 || p->max_queues > EWSJF_MAX_QUEUES) return false;
  if (p->min_width < 0) return false;
  if (p->max_len < 1 || p->max_len > EWSJF_MAX_LEN) return false;
  if (p->gap_mode != EWSJF_GAPS_DISTINCT && p->gap_mode != EWSJF_GAPS_MULTISET) return false;
  if (!(p->alpha > 1.0) || !std::isfinite(p->alpha)) return false;
  if (!(p->eps > 0.0) || !std::isfinite(p->eps)) return false;
  return true;
}

constexpr int64_t kMaxN = 0x7fffffffLL;  // request ids are int32

ewsjf_status launched(hipError_t e) { return e == hipSuccess ? EWSJF_OK : EWSJF_ERR_LAUNCH; }

}  // namespace

extern "C" {

int32_t ewsjf_version(void) { return 10000; }

const char* ewsjf_status_string(ewsjf_status s) {
  switch (s) {
    case EWSJF_OK: return "ok";
    case EWSJF_ERR_NULL: return "a required pointer is NULL";
    case EWSJF_ERR_ARG: return "a size or parameter is out of range";
    case EWSJF_ERR_WORKSPACE: return "workspace too small";
    case EWSJF_ERR_LAUNCH: return "kernel launch or copy failed";
    case EWSJF_ERR_ALIGN: return "a pool array is not 16-byte aligned";
    case EWSJF_ERR_DEVICE: return "no usable gfx950 device is current";
  }
  return "unknown status";
}

size_t ewsjf_queue_table_bytes(void) { return sizeof(ewsjf_queue_table); }

size_t ewsjf_workspace_bytes(int op, int64_t n, int32_t n_theta, int32_t B, const ewsjf_partition_params* p) {
  if (n < 0 || n > kMaxN) return 0;
  if (op == EWSJF_OP_PARTITION) {
    if (p == nullptr || !params_ok(p)) return 0;
    return ewsjf::partition_ws_bytes(n, *p);
  }
  if (op == EWSJF_OP_SELECT || op == EWSJF_OP_STEP) {
    if (n_theta < 1 || n_theta > EWSJF_MAX_THETA || B < 1 || B > EWSJF_MAX_B) return 0;
    return op == EWSJF_OP_STEP ? ewsjf::plan_step(n, n_theta, B).ws_bytes : ewsjf::plan_select(n, n_theta, B).ws_bytes;
  }
  if (op == EWSJF_OP_TRIAL) {
    if (n_theta < 1 || n_theta > EWSJF_MAX_THETA || B < 1 || B > EWSJF_MAX_B) return 0;
    return ewsjf::plan_trial(n, n_theta, B).ws_bytes;
  }
  if (op == EWSJF_OP_TACTICAL) {
    if (B < 1 || B > EWSJF_MAX_B) return 0;
    return ewsjf::tactical_ws_bytes(n, B);
  }
  return 0;
}

ewsjf_status ewsjf_table_upload(const ewsjf_queue_table* host_table, void* table, hipStream_t stream) {
  if (host_table == nullptr || table == nullptr) return EWSJF_ERR_NULL;
  const ewsjf_queue_table& h = *host_table;
  if (h.k < 1 || h.k > EWSJF_MAX_QUEUES || h.max_len < 1 || h.max_len > EWSJF_MAX_LEN) return EWSJF_ERR_ARG;
  for (int i = 0; i < h.k - 1; ++i) {
    if (h.bounds[i] < 1 || h.bounds[i] > h.max_len) return EWSJF_ERR_ARG;
    if (i > 0 && h.bounds[i] <= h.bounds[i - 1]) return EWSJF_ERR_ARG;
  }
  for (int i = 0; i < h.k; ++i)
    if (!std::isfinite(h.mean[i])) return EWSJF_ERR_ARG;
  if (h.gapped != 0 && h.gapped != 1) return EWSJF_ERR_ARG;
  if (h.gapped)
    for (int i = 0; i < h.k; ++i)
      if (h.lo[i] < 1 || h.hi[i] < h.lo[i] || h.hi[i] > h.max_len || (i > 0 && h.lo[i] <= h.hi[i - 1]))
        return EWSJF_ERR_ARG;
  // Contiguous: queue i > 0 starts at its bound, the table Refine-and-Prune
  // writes, so a later removal of a queue (ewsjf_tactical_step) that deletes
  // the boundary it shares with its absorber leaves lo consistent.
  if (!h.gapped)
    for (int i = 1; i < h.k; ++i)
      if (h.lo[i] != h.bounds[i - 1]) return EWSJF_ERR_ARG;
  const ewsjf_status ds = check_device();
  if (ds != EWSJF_OK) return ds;
  std::unique_ptr<ewsjf_queue_table> copy(new ewsjf_queue_table(h));
  copy->n_distinct = copy->n_coarse = copy->n_leaves = 0;
  const size_t head = offsetof(ewsjf_queue_table, lut);
  if (hipMemcpyAsync(table, copy.get(), head, hipMemcpyHostToDevice, stream) != hipSuccess) return EWSJF_ERR_LAUNCH;
  if (ewsjf::launch_build_lut(static_cast<ewsjf_queue_table*>(table), stream) != hipSuccess)
    return EWSJF_ERR_LAUNCH;
  // The host copy must outlive the transfer.
  if (hipStreamSynchronize(stream) != hipSuccess) return EWSJF_ERR_LAUNCH;
  return EWSJF_OK;
}

ewsjf_status ewsjf_partition(const int32_t* window, int64_t n_window, const ewsjf_partition_params* p, void* table,
                             void* ws, size_t ws_bytes, hipStream_t stream) {
  if (window == nullptr || p == nullptr || table == nullptr || ws == nullptr) return EWSJF_ERR_NULL;
  if (n_window < 1 || n_window > kMaxN || !params_ok(p)) return EWSJF_ERR_ARG;
  if (ws_bytes < ewsjf::partition_ws_bytes(n_window, *p)) return EWSJF_ERR_WORKSPACE;
  if (!aligned16(ws)) return EWSJF_ERR_ALIGN;
  const ewsjf_status ds = check_device();
  if (ds != EWSJF_OK) return ds;
  return launched(
      ewsjf::launch_partition(window, n_window, *p, static_cast<ewsjf_queue_table*>(table), ws, stream));
}

ewsjf_status ewsjf_ring_insert(int32_t* ring_len, float* ring_arrival, int64_t capacity, int64_t pos,
                               int32_t* window, int64_t window_cap, int64_t wpos, const int32_t* new_len,
                               const float* new_arrival, int64_t n, hipStream_t stream) {
  if (n > 0 && (ring_len == nullptr || ring_arrival == nullptr || new_len == nullptr || new_arrival == nullptr))
    return EWSJF_ERR_NULL;
  if (window_cap > 0 && window == nullptr) return EWSJF_ERR_NULL;
  if (capacity < 1 || capacity > kMaxN || pos < 0 || pos >= capacity || n < 0 || n > capacity) return EWSJF_ERR_ARG;
  if (window_cap < 0 || window_cap > kMaxN || wpos < 0 || (window_cap > 0 && (wpos >= window_cap || n > window_cap)) ||
      (window_cap == 0 && wpos != 0))
    return EWSJF_ERR_ARG;
  if (n == 0) return EWSJF_OK;
  const ewsjf_status ds = check_device();
  if (ds != EWSJF_OK) return ds;
  return launched(ewsjf::launch_ring_insert(ring_len, ring_arrival, capacity, pos, window, window_cap, wpos, new_len,
                                            new_arrival, n, stream));
}

ewsjf_status ewsjf_window_histogram(const int32_t* ring, int64_t ring_cap, int64_t begin, int64_t n, int32_t max_len,
                                    uint32_t* hist, hipStream_t stream) {
  if (hist == nullptr || (n > 0 && ring == nullptr)) return EWSJF_ERR_NULL;
  if (ring_cap < 0 || ring_cap > kMaxN || n < 0 || n > ring_cap || begin < 0 ||
      begin >= (ring_cap > 0 ? ring_cap : 1) || max_len < 1 || max_len > EWSJF_MAX_LEN)
    return EWSJF_ERR_ARG;
  const ewsjf_status ds = check_device();
  if (ds != EWSJF_OK) return ds;
  return launched(ewsjf::launch_window_histogram(ring, ring_cap, begin, n, max_len, hist, stream));
}

ewsjf_status ewsjf_window_advance(const int32_t* ring, int64_t ring_cap, int64_t add_pos, int64_t sub_pos, int64_t n,
                                  int32_t max_len, uint32_t* hist, hipStream_t stream) {
  if (n > 0 && (ring == nullptr || hist == nullptr)) return EWSJF_ERR_NULL;
  if (ring_cap < 1 || ring_cap > kMaxN || n < 0 || n > ring_cap || add_pos < 0 || add_pos >= ring_cap ||
      sub_pos < 0 || sub_pos >= ring_cap || max_len < 1 || max_len > EWSJF_MAX_LEN)
    return EWSJF_ERR_ARG;
  if (n == 0) return EWSJF_OK;
  const ewsjf_status ds = check_device();
  if (ds != EWSJF_OK) return ds;
  return launched(ewsjf::launch_window_advance(ring, ring_cap, add_pos, sub_pos, n, max_len, hist, stream));
}

ewsjf_status ewsjf_partition_hist(const uint32_t* hist, const ewsjf_partition_params* p, void* table, void* ws,
                                  size_t ws_bytes, hipStream_t stream) {
  if (hist == nullptr || p == nullptr || table == nullptr || ws == nullptr) return EWSJF_ERR_NULL;
  if (!params_ok(p)) return EWSJF_ERR_ARG;
  if (ws_bytes < ewsjf::partition_ws_bytes(0, *p)) return EWSJF_ERR_WORKSPACE;
  if (!aligned16(ws)) return EWSJF_ERR_ALIGN;
  const ewsjf_status ds = check_device();
  if (ds != EWSJF_OK) return ds;
  return launched(ewsjf::launch_partition_hist(hist, *p, static_cast<ewsjf_queue_table*>(table), ws, stream));
}

ewsjf_status ewsjf_trial_step(int32_t* len, float* arrival, int64_t capacity, int32_t n_pools, int64_t pos,
                              const int32_t* new_len, const float* new_arrival, int64_t n_new, float now,
                              const void* table, const ewsjf_theta* theta, const ewsjf_cost* cost, int32_t B,
                              int32_t* ids, float* top, int32_t* n_sel, double* stats, int64_t* queue_admits, void* ws,
                              size_t ws_bytes, hipStream_t stream) {
  if (len == nullptr || arrival == nullptr || table == nullptr || theta == nullptr || cost == nullptr ||
      ids == nullptr || top == nullptr || n_sel == nullptr || stats == nullptr || queue_admits == nullptr ||
      ws == nullptr || (n_new > 0 && (new_len == nullptr || new_arrival == nullptr)))
    return EWSJF_ERR_NULL;
  if (capacity < 4 || capacity > kMaxN || capacity % 4 != 0 || n_pools < 1 || n_pools > EWSJF_MAX_THETA ||
      pos < 0 || pos >= capacity || n_new < 0 || n_new > capacity || B < 1 || B > EWSJF_MAX_B || !cost_ok(cost) ||
      !std::isfinite(now))
    return EWSJF_ERR_ARG;
  if (ws_bytes < ewsjf::plan_trial(capacity, n_pools, B).ws_bytes) return EWSJF_ERR_WORKSPACE;
  if (!aligned16(len) || !aligned16(arrival) || !aligned16(ws)) return EWSJF_ERR_ALIGN;
  const ewsjf_status ds = check_device();
  if (ds != EWSJF_OK) return ds;
  const auto* tab = static_cast<const ewsjf_queue_table*>(table);
  const hipError_t e = ewsjf::launch_trial_select(len, arrival, capacity, n_pools, pos, new_len, new_arrival, n_new,
                                                  now, tab, theta, *cost, B, ids, top, n_sel, ws, stream);
  if (e != hipSuccess) return EWSJF_ERR_LAUNCH;
  return launched(ewsjf::launch_trial_stats(len, arrival, capacity, n_pools, now, tab, B, ids, n_sel, stats,
                                            queue_admits, stream));
}

ewsjf_status ewsjf_trial_finish(const int32_t* len, const float* arrival, int64_t capacity, int32_t n_pools, float now,
                                const void* table, const int64_t* queue_admits, const double* lambda, double* stats,
                                double* reward, hipStream_t stream) {
  if (len == nullptr || arrival == nullptr || table == nullptr || queue_admits == nullptr || lambda == nullptr ||
      stats == nullptr || reward == nullptr)
    return EWSJF_ERR_NULL;
  if (capacity < 4 || capacity > kMaxN || capacity % 4 != 0 || n_pools < 1 || n_pools > EWSJF_MAX_THETA ||
      !std::isfinite(now))
    return EWSJF_ERR_ARG;
  for (int i = 0; i < 4; ++i)
    if (!std::isfinite(lambda[i])) return EWSJF_ERR_ARG;
  const ewsjf_status ds = check_device();
  if (ds != EWSJF_OK) return ds;
  return launched(ewsjf::launch_trial_finish(len, arrival, capacity, n_pools, now,
                                             static_cast<const ewsjf_queue_table*>(table), queue_admits, lambda, stats,
                                             reward, stream));
}

ewsjf_status ewsjf_dispatch(const int32_t* len, const float* arrival, int64_t n, void* table, int32_t bubble_width,
                            int32_t max_queues, int32_t* qid, hipStream_t stream) {
  if (table == nullptr || (n > 0 && (len == nullptr || arrival == nullptr || qid == nullptr))) return EWSJF_ERR_NULL;
  if (n < 0 || n > EWSJF_MAX_DISPATCH || bubble_width < 1 || max_queues < 1 || max_queues > EWSJF_MAX_QUEUES)
    return EWSJF_ERR_ARG;
  const ewsjf_status ds = check_device();
  if (ds != EWSJF_OK) return ds;
  return launched(ewsjf::launch_dispatch(len, arrival, (int)n, static_cast<ewsjf_queue_table*>(table), bubble_width,
                                         max_queues, qid, stream));
}

ewsjf_status ewsjf_route(const int32_t* len, int64_t n, const void* table, int32_t* qid, hipStream_t stream) {
  if (table == nullptr || (n > 0 && (len == nullptr || qid == nullptr))) return EWSJF_ERR_NULL;
  if (n < 0 || n > kMaxN) return EWSJF_ERR_ARG;
  if (n == 0) return EWSJF_OK;
  if (!aligned16(len) || !aligned16(qid)) return EWSJF_ERR_ALIGN;
  const ewsjf_status ds = check_device();
  if (ds != EWSJF_OK) return ds;
  return launched(ewsjf::launch_route(len, n, static_cast<const ewsjf_queue_table*>(table), qid, stream));
}

ewsjf_status ewsjf_score(const int32_t* len, const float* arrival, int64_t n, float now, const void* table,
                         const ewsjf_theta* theta, int32_t n_theta, const ewsjf_cost* cost, float* score,
                         hipStream_t stream) {
  if (table == nullptr || theta == nullptr || cost == nullptr ||
      (n > 0 && (len == nullptr || arrival == nullptr || score == nullptr)))
    return EWSJF_ERR_NULL;
  if (n < 0 || n > kMaxN || n_theta < 1 || n_theta > EWSJF_MAX_THETA || !cost_ok(cost) || !std::isfinite(now))
    return EWSJF_ERR_ARG;
  if (n == 0) return EWSJF_OK;
  if (!aligned16(len) || !aligned16(arrival) || !aligned16(score)) return EWSJF_ERR_ALIGN;
  const ewsjf_status ds = check_device();
  if (ds != EWSJF_OK) return ds;
  return launched(ewsjf::launch_score(len, arrival, n, now, static_cast<const ewsjf_queue_table*>(table), theta,
                                      n_theta, *cost, score, stream));
}

ewsjf_status ewsjf_select(const float* score, int64_t n, int32_t n_theta, int32_t B, int32_t* ids, float* top,
                          int32_t* n_sel, void* ws, size_t ws_bytes, hipStream_t stream) {
  if ((n > 0 && score == nullptr) || ids == nullptr || top == nullptr || n_sel == nullptr || ws == nullptr)
    return EWSJF_ERR_NULL;
  if (n < 0 || n > kMaxN || n_theta < 1 || n_theta > EWSJF_MAX_THETA || B < 1 || B > EWSJF_MAX_B)
    return EWSJF_ERR_ARG;
  if (ws_bytes < ewsjf::plan_select(n, n_theta, B).ws_bytes) return EWSJF_ERR_WORKSPACE;
  if ((n > 0 && !aligned16(score)) || !aligned16(ws)) return EWSJF_ERR_ALIGN;
  const ewsjf_status ds = check_device();
  if (ds != EWSJF_OK) return ds;
  return launched(ewsjf::launch_select(score, n, n_theta, B, ids, top, n_sel, ws, stream));
}

ewsjf_status ewsjf_step_timed(int32_t* len, const float* arrival, int64_t n, float now, const void* table,
                              const ewsjf_theta* theta, int32_t n_theta, const ewsjf_cost* cost, int32_t B,
                              int32_t flags, int32_t* ids, float* top, int32_t* n_sel, void* ws, size_t ws_bytes,
                              hipStream_t stream, hipEvent_t* marks) {
  if ((n > 0 && (len == nullptr || arrival == nullptr)) || table == nullptr || theta == nullptr ||
      cost == nullptr || ids == nullptr || top == nullptr || n_sel == nullptr || ws == nullptr)
    return EWSJF_ERR_NULL;
  if (n < 0 || n > kMaxN || n_theta < 1 || n_theta > EWSJF_MAX_THETA || B < 1 || B > EWSJF_MAX_B ||
      !cost_ok(cost) || !std::isfinite(now))
    return EWSJF_ERR_ARG;
  if ((flags & ~EWSJF_STEP_TOMBSTONE) != 0) return EWSJF_ERR_ARG;
  if ((flags & EWSJF_STEP_TOMBSTONE) && n_theta != 1) return EWSJF_ERR_ARG;
  if (ws_bytes < ewsjf::plan_step(n, n_theta, B).ws_bytes) return EWSJF_ERR_WORKSPACE;
  if ((n > 0 && (!aligned16(len) || !aligned16(arrival))) || !aligned16(ws)) return EWSJF_ERR_ALIGN;
  const ewsjf_status ds = check_device();
  if (ds != EWSJF_OK) return ds;
  return launched(ewsjf::launch_step(len, arrival, n, now, static_cast<const ewsjf_queue_table*>(table), theta,
                                     n_theta, *cost, B, (flags & EWSJF_STEP_TOMBSTONE) ? len : nullptr, ids, top,
                                     n_sel, ws, stream, marks));
}

ewsjf_status ewsjf_step(int32_t* len, const float* arrival, int64_t n, float now, const void* table,
                        const ewsjf_theta* theta, int32_t n_theta, const ewsjf_cost* cost, int32_t B, int32_t flags,
                        int32_t* ids, float* top, int32_t* n_sel, void* ws, size_t ws_bytes, hipStream_t stream) {
  return ewsjf_step_timed(len, arrival, n, now, table, theta, n_theta, cost, B, flags, ids, top, n_sel, ws, ws_bytes,
                          stream, nullptr);
}

ewsjf_status ewsjf_tactical_step(int32_t* len, const float* arrival, int64_t n, float now, void* table,
                                 const ewsjf_theta* theta, const ewsjf_cost* cost, int32_t B, int32_t empty_threshold,
                                 int32_t* empty_cnt, double eps, int32_t flags, int32_t* ids, int32_t* n_sel,
                                 int32_t* q_prim, float* head_score, int32_t* removed, void* ws, size_t ws_bytes,
                                 hipStream_t stream) {
  if ((n > 0 && (len == nullptr || arrival == nullptr)) || table == nullptr || theta == nullptr || cost == nullptr ||
      empty_cnt == nullptr || ids == nullptr || n_sel == nullptr || q_prim == nullptr || ws == nullptr)
    return EWSJF_ERR_NULL;
  if (n < 0 || n > kMaxN || B < 1 || B > EWSJF_MAX_B || empty_threshold < 0 || !cost_ok(cost) ||
      !std::isfinite(now) || !(eps > 0.0) || !std::isfinite(eps))
    return EWSJF_ERR_ARG;
  if ((flags & ~EWSJF_STEP_TOMBSTONE) != 0) return EWSJF_ERR_ARG;
  if (ws_bytes < ewsjf::tactical_ws_bytes(n, B)) return EWSJF_ERR_WORKSPACE;
  if ((n > 0 && (!aligned16(len) || !aligned16(arrival))) || !aligned16(ws)) return EWSJF_ERR_ALIGN;
  const ewsjf_status ds = check_device();
  if (ds != EWSJF_OK) return ds;
  return launched(ewsjf::launch_tactical_step(len, arrival, n, now, static_cast<ewsjf_queue_table*>(table), theta,
                                              *cost, B, empty_threshold, empty_cnt, eps,
                                              (flags & EWSJF_STEP_TOMBSTONE) ? len : nullptr, ids, n_sel, q_prim,
                                              head_score, removed, ws, stream));
}

ewsjf_status ewsjf_ring_step(int32_t* ring_len, float* ring_arrival, int64_t capacity, int64_t pos, int32_t* window,
                             int64_t window_cap, int64_t wpos, const int32_t* new_len, const float* new_arrival,
                             int64_t n_new, float now, const void* table, const ewsjf_theta* theta,
                             const ewsjf_cost* cost, int32_t B, int32_t flags, int32_t* ids, float* top,
                             int32_t* n_sel, void* ws, size_t ws_bytes, hipStream_t stream) {
  if (ring_len == nullptr || ring_arrival == nullptr || table == nullptr || theta == nullptr || cost == nullptr ||
      ids == nullptr || top == nullptr || n_sel == nullptr || ws == nullptr)
    return EWSJF_ERR_NULL;
  if (n_new > 0 && (new_len == nullptr || new_arrival == nullptr)) return EWSJF_ERR_NULL;
  if (window_cap > 0 && window == nullptr) return EWSJF_ERR_NULL;
  if (capacity < 1 || capacity > kMaxN || pos < 0 || pos >= capacity || n_new < 0 || n_new > capacity)
    return EWSJF_ERR_ARG;
  if (window_cap < 0 || window_cap > kMaxN || wpos < 0 || (window_cap > 0 && (wpos >= window_cap || n_new > window_cap)) ||
      (window_cap == 0 && wpos != 0))
    return EWSJF_ERR_ARG;
  if (B < 1 || B > EWSJF_MAX_B || !cost_ok(cost) || !std::isfinite(now)) return EWSJF_ERR_ARG;
  if ((flags & ~EWSJF_STEP_TOMBSTONE) != 0) return EWSJF_ERR_ARG;
  if (ws_bytes < ewsjf::plan_select(capacity, 1, B).ws_bytes) return EWSJF_ERR_WORKSPACE;
  if (!aligned16(ring_len) || !aligned16(ring_arrival) || !aligned16(ws)) return EWSJF_ERR_ALIGN;
  const ewsjf_status ds = check_device();
  if (ds != EWSJF_OK) return ds;
  return launched(ewsjf::launch_ring_step(ring_len, ring_arrival, capacity, pos, window, window_cap, wpos, new_len,
                                          new_arrival, n_new, now, static_cast<const ewsjf_queue_table*>(table),
                                          theta, *cost, B, (flags & EWSJF_STEP_TOMBSTONE) ? ring_len : nullptr, ids,
                                          top, n_sel, ws, stream));
}

// ---------------------------------------------------------------------------
// ewsjf_step_static: ewsjf_step with its workspace in a fixed device array,
// for callers that cannot allocate.  Each device holds its own copy of
// `scratch` (until the process ends); host code reaches it only through the
// device address looked up on the first call on that device.
// ---------------------------------------------------------------------------
static __device__ __align__(256) uint8_t scratch[EWSJF_STATIC_SCRATCH_BYTES];

static std::atomic<void*> g_scratch_ptr[kMaxDevices];
static std::mutex g_scratch_mu;

static ewsjf_status static_scratch(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return EWSJF_ERR_DEVICE;
  void* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (p == nullptr) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    p = g_scratch_ptr[dev].load(std::memory_order_relaxed);
    if (p == nullptr) {
      if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return EWSJF_ERR_LAUNCH;
      g_scratch_ptr[dev].store(p, std::memory_order_release);
    }
  }
  *out = p;
  return EWSJF_OK;
}

ewsjf_status ewsjf_step_static(int32_t* len, const float* arrival, int64_t n, float now, const void* table,
                               const ewsjf_theta* theta, int32_t n_theta, const ewsjf_cost* cost, int32_t B,
                               int32_t flags, int32_t* ids, float* top, int32_t* n_sel, hipStream_t stream) {
  if ((n > 0 && (len == nullptr || arrival == nullptr)) || table == nullptr || theta == nullptr ||
      cost == nullptr || ids == nullptr || top == nullptr || n_sel == nullptr)
    return EWSJF_ERR_NULL;
  if (n < 0 || n > kMaxN || n_theta < 1 || n_theta > EWSJF_MAX_THETA || B < 1 || B > EWSJF_MAX_B ||
      !cost_ok(cost) || !std::isfinite(now))
    return EWSJF_ERR_ARG;
  if ((flags & ~EWSJF_STEP_TOMBSTONE) != 0) return EWSJF_ERR_ARG;
  if ((flags & EWSJF_STEP_TOMBSTONE) && n_theta != 1) return EWSJF_ERR_ARG;
  const size_t need = ewsjf::plan_step(n, n_theta, B).ws_bytes;
  if (need > (size_t)EWSJF_STATIC_SCRATCH_BYTES) return EWSJF_ERR_WORKSPACE;
  if (n > 0 && (!aligned16(len) || !aligned16(arrival))) return EWSJF_ERR_ALIGN;
  const ewsjf_status ds = check_device();
  if (ds != EWSJF_OK) return ds;
  void* ws = nullptr;
  const ewsjf_status ss = static_scratch(&ws);
  if (ss != EWSJF_OK) return ss;
  return launched(ewsjf::launch_step(len, arrival, n, now, static_cast<const ewsjf_queue_table*>(table), theta,
                                     n_theta, *cost, B, (flags & EWSJF_STEP_TOMBSTONE) ? len : nullptr, ids, top,
                                     n_sel, ws, stream, nullptr));
}

}  // extern "C"
