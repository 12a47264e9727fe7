// Host-side launch entry points of the kernel translation units, called by
// the C ABI layer after it has validated every argument.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "ewsjf.h"

namespace ewsjf {

// Launch geometry and workspace layout of the two-kernel top-B selection.
struct SelectPlan {
  int G = 1;        // streaming workgroups
  int lg = 2;       // log2 of the lane groups per wave that set the candidate bar
  int M = 16;       // list entries kept per workgroup
  int n_theta = 1;
  size_t lists_bytes = 0, counts_bytes = 0, bounds_bytes = 0;
  size_t over_bytes = 0, over_cnt_bytes = 0, bounds2_bytes = 0;
  size_t ws_bytes = 0;
};

// Per-workgroup candidate buffers in the step/select workspace, indexed by
// slot = theta * G + workgroup.
struct CandBufs {
  uint64_t* lists;     // [slot][M]: the M largest composites (0 = empty)
  uint32_t* counts;    // [slot]
  uint64_t* bounds;    // [slot]: every composite >= bound of the share is in its M slots
  uint64_t* over;      // [slot][kOverCap]: the next entries below the M slots
  uint32_t* over_cnt;  // [slot]
  uint64_t* bounds2;   // [slot]: every composite >= bound2 is in the slots or the overflow
};

// packed: each workgroup takes a full pass of chunks (the many-vector step).
// max_grid > 0 caps the streaming workgroups per row (default: one per CU).
// spread: the source's highest keys are not expected to cluster in one
// share (the pool and ring steps), so the candidate bars are set from the
// expected spread of the B; otherwise for the worst case (all of a
// workgroup's share of the B in one wave).  Sizes do not depend on it.
SelectPlan plan_select(int64_t n, int32_t n_theta, int32_t B, bool packed = false, int max_grid = 0,
                       bool spread = false);
// The plan ewsjf_step uses: packed for several vectors over a pool that fits
// one pass per workgroup.
SelectPlan plan_step(int64_t n, int32_t n_theta, int32_t B);

// Tactical step (Algorithm 1): the batch plan computed on the device after
// the head-of-line pass.  Row 0 of the queue-order selection drains q_sel[0]
// (the ArgMax queue); rows 1 and 2 the backfill neighbours in order.
constexpr int kTacticalRows = 3;
struct TacticalPlan {
  int32_t q_sel[kTacticalRows];  // queue of each row, -1 if none
  int32_t take[kTacticalRows];   // requests the batch takes from each row
  int32_t q_prim;                // -1 when every queue is empty
  int32_t k;                     // queues at the start of the step
  int32_t n_removed;             // queues past the empty threshold
  int32_t pad;
};

hipError_t launch_fifo_select(const int32_t* len, const float* arrival, int64_t n, const ewsjf_queue_table* table,
                              const TacticalPlan* plan, int32_t B, int32_t* ids, float* top, int32_t* n_sel, void* ws,
                              hipStream_t stream);

// ring insert + one-vector step in the same two kernels (ewsjf_ring_step)
hipError_t launch_ring_step(int32_t* ring_len, float* ring_arrival, int64_t capacity, int64_t pos, int32_t* window,
                            int64_t window_cap, int64_t wpos, const int32_t* new_len, const float* new_arrival,
                            int64_t n_new, float now, const ewsjf_queue_table* table, const ewsjf_theta* theta,
                            const ewsjf_cost& cost, int32_t B, int32_t* tomb_len, int32_t* ids, float* top,
                            int32_t* n_sel, void* ws, hipStream_t stream);

SelectPlan plan_trial(int64_t capacity, int32_t n_pools, int32_t B);
// Trials: the step's two kernels over n_pools pools of `capacity` slots
// (pool t = proposal t, slots [t * capacity, (t + 1) * capacity)), each taking
// the same arrivals at ring position pos; no tombstones (the statistics
// kernel reads the admitted requests first).  Workspace plan_trial(capacity,
// n_pools, B).
hipError_t launch_trial_select(int32_t* len, float* arrival, int64_t capacity, int32_t n_pools, int64_t pos,
                               const int32_t* new_len, const float* new_arrival, int64_t n_new, float now,
                               const ewsjf_queue_table* table, const ewsjf_theta* theta, const ewsjf_cost& cost,
                               int32_t B, int32_t* ids, float* top, int32_t* n_sel, void* ws, hipStream_t stream);
// Trial statistics of the admitted requests (then tombstoned), and the
// trial's end: pending statistics and the reward.
hipError_t launch_trial_stats(int32_t* len, const float* arrival, int64_t capacity, int32_t n_pools, float now,
                              const ewsjf_queue_table* table, int32_t B, const int32_t* ids, const int32_t* n_sel,
                              double* stats, int64_t* queue_admits, hipStream_t stream);
hipError_t launch_trial_finish(const int32_t* len, const float* arrival, int64_t capacity, int32_t n_pools,
                               float now, const ewsjf_queue_table* table, const int64_t* queue_admits,
                               const double* lambda, double* stats, double* reward, hipStream_t stream);

size_t tactical_ws_bytes(int64_t n, int32_t B);
hipError_t launch_tactical_step(int32_t* len, const float* arrival, int64_t n, float now, ewsjf_queue_table* table,
                                const ewsjf_theta* theta, const ewsjf_cost& cost, int32_t B, int32_t empty_threshold,
                                int32_t* empty_cnt, double eps, int32_t* tomb_len, int32_t* ids, int32_t* n_sel,
                                int32_t* q_prim, float* head_score, int32_t* removed, void* ws, hipStream_t stream);

// marks (optional, may be NULL): four events taking the start and end
// timestamps of the streaming kernel and of the merge kernel.
hipError_t launch_step(const int32_t* len, const float* arrival, int64_t n, float now,
                       const ewsjf_queue_table* table, const ewsjf_theta* theta, int32_t n_theta,
                       const ewsjf_cost& cost, int32_t B, int32_t* tomb_len, int32_t* ids, float* top,
                       int32_t* n_sel, void* ws, hipStream_t stream, hipEvent_t* marks = nullptr);

hipError_t launch_select(const float* score, int64_t n, int32_t n_theta, int32_t B, int32_t* ids, float* top,
                         int32_t* n_sel, void* ws, hipStream_t stream);

hipError_t launch_route(const int32_t* len, int64_t n, const ewsjf_queue_table* table, int32_t* qid,
                        hipStream_t stream);

hipError_t launch_score(const int32_t* len, const float* arrival, int64_t n, float now,
                        const ewsjf_queue_table* table, const ewsjf_theta* theta, int32_t n_theta,
                        const ewsjf_cost& cost, float* score, hipStream_t stream);

// Builds the routing lut of a device table whose header and bounds are set.
hipError_t launch_build_lut(ewsjf_queue_table* table, hipStream_t stream);
hipError_t launch_ring_insert(int32_t* ring_len, float* ring_arrival, int64_t capacity, int64_t pos, int32_t* window,
                              int64_t window_cap, int64_t wpos, const int32_t* new_len, const float* new_arrival,
                              int64_t n, hipStream_t stream);

// Dispatcher with on-demand bubble queues (n <= EWSJF_MAX_DISPATCH).
hipError_t launch_dispatch(const int32_t* len, const float* arrival, int n, ewsjf_queue_table* table,
                           int32_t bubble_width, int32_t max_queues, int32_t* qid, hipStream_t stream);

// Refine-and-Prune.
size_t partition_ws_bytes(int64_t n_window, const ewsjf_partition_params& p);
hipError_t launch_partition(const int32_t* window, int64_t n_window, const ewsjf_partition_params& p,
                            ewsjf_queue_table* table, void* ws, hipStream_t stream);
// from a histogram of clamped lengths (hist[0..p.max_len]); workspace
// partition_ws_bytes(0, p)
hipError_t launch_partition_hist(const uint32_t* hist, const ewsjf_partition_params& p, ewsjf_queue_table* table,
                                 void* ws, hipStream_t stream);
// hist[0..L] := histogram of ring[(begin + i) mod cap], i < n, clamped to [1, L]
// (n <= cap, begin < cap)
hipError_t launch_window_histogram(const int32_t* ring, int64_t cap, int64_t begin, int64_t n, int L, uint32_t* hist,
                                   hipStream_t stream);
// hist += counts of ring[(add + i) mod cap], hist -= counts of ring[(sub + i) mod cap],
// i < n (add, sub < cap; n <= cap)
hipError_t launch_window_advance(const int32_t* ring, int64_t cap, int64_t add, int64_t sub, int64_t n, int L,
                                 uint32_t* hist, hipStream_t stream);

}  // namespace ewsjf
