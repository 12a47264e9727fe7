// The Dispatcher with on-demand bubble queues (Section 4.3; the appendix's
// Algorithm 2) on the GPU: one workgroup per call, everything in LDS.
//
//   1. The table's queue set goes to LDS and every request is placed against
//      it.  A length inside a queue, below the first or above the last keeps
//      that queue whatever bubbles appear later (bubbles only fill gaps).  A
//      length in a gap is listed with its arrival-order key, and counted when
//      it is a true gap (outside both tolerances).
//   2. No true gap (or no room for another queue): no bubble can appear, since
//      a request the set covers stays covered as bubbles are added, so every
//      listed request takes its neighbour by the tolerance rule (or the
//      nearer neighbour when the set is full).
//   3. Otherwise the listed requests are sorted by arrival (equal arrivals by
//      id, NaN last) and wave 0 runs the algorithm one request at a time: a
//      ballot over the (at most 256) queue starts finds the request's place
//      in the current set, and a bubble is inserted by shifting the queues
//      above it one place up.
//   4. Queues are renumbered in length order, the table is rewritten in its
//      gapped reading and the routing lut rebuilt.
#include <hip/hip_runtime.h>

#include "ewsjf_device.h"
#include "ewsjf_launch.h"
#include "ewsjf_lut.h"

namespace ewsjf {

namespace {

constexpr int kQ = EWSJF_MAX_QUEUES;
constexpr int kRoundsPerSet = kQ / kWave;  // ballot rounds over the queue starts

struct DispatchShared {
  int32_t lo[kQ], hi[kQ];  // the current set in length order
  int64_t n[kQ], S[kQ];
  double mean[kQ];
  int32_t ident[kQ];  // identity of the queue at each place (base queues 0..k0-1, then bubbles)
  int32_t place[kQ];  // final place of each identity
  uint64_t key[EWSJF_MAX_DISPATCH];  // listed requests: ~(arrival key << 32 | id)
  int32_t len[EWSJF_MAX_DISPATCH];
  int32_t who[EWSJF_MAX_DISPATCH];  // identity of each request's queue, -1 for an empty slot
  int nlist, ntrue, kcur;
};

// Places [from, k) of the set move one place up (k < kQ).  Every lane reads
// its entries before any lane writes, in one wave.
__device__ void shift_up(DispatchShared& sm, int from, int k, int lane) {
  int32_t lo[kRoundsPerSet], hi[kRoundsPerSet], id[kRoundsPerSet];
  int64_t n[kRoundsPerSet], S[kRoundsPerSet];
  double m[kRoundsPerSet];
#pragma unroll
  for (int r = 0; r < kRoundsPerSet; ++r) {
    const int p = lane + r * kWave;
    if (p >= from && p < k) {
      lo[r] = sm.lo[p];
      hi[r] = sm.hi[p];
      id[r] = sm.ident[p];
      n[r] = sm.n[p];
      S[r] = sm.S[p];
      m[r] = sm.mean[p];
    }
  }
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
#pragma unroll
  for (int r = 0; r < kRoundsPerSet; ++r) {
    const int p = lane + r * kWave;
    if (p >= from && p < k) {
      sm.lo[p + 1] = lo[r];
      sm.hi[p + 1] = hi[r];
      sm.ident[p + 1] = id[r];
      sm.n[p + 1] = n[r];
      sm.S[p + 1] = S[r];
      sm.mean[p + 1] = m[r];
    }
  }
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
}

// Algorithm 2 over the sorted list, one request at a time (wave 0).
__device__ void dispatch_in_order(DispatchShared& sm, int nlist, int k0, int width, int max_queues) {
  const int lane = threadIdx.x;
  int k = k0;
  int next_ident = k0;
  for (int j = 0; j < nlist; ++j) {
    const uint32_t id = (uint32_t)~sm.key[j];
    const int b = sm.len[id];
    int c = 0;  // queue starts <= b
#pragma unroll
    for (int r = 0; r < kRoundsPerSet; ++r) {
      const int p = lane + r * kWave;
      c += __popcll(__ballot(p < k && sm.lo[p] <= b));
    }
    const int i = c - 1;
    int w;
    if (i < 0) {
      w = sm.ident[0];
    } else if (b <= sm.hi[i] || i == k - 1) {
      w = sm.ident[i];
    } else {
      const int hi_i = sm.hi[i], lo_next = sm.lo[i + 1];
      int t = gap_tolerance(b, hi_i, lo_next, i);
      if (t < 0 && k < max_queues) {  // a true gap: a bubble queue centred on b, clipped to the gap
        const int64_t max_len = (int64_t)hi_i + 1, min_len = lo_next;
        const int64_t range = min((int64_t)width, min_len - max_len);
        const int64_t new_min = max((int64_t)b - range / 2, max_len);
        const int64_t new_max = min((int64_t)b - range / 2 + range, min_len);
        shift_up(sm, i + 1, k, lane);
        if (lane == 0) {
          sm.lo[i + 1] = (int32_t)new_min;
          sm.hi[i + 1] = (int32_t)(new_max - 1);
          sm.n[i + 1] = 1;
          sm.S[i + 1] = b;
          sm.mean[i + 1] = (double)b;
          sm.ident[i + 1] = next_ident;
        }
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
        w = next_ident++;
        ++k;
      } else {
        if (t < 0) t = gap_nearer(b, hi_i, lo_next, i);
        w = sm.ident[t];
      }
    }
    if (lane == 0) sm.who[id] = w;
  }
  if (lane == 0) sm.kcur = k;
}

__global__ __launch_bounds__(kBlock) void dispatch_kernel(const int32_t* __restrict__ len,
                                                          const float* __restrict__ arrival, int n,
                                                          ewsjf_queue_table* tab, int width, int max_queues,
                                                          int32_t* __restrict__ qid) {
  __shared__ DispatchShared sm;
  const int tid = threadIdx.x;
  const int k0 = tab->k;
  const bool was_gapped = tab->gapped != 0;
  const int L = tab->max_len;
  if (tid < k0) {
    sm.lo[tid] = tab->lo[tid];
    sm.hi[tid] = tab->hi[tid];
    sm.n[tid] = tab->count[tid];
    sm.S[tid] = tab->sum[tid];
    sm.mean[tid] = tab->mean[tid];
    sm.ident[tid] = tid;
  }
  if (tid == 0) {
    sm.nlist = 0;
    sm.ntrue = 0;
    sm.kcur = k0;
  }
  __syncthreads();
  for (int i = tid; i < n; i += kBlock) {
    const int b = len[i];
    sm.len[i] = b;
    int w = -1;
    if (b > 0) {
      const int q = count_le(sm.lo, k0, b) - 1;
      if (q < 0) {
        w = 0;
      } else if (b <= sm.hi[q] || q == k0 - 1) {
        w = q;
      } else {
        const int t = gap_tolerance(b, sm.hi[q], sm.lo[q + 1], q);
        w = t >= 0 ? t : gap_nearer(b, sm.hi[q], sm.lo[q + 1], q);  // final unless a bubble appears
        const int slot = atomicAdd(&sm.nlist, 1);
        sm.key[slot] = ~(((uint64_t)arrival_key(arrival[i]) << 32) | (uint32_t)i);
        if (t < 0) atomicAdd(&sm.ntrue, 1);
      }
    }
    sm.who[i] = w;
  }
  __syncthreads();
  const int nlist = sm.nlist;
  if (sm.ntrue > 0 && k0 < max_queues) {
    int P = 1;
    while (P < nlist) P <<= 1;
    for (int i = nlist + tid; i < P; i += kBlock) sm.key[i] = 0ull;
    __syncthreads();
    block_sort_desc(sm.key, P);  // descending complemented keys: oldest first
    if (tid < kWave) dispatch_in_order(sm, nlist, k0, width, max_queues);
    __syncthreads();
  }
  const int k1 = sm.kcur;
  if (tid < k1) sm.place[sm.ident[tid]] = tid;
  __syncthreads();
  for (int i = tid; i < n; i += kBlock) {
    const int w = sm.who[i];
    qid[i] = w < 0 ? -1 : sm.place[w];
  }
  if (k1 == k0 && was_gapped) return;  // the set and its lut are unchanged
  if (tid < k1) {
    tab->lo[tid] = sm.lo[tid];
    tab->hi[tid] = sm.hi[tid];
    tab->count[tid] = sm.n[tid];
    tab->sum[tid] = sm.S[tid];
    tab->mean[tid] = sm.mean[tid];
    if (tid > 0) tab->bounds[tid - 1] = sm.lo[tid];
  }
  if (tid == 0) {
    tab->k = k1;
    tab->gapped = 1;
  }
  lut_fill(tab->lut, tid, kBlock, L, true, sm.lo, sm.lo, sm.hi, k1);
  route_fill(tab->route, tid, kBlock, L, true, sm.lo, sm.lo, sm.hi, k1);
}

}  // namespace

hipError_t launch_dispatch(const int32_t* len, const float* arrival, int n, ewsjf_queue_table* table,
                           int32_t bubble_width, int32_t max_queues, int32_t* qid, hipStream_t stream) {
  hipLaunchKernelGGL(dispatch_kernel, dim3(1), dim3(kBlock), 0, stream, len, arrival, n, table, bubble_width,
                     max_queues, qid);
  return hipGetLastError();
}

}  // namespace ewsjf
