// Trials of scoring-parameter proposals: the simulator side of the
// meta-optimizer (Section 4.4.2).  Each proposal runs the per-request step on
// its own pool for a trial of several steps; these kernels keep the trial's
// statistics (Eq. 5's reward is built from them at the end).
//
//   trial_stats_kernel    one workgroup per pool: wait, tokens and queue of
//                         every admitted request, reduced in a fixed order
//                         (the sums are deterministic), added to the pool's
//                         statistics; then the admitted slots are emptied.
//   trial_pending_kernel  the pending requests at the trial's end: count and
//                         largest wait (integer-valued adds and a maximum, so
//                         the order of the atomics does not matter).
//   trial_reward_kernel   Eq. 5 per pool: C from the queue intervals, L from
//                         the admissions per queue, S from the queue count, U
//                         the mean wait of the admitted requests.
#include <hip/hip_runtime.h>

#include "ewsjf_device.h"
#include "ewsjf_launch.h"

namespace ewsjf {

namespace {

constexpr int kStatThreads = 256;
enum {
  kAdmitted = 0,
  kTokens,
  kWaitSum,
  kWaitSqSum,
  kWaitMax,
  kPending,
  kPendingWaitMax,
  kSteps,
};
static_assert(kSteps + 1 == EWSJF_TRIAL_STATS, "statistics layout");

// Wait W = max(0, now - arrival) in binary64; a NaN arrival waits 0.
__device__ __forceinline__ double wait_of(float now, float a) {
  const double w = (double)now - (double)a;
  return w > 0.0 ? w : 0.0;
}

__global__ __launch_bounds__(kStatThreads) void trial_stats_kernel(int32_t* __restrict__ len,
                                                                   const float* __restrict__ arrival, int64_t cap,
                                                                   float now, const ewsjf_queue_table* tab, int B,
                                                                   const int32_t* __restrict__ ids,
                                                                   const int32_t* __restrict__ n_sel,
                                                                   double* __restrict__ stats,
                                                                   int64_t* __restrict__ queue_admits) {
  __shared__ uint32_t qc[EWSJF_MAX_QUEUES];
  __shared__ double rw[kStatThreads], rw2[kStatThreads], rmax[kStatThreads];
  __shared__ int64_t rtok[kStatThreads];
  const int p = blockIdx.x, tid = threadIdx.x;
  int32_t* L = len + (int64_t)p * cap;
  const float* A = arrival + (int64_t)p * cap;
  const int32_t* id = ids + (int64_t)p * B;
  const int sel = n_sel[p];
  const int k = tab->k, Lmax = tab->max_len;
  for (int q = tid; q < EWSJF_MAX_QUEUES; q += kStatThreads) qc[q] = 0u;
  __syncthreads();
  double w1 = 0.0, w2 = 0.0, wm = 0.0;
  int64_t tok = 0;
  for (int r = tid; r < sel; r += kStatThreads) {
    const int i = id[r];
    const int b = L[i];  // admitted, so b >= 1
    const double w = wait_of(now, A[i]);
    w1 += w;
    w2 += w * w;
    wm = w > wm ? w : wm;
    tok += b;
    atomicAdd(&qc[tab->lut[b < Lmax ? b : Lmax]], 1u);
  }
  rw[tid] = w1;
  rw2[tid] = w2;
  rmax[tid] = wm;
  rtok[tid] = tok;
  __syncthreads();
  for (int s = kStatThreads / 2; s > 0; s >>= 1) {
    if (tid < s) {
      rw[tid] += rw[tid + s];
      rw2[tid] += rw2[tid + s];
      rmax[tid] = rmax[tid + s] > rmax[tid] ? rmax[tid + s] : rmax[tid];
      rtok[tid] += rtok[tid + s];
    }
    __syncthreads();
  }
  // every read of the admitted slots is done (barrier above): empty them
  for (int r = tid; r < sel; r += kStatThreads) L[id[r]] = 0;
  if (tid == 0) {
    double* st = stats + (int64_t)p * EWSJF_TRIAL_STATS;
    st[kAdmitted] += (double)sel;
    st[kTokens] += (double)rtok[0];
    st[kWaitSum] += rw[0];
    st[kWaitSqSum] += rw2[0];
    st[kWaitMax] = rmax[0] > st[kWaitMax] ? rmax[0] : st[kWaitMax];
    st[kSteps] += 1.0;
  }
  int64_t* qa = queue_admits + (int64_t)p * EWSJF_MAX_QUEUES;
  for (int q = tid; q < k; q += kStatThreads)
    if (qc[q]) qa[q] += (int64_t)qc[q];
}

__global__ void trial_pending_reset(double* stats, int n_pools) {
  const int p = blockIdx.x * blockDim.x + threadIdx.x;
  if (p < n_pools) {
    stats[(int64_t)p * EWSJF_TRIAL_STATS + kPending] = 0.0;
    stats[(int64_t)p * EWSJF_TRIAL_STATS + kPendingWaitMax] = 0.0;
  }
}

__global__ __launch_bounds__(kStatThreads) void trial_pending_kernel(const int32_t* __restrict__ len,
                                                                     const float* __restrict__ arrival, int64_t cap,
                                                                     float now, double* __restrict__ stats) {
  __shared__ uint32_t rc[kStatThreads];
  __shared__ double rmax[kStatThreads];
  const int p = blockIdx.y, tid = threadIdx.x;
  const int32_t* L = len + (int64_t)p * cap;
  const float* A = arrival + (int64_t)p * cap;
  uint32_t c = 0;
  double wm = 0.0;
  for (int64_t i = (int64_t)blockIdx.x * kStatThreads + tid; i < cap; i += (int64_t)gridDim.x * kStatThreads) {
    if (L[i] > 0) {
      ++c;
      const double w = wait_of(now, A[i]);
      wm = w > wm ? w : wm;
    }
  }
  rc[tid] = c;
  rmax[tid] = wm;
  __syncthreads();
  for (int s = kStatThreads / 2; s > 0; s >>= 1) {
    if (tid < s) {
      rc[tid] += rc[tid + s];
      rmax[tid] = rmax[tid + s] > rmax[tid] ? rmax[tid + s] : rmax[tid];
    }
    __syncthreads();
  }
  if (tid == 0) {
    double* st = stats + (int64_t)p * EWSJF_TRIAL_STATS;
    if (rc[0]) atomicAdd(&st[kPending], (double)rc[0]);  // integer values: exact in any order
    // non-negative binary64 values order like their bit patterns
    atomicMax(reinterpret_cast<unsigned long long*>(&st[kPendingWaitMax]),
              (unsigned long long)__double_as_longlong(rmax[0]));
  }
}

struct Lambda {
  double c, l, s, u;
};

__global__ __launch_bounds__(kStatThreads) void trial_reward_kernel(const ewsjf_queue_table* tab, int n_pools,
                                                                    const int64_t* __restrict__ queue_admits,
                                                                    const double* __restrict__ stats, Lambda lam,
                                                                    double* __restrict__ reward) {
  const int k = tab->k;
  double csum = 0.0;
  for (int q = 0; q < k; ++q) csum += (double)(tab->hi[q] - tab->lo[q]) / (double)(tab->hi[q] + tab->lo[q]);
  const double C = -(csum / (double)k);
  const double S = (double)k / (double)EWSJF_MAX_QUEUES;
  for (int p = threadIdx.x; p < n_pools; p += kStatThreads) {
    const int64_t* qa = queue_admits + (int64_t)p * EWSJF_MAX_QUEUES;
    double sum = 0.0;
    for (int q = 0; q < k; ++q) sum += (double)qa[q];
    const double m = sum / (double)k;
    double var = 0.0;
    for (int q = 0; q < k; ++q) {
      const double d = (double)qa[q] - m;
      var += d * d;
    }
    const double Lb = m > 0.0 ? -(sqrt(var / (double)k) / m) : 0.0;
    const double* st = stats + (int64_t)p * EWSJF_TRIAL_STATS;
    const double U = st[kAdmitted] > 0.0 ? st[kWaitSum] / st[kAdmitted] : 0.0;
    reward[p] = lam.c * C + lam.l * Lb - lam.s * S - lam.u * U;
  }
}

}  // namespace

hipError_t launch_trial_stats(int32_t* len, const float* arrival, int64_t capacity, int32_t n_pools, float now,
                              const ewsjf_queue_table* table, int32_t B, const int32_t* ids, const int32_t* n_sel,
                              double* stats, int64_t* queue_admits, hipStream_t stream) {
  hipLaunchKernelGGL(trial_stats_kernel, dim3(n_pools), dim3(kStatThreads), 0, stream, len, arrival, capacity, now,
                     table, B, ids, n_sel, stats, queue_admits);
  return hipGetLastError();
}

hipError_t launch_trial_finish(const int32_t* len, const float* arrival, int64_t capacity, int32_t n_pools,
                               float now, const ewsjf_queue_table* table, const int64_t* queue_admits,
                               const double* lambda, double* stats, double* reward, hipStream_t stream) {
  hipLaunchKernelGGL(trial_pending_reset, dim3((n_pools + 255) / 256), dim3(256), 0, stream, stats, n_pools);
  int64_t gx = (capacity + 16383) / 16384;  // 16,384 slots (64 per thread) per workgroup
  if (gx < 1) gx = 1;
  if (gx > 256) gx = 256;
  hipLaunchKernelGGL(trial_pending_kernel, dim3((unsigned)gx, n_pools), dim3(kStatThreads), 0, stream, len, arrival,
                     capacity, now, stats);
  const Lambda lam{lambda[0], lambda[1], lambda[2], lambda[3]};
  hipLaunchKernelGGL(trial_reward_kernel, dim3(1), dim3(kStatThreads), 0, stream, table, n_pools, queue_admits, stats,
                     lam, reward);
  return hipGetLastError();
}

}  // namespace ewsjf
