// Routing lut construction, Dynamic Queue Routing and Density-Weighted
// Scoring kernels.
#include <hip/hip_runtime.h>

#include "ewsjf_device.h"
#include "ewsjf_launch.h"
#include "ewsjf_lut.h"

namespace ewsjf {

// lut[b] = the queue holding length b under the table's reading: the number
// of bounds <= b (contiguous cover; Section 3.2 Dispatcher), or the gapped
// rule of lo/hi (Section 4.3).
__global__ __launch_bounds__(256) void build_lut_kernel(ewsjf_queue_table* tab) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  lut_fill(tab->lut, t, gridDim.x * blockDim.x, tab->max_len, tab->gapped != 0, tab->bounds, tab->lo, tab->hi,
           tab->k);
  route_fill(tab->route, t, gridDim.x * blockDim.x, tab->max_len, tab->gapped != 0, tab->bounds, tab->lo, tab->hi,
             tab->k);
}

hipError_t launch_build_lut(ewsjf_queue_table* table, hipStream_t stream) {
  hipLaunchKernelGGL(build_lut_kernel, dim3(8), dim3(256), 0, stream, table);  // 4 words per thread
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Routing: qid[i] = queue of len[i] (-1 for an empty slot).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kBlock) void route_kernel(const int32_t* __restrict__ len, int64_t n,
                                                       const ewsjf_queue_table* __restrict__ tab,
                                                       int32_t* __restrict__ qid) {
  __shared__ uint8_t lut[kLutBytes];
  __shared__ QParams qp_unused[1];
  stage_policy(tab, nullptr, lut, qp_unused);
  const int L = tab->max_len;
  __syncthreads();
  const int64_t nvec = n / 4;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t v = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; v < nvec; v += stride) {
    const i32x4 b = load_i32x4(len + 4 * v);
    i32x4 q;
    q.x = route_lut(b.x, L, lut);
    q.y = route_lut(b.y, L, lut);
    q.z = route_lut(b.z, L, lut);
    q.w = route_lut(b.w, L, lut);
    *reinterpret_cast<i32x4*>(qid + 4 * v) = q;
  }
  for (int64_t i = nvec * 4 + blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += stride)
    qid[i] = route_lut(len[i], L, lut);
}

// ---------------------------------------------------------------------------
// Streaming pool update: new requests into consecutive ring slots and their
// lengths into the window ring.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void ring_insert_kernel(int32_t* __restrict__ ring_len,
                                                          float* __restrict__ ring_arrival, int64_t capacity,
                                                          int64_t pos, int32_t* __restrict__ window,
                                                          int64_t window_cap, int64_t wpos,
                                                          const int32_t* __restrict__ new_len,
                                                          const float* __restrict__ new_arrival, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int32_t b = new_len[i];
  int64_t slot = pos + i;
  if (slot >= capacity) slot -= capacity;  // n <= capacity and pos < capacity
  ring_len[slot] = b;
  ring_arrival[slot] = new_arrival[i];
  if (window_cap > 0) {
    int64_t w = wpos + i;
    if (w >= window_cap) w -= window_cap;  // n <= window_cap and wpos < window_cap
    window[w] = b;
  }
}

hipError_t launch_ring_insert(int32_t* ring_len, float* ring_arrival, int64_t capacity, int64_t pos, int32_t* window,
                              int64_t window_cap, int64_t wpos, const int32_t* new_len, const float* new_arrival,
                              int64_t n, hipStream_t stream) {
  const int64_t blocks = (n + 255) / 256;
  hipLaunchKernelGGL(ring_insert_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, ring_len, ring_arrival,
                     capacity, pos, window, window_cap, wpos, new_len, new_arrival, n);
  return hipGetLastError();
}

hipError_t launch_route(const int32_t* len, int64_t n, const ewsjf_queue_table* table, int32_t* qid,
                        hipStream_t stream) {
  int64_t blocks = (n / 4 + kBlock - 1) / kBlock;
  if (blocks < 1) blocks = 1;
  if (blocks > 2 * kMaxGrid) blocks = 2 * kMaxGrid;
  hipLaunchKernelGGL(route_kernel, dim3((unsigned)blocks), dim3(kBlock), 0, stream, len, n, table, qid);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Scoring: score[t][i] = Phi of request i under parameter vector t.
// ---------------------------------------------------------------------------
__device__ __forceinline__ float score1(int b, float a, float now, int L, const uint8_t* lut, const QParams* qp,
                                        const CostF& c) {
  if (b <= 0) return __builtin_nanf("");
  const float phi = phi_f32(b, a, now, qp[lut[b < L ? b : L]], c);
  return (phi != phi) ? -__builtin_inff() : phi;
}

__global__ __launch_bounds__(kBlock) void score_kernel(const int32_t* __restrict__ len,
                                                       const float* __restrict__ arrival, int64_t n, float now,
                                                       const ewsjf_queue_table* __restrict__ tab,
                                                       const ewsjf_theta* __restrict__ theta, CostF cost,
                                                       float* __restrict__ score) {
  __shared__ uint8_t lut[kLutBytes];
  __shared__ QParams qp[EWSJF_MAX_QUEUES];
  const int t = blockIdx.y;
  stage_policy(tab, theta + t, lut, qp);
  const int L = tab->max_len;
  __syncthreads();
  float* out = score + (int64_t)t * n;
  const bool vec_out = (reinterpret_cast<uintptr_t>(out) & 15) == 0;
  const int64_t nvec = n / 4;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t v = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; v < nvec; v += stride) {
    const i32x4 b = load_i32x4(len + 4 * v);
    const f32x4 a = load_f32x4(arrival + 4 * v);
    f32x4 s;
    s.x = score1(b.x, a.x, now, L, lut, qp, cost);
    s.y = score1(b.y, a.y, now, L, lut, qp, cost);
    s.z = score1(b.z, a.z, now, L, lut, qp, cost);
    s.w = score1(b.w, a.w, now, L, lut, qp, cost);
    if (vec_out) {
      *reinterpret_cast<f32x4*>(out + 4 * v) = s;
    } else {
      out[4 * v + 0] = s.x;
      out[4 * v + 1] = s.y;
      out[4 * v + 2] = s.z;
      out[4 * v + 3] = s.w;
    }
  }
  for (int64_t i = nvec * 4 + blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += stride)
    out[i] = score1(len[i], arrival[i], now, L, lut, qp, cost);
}

hipError_t launch_score(const int32_t* len, const float* arrival, int64_t n, float now,
                        const ewsjf_queue_table* table, const ewsjf_theta* theta, int32_t n_theta,
                        const ewsjf_cost& cost, float* score, hipStream_t stream) {
  int64_t blocks = (n / 4 + kBlock - 1) / kBlock;
  if (blocks < 1) blocks = 1;
  if (blocks > 2 * kMaxGrid) blocks = 2 * kMaxGrid;
  const CostF c{(float)cost.c0, (float)cost.c1, (float)cost.c2};
  hipLaunchKernelGGL(score_kernel, dim3((unsigned)blocks, n_theta), dim3(kBlock), 0, stream, len, arrival, n, now,
                     table, theta, c, score);
  return hipGetLastError();
}

}  // namespace ewsjf
