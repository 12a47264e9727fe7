// Tactical step (Algorithm 1, Section 3.2): the paper's own batch rule.
//
//   tac_scan    (G workgroups)  one pass over the pool: per queue, the number
//                               of pending requests and the oldest one (its
//                               head), per workgroup.
//   tac_reduce  (k workgroups)  per queue: the totals, and Phi of the head
//                               (Eq. 1 / Eq. 4) in binary64.
//   tac_plan    (1 workgroup)   empty counters, ArgMax queue, how many
//                               requests GreedyFill and Backfill take from the
//                               queue and its two neighbours.
//   queue-order selection       local_candidates / merge_candidates with
//                               FifoSource: the oldest requests of each of
//                               the (up to) three queues.
//   tac_finish  (1 workgroup)   the batch in order, tombstones, and the
//                               removal of queues empty past the threshold
//                               (re-absorbed by the neighbour of lower Eq. 3
//                               utility), with the routing lut rebuilt.
//
// Readings the paper leaves open (the oracle takes the same ones): a queue
// is a FIFO in arrival order (equal arrivals by id, NaN arrival last);
// ArgMax ties go to the lower queue; the two neighbours backfill in order of
// their head scores (ties: the lower queue first); empty counters count
// consecutive empty steps; removals apply after the batch is built, lowest
// index first, and the last queue is never removed.
#include <hip/hip_runtime.h>

#include "ewsjf_device.h"
#include "ewsjf_launch.h"
#include "ewsjf_lut.h"

namespace ewsjf {
namespace {

constexpr int kLutVecs = kLutBytes / 16;
constexpr int kReduceThreads = 256;

struct TacWs {
  uint32_t* part_cnt;   // [EWSJF_MAX_QUEUES][G]
  uint64_t* part_head;  // [EWSJF_MAX_QUEUES][G]: (arrival_key << 32) | id, ~0 = none
  uint32_t* cnt;        // [EWSJF_MAX_QUEUES]
  uint64_t* head;       // [EWSJF_MAX_QUEUES]
  float* score;         // [EWSJF_MAX_QUEUES]: Phi of the head, NaN if empty
  TacticalPlan* plan;
  int32_t* row_ids;     // [kTacticalRows][B]
  float* row_top;       // [kTacticalRows][B]
  int32_t* row_n;       // [kTacticalRows]
  void* select_ws;
};

int scan_grid(int64_t n) {
  const int64_t nchunks = (n + kChunk - 1) / kChunk;
  int64_t G = (nchunks + 4 * kWavesPerBlock - 1) / (4 * kWavesPerBlock);
  if (G < 1) G = 1;
  if (G > kMaxGrid) G = kMaxGrid;
  return (int)G;
}

size_t up256(size_t x) { return (x + 255) & ~(size_t)255; }

size_t carve_tac(int64_t n, int32_t B, void* ws, TacWs* w) {
  const int G = scan_grid(n);
  char* b = static_cast<char*>(ws);
  size_t o = 0;
  auto take = [&](size_t bytes) {
    char* p = b ? b + o : nullptr;
    o += up256(bytes);
    return p;
  };
  TacWs t;
  t.part_cnt = reinterpret_cast<uint32_t*>(take((size_t)EWSJF_MAX_QUEUES * G * 4));
  t.part_head = reinterpret_cast<uint64_t*>(take((size_t)EWSJF_MAX_QUEUES * G * 8));
  t.cnt = reinterpret_cast<uint32_t*>(take(EWSJF_MAX_QUEUES * 4));
  t.head = reinterpret_cast<uint64_t*>(take(EWSJF_MAX_QUEUES * 8));
  t.score = reinterpret_cast<float*>(take(EWSJF_MAX_QUEUES * 4));
  t.plan = reinterpret_cast<TacticalPlan*>(take(sizeof(TacticalPlan)));
  t.row_ids = reinterpret_cast<int32_t*>(take((size_t)kTacticalRows * B * 4));
  t.row_top = reinterpret_cast<float*>(take((size_t)kTacticalRows * B * 4));
  t.row_n = reinterpret_cast<int32_t*>(take(kTacticalRows * 4));
  t.select_ws = take(plan_select(n, kTacticalRows, B).ws_bytes);
  if (w) *w = t;
  return o;
}

// ---------------------------------------------------------------------------
// Head-of-line pass.  Chunk c of workgroup w at local index lc is
// c = w + G * lc; each wave keeps four chunks in flight.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kBlock) void tac_scan(const int32_t* __restrict__ len, const float* __restrict__ arrival,
                                                   int64_t n, const ewsjf_queue_table* __restrict__ tab, int G,
                                                   uint32_t* __restrict__ part_cnt, uint64_t* __restrict__ part_head) {
  __shared__ uint8_t lut[kLutBytes];
  __shared__ uint32_t cnt[EWSJF_MAX_QUEUES];
  __shared__ uint64_t head[EWSJF_MAX_QUEUES];
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wv = tid / kWave;
  {
    const i32x4* src = reinterpret_cast<const i32x4*>(tab->lut);
    i32x4* dst = reinterpret_cast<i32x4*>(lut);
    for (int i = tid; i < kLutVecs; i += kBlock) dst[i] = src[i];
  }
  if (tid < EWSJF_MAX_QUEUES) {
    cnt[tid] = 0u;
    head[tid] = ~0ull;
  }
  const int L = tab->max_len, k = tab->k;
  __syncthreads();
  const int64_t nchunks = (n + kChunk - 1) / kChunk;
  for (int64_t lc0 = wv;; lc0 += 4 * kWavesPerBlock) {
    const int64_t c0 = (int64_t)blockIdx.x + (int64_t)G * lc0;
    if (c0 >= nchunks) break;
    i32x4 l[4], a[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {  // chunks past the end read zeros
      const int64_t first = ((int64_t)blockIdx.x + (int64_t)G * (lc0 + (int64_t)j * kWavesPerBlock)) * kChunk;
      l[j] = chunk_load_i32x4(chunk_rsrc(len + first, n - first), lane);
      a[j] = chunk_load_i32x4(chunk_rsrc(arrival + first, n - first), lane);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t first = ((int64_t)blockIdx.x + (int64_t)G * (lc0 + (int64_t)j * kWavesPerBlock)) * kChunk;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int b = l[j][e];
        if (b > 0) {
          const int q = lut[min(b, L)];
          atomicAdd(&cnt[q], 1u);
          const uint64_t hk = ((uint64_t)arrival_key(__int_as_float(a[j][e])) << 32) |
                              (uint64_t)(first + 4 * lane + e);
          if (hk < head[q]) atomicMin(reinterpret_cast<unsigned long long*>(&head[q]), (unsigned long long)hk);
        }
      }
    }
  }
  __syncthreads();
  if (tid < k) {
    part_cnt[(size_t)tid * G + blockIdx.x] = cnt[tid];
    part_head[(size_t)tid * G + blockIdx.x] = head[tid];
  }
}

// ---------------------------------------------------------------------------
// Per queue: totals over the workgroups, and the head's score in binary64
// (Eq. 1 / Eq. 4, the oracle's expression order; no contraction).
// ---------------------------------------------------------------------------
__device__ float head_phi(int32_t len, float arrival, float now, int q, double mean, const ewsjf_theta& th,
                          const ewsjf_cost& c) {
#pragma clang fp contract(off)
  const double m = mean;
  const double w_base = (double)th.a_base * m + (double)th.b_base;
  const double w_urg = (double)th.a_urg * m + (double)th.b_urg;
  const double w_fair = (double)th.a_fair * m + (double)th.b_fair;
  double W = (double)now - (double)arrival;
  if (!(W > 0.0)) W = 0.0;
  const double b = (double)len;
  const double C = c.c0 + c.c1 * b + c.c2 * b * b;
  const double cs = W / C;
  const double qf = (double)(q + 1) / (b + 1.0);
  const double phi = qf * ((w_base + w_urg * cs) + w_fair * log(b + 1.0));
  const float key = (float)phi;
  return key != key ? -__builtin_huge_valf() : key;
}

__global__ __launch_bounds__(kReduceThreads) void tac_reduce(const uint32_t* __restrict__ part_cnt,
                                                             const uint64_t* __restrict__ part_head, int G,
                                                             const int32_t* __restrict__ len,
                                                             const float* __restrict__ arrival, float now,
                                                             const ewsjf_queue_table* __restrict__ tab,
                                                             const ewsjf_theta* __restrict__ theta, ewsjf_cost cost,
                                                             uint32_t* cnt, uint64_t* head, float* score) {
  __shared__ uint32_t sc[kReduceThreads / kWave];
  __shared__ uint64_t sh[kReduceThreads / kWave];
  const int q = blockIdx.x, tid = threadIdx.x, lane = tid & (kWave - 1), wv = tid / kWave;
  if (q >= tab->k) return;  // uniform over the workgroup
  uint32_t c = 0;
  uint64_t h = ~0ull;
  for (int w = tid; w < G; w += kReduceThreads) {
    c += part_cnt[(size_t)q * G + w];
    const uint64_t x = part_head[(size_t)q * G + w];
    h = x < h ? x : h;
  }
  c = __ockl_wfred_add_u32(c);
  h = wave_min_u64(h);
  if (lane == 0) {
    sc[wv] = c;
    sh[wv] = h;
  }
  __syncthreads();
  if (tid == 0) {
    for (int i = 1; i < kReduceThreads / kWave; ++i) {
      c += sc[i];
      h = sh[i] < h ? sh[i] : h;
    }
    cnt[q] = c;
    head[q] = h;
    float s = __builtin_nanf("");
    if (c > 0) {
      const uint32_t id = (uint32_t)h;
      s = head_phi(len[id], arrival[id], now, q, tab->mean[q], theta[0], cost);
    }
    score[q] = s;
  }
}

// ---------------------------------------------------------------------------
// The batch plan (one workgroup, one thread per queue).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(EWSJF_MAX_QUEUES) void tac_plan(const ewsjf_queue_table* __restrict__ tab,
                                                             const uint32_t* __restrict__ cnt,
                                                             const float* __restrict__ score, int32_t B,
                                                             int32_t empty_threshold, int32_t* empty_cnt,
                                                             TacticalPlan* plan, int32_t* q_prim, float* head_score) {
  __shared__ uint64_t wbest[EWSJF_MAX_QUEUES / kWave];
  __shared__ int nmark[EWSJF_MAX_QUEUES / kWave];
  const int q = threadIdx.x, lane = q & (kWave - 1), wv = q / kWave;
  const int k = tab->k;
  const bool live = q < k;
  const uint32_t c = live ? cnt[q] : 0u;
  const float s = live ? score[q] : __builtin_nanf("");
  bool mark = false;
  if (live) {
    const int ec = c > 0 ? 0 : empty_cnt[q] + 1;
    empty_cnt[q] = ec;
    mark = c == 0 && ec > empty_threshold;
    if (head_score) head_score[q] = s;
  }
  // ArgMax over the non-empty queues; equal scores go to the lower queue.
  const uint64_t key = c > 0 ? make_comp(ukey_of(s), (uint32_t)q) : 0ull;
  const uint64_t wm = wave_max_u64(key);
  const int nm = (int)__popcll(__ballot(mark));
  if (lane == 0) {
    wbest[wv] = wm;
    nmark[wv] = nm;
  }
  __syncthreads();
  if (q == 0) {
    uint64_t best = 0;
    int marks = 0;
    for (int i = 0; i < EWSJF_MAX_QUEUES / kWave; ++i) {
      best = wbest[i] > best ? wbest[i] : best;
      marks += nmark[i];
    }
    TacticalPlan p;
    p.k = k;
    p.n_removed = marks;
    p.pad = 0;
    for (int r = 0; r < kTacticalRows; ++r) {
      p.q_sel[r] = -1;
      p.take[r] = 0;
    }
    p.q_prim = best == 0 ? -1 : (int)comp_id(best);
    if (p.q_prim >= 0) {
      const int prim = p.q_prim;
      p.q_sel[0] = prim;
      int64_t left = B;
      const int64_t t0 = (int64_t)cnt[prim] < left ? (int64_t)cnt[prim] : left;
      p.take[0] = (int)t0;
      left -= t0;
      // Backfill: the non-empty neighbours, higher head score first.
      int nb[2], nn = 0;
      if (prim > 0 && cnt[prim - 1] > 0) nb[nn++] = prim - 1;
      if (prim + 1 < k && cnt[prim + 1] > 0) nb[nn++] = prim + 1;
      if (nn == 2 && score[nb[1]] > score[nb[0]]) {
        const int x = nb[0];
        nb[0] = nb[1];
        nb[1] = x;
      }
      for (int i = 0; i < nn; ++i) {
        const int64_t ti = (int64_t)cnt[nb[i]] < left ? (int64_t)cnt[nb[i]] : left;
        p.q_sel[1 + i] = nb[i];
        p.take[1 + i] = (int)ti;
        left -= ti;
      }
    }
    *plan = p;
    *q_prim = p.q_prim;
  }
}

// ---------------------------------------------------------------------------
// The batch, tombstones, and queue removal.
// ---------------------------------------------------------------------------
__device__ double eq3_utility(int64_t na, int64_t Sa, int32_t loa, int32_t hia, int64_t nb, int64_t Sb, int32_t lob,
                              int32_t hib, double eps) {
#pragma clang fp contract(off)
  const double rho_a = (double)na / (double)((int64_t)hia - (int64_t)loa + 1);
  const double rho_b = (double)nb / (double)((int64_t)hib - (int64_t)lob + 1);
  const double m_a = (double)Sa / (double)na;
  const double m_b = (double)Sb / (double)nb;
  return (rho_a + rho_b) / (fabs(m_b - m_a) + eps);
}

__global__ __launch_bounds__(kBlock) void tac_finish(const TacticalPlan* __restrict__ plan,
                                                     const int32_t* __restrict__ row_ids, int32_t B,
                                                     int32_t* tomb_len, int32_t* ids, int32_t* n_sel,
                                                     ewsjf_queue_table* tab, const uint32_t* __restrict__ cnt,
                                                     int32_t empty_threshold, int32_t* empty_cnt, double eps,
                                                     int32_t* removed) {
  __shared__ int64_t qn[EWSJF_MAX_QUEUES], qS[EWSJF_MAX_QUEUES];
  __shared__ int32_t qlo[EWSJF_MAX_QUEUES], qhi[EWSJF_MAX_QUEUES], qec[EWSJF_MAX_QUEUES], qorig[EWSJF_MAX_QUEUES];
  __shared__ int32_t qb[EWSJF_MAX_QUEUES];  // bounds: qb[i] separates queues i and i + 1
  __shared__ uint8_t qmark[EWSJF_MAX_QUEUES];
  __shared__ int k2s;
  const int tid = threadIdx.x;
  const TacticalPlan p = *plan;
  const int t0 = p.take[0], t1 = p.take[1], t2 = p.take[2];
  for (int r = tid; r < B; r += kBlock) {
    int id = -1;
    if (r < t0) id = row_ids[r];
    else if (r < t0 + t1) id = row_ids[B + (r - t0)];
    else if (r < t0 + t1 + t2) id = row_ids[2 * B + (r - t0 - t1)];
    ids[r] = id;
    if (tomb_len != nullptr && id >= 0) tomb_len[id] = 0;
  }
  if (tid == 0) *n_sel = t0 + t1 + t2;
  const int k = p.k;
  if (removed != nullptr && tid < k) removed[tid] = 0;
  if (p.n_removed == 0 || k == 1) return;  // uniform: no barrier skipped by part of the block

  // Sequential removal on an LDS copy of the queue list (k <= 256).
  if (tid < k) {
    qn[tid] = tab->count[tid];
    qS[tid] = tab->sum[tid];
    qlo[tid] = tab->lo[tid];
    qhi[tid] = tab->hi[tid];
    qec[tid] = empty_cnt[tid];
    qorig[tid] = tid;
    qmark[tid] = cnt[tid] == 0 && empty_cnt[tid] > empty_threshold;
    if (tid + 1 < k) qb[tid] = tab->bounds[tid];
  }
  __syncthreads();
  if (tid == 0) {
    int kk = k;
    for (;;) {
      int r = -1;
      for (int i = 0; i < kk; ++i)
        if (qmark[i]) {
          r = i;
          break;
        }
      if (r < 0 || kk == 1) break;
      int a;
      if (r == 0) a = 1;
      else if (r + 1 == kk) a = r - 1;
      else
        a = eq3_utility(qn[r - 1], qS[r - 1], qlo[r - 1], qhi[r - 1], qn[r], qS[r], qlo[r], qhi[r], eps) <=
                    eq3_utility(qn[r], qS[r], qlo[r], qhi[r], qn[r + 1], qS[r + 1], qlo[r + 1], qhi[r + 1], eps)
                ? r - 1
                : r + 1;
      qn[a] += qn[r];
      qS[a] += qS[r];
      qlo[a] = min(qlo[a], qlo[r]);
      qhi[a] = max(qhi[a], qhi[r]);
      if (removed != nullptr) removed[qorig[r]] = 1;
      for (int i = min(r, a); i + 2 < kk; ++i) qb[i] = qb[i + 1];  // the boundary between r and a goes
      for (int i = r; i + 1 < kk; ++i) {
        qn[i] = qn[i + 1];
        qS[i] = qS[i + 1];
        qlo[i] = qlo[i + 1];
        qhi[i] = qhi[i + 1];
        qec[i] = qec[i + 1];
        qorig[i] = qorig[i + 1];
        qmark[i] = qmark[i + 1];
      }
      --kk;
    }
    k2s = kk;
  }
  __syncthreads();
  const int k2 = k2s;
  if (tid < k2) {
    tab->count[tid] = qn[tid];
    tab->sum[tid] = qS[tid];
    tab->lo[tid] = qlo[tid];
    tab->hi[tid] = qhi[tid];
    tab->mean[tid] = (double)qS[tid] / (double)qn[tid];
    if (tid > 0) tab->bounds[tid - 1] = qb[tid - 1];
    empty_cnt[tid] = qec[tid];
  }
  if (tid == 0) tab->k = k2;
  // Routing lut of the new set, in the table's reading (contiguous bounds or
  // gapped intervals).
  const int L = tab->max_len;
  const bool gapped = tab->gapped != 0;
  lut_fill(tab->lut, tid, kBlock, L, gapped, qb, qlo, qhi, k2);
  route_fill(tab->route, tid, kBlock, L, gapped, qb, qlo, qhi, k2);
}

}  // namespace

size_t tactical_ws_bytes(int64_t n, int32_t B) { return carve_tac(n, B, nullptr, nullptr); }

hipError_t launch_tactical_step(int32_t* len, const float* arrival, int64_t n, float now, ewsjf_queue_table* table,
                                const ewsjf_theta* theta, const ewsjf_cost& cost, int32_t B, int32_t empty_threshold,
                                int32_t* empty_cnt, double eps, int32_t* tomb_len, int32_t* ids, int32_t* n_sel,
                                int32_t* q_prim, float* head_score, int32_t* removed, void* ws, hipStream_t stream) {
  TacWs w;
  carve_tac(n, B, ws, &w);
  const int G = scan_grid(n);
  hipLaunchKernelGGL(tac_scan, dim3(G), dim3(kBlock), 0, stream, len, arrival, n, table, G, w.part_cnt, w.part_head);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(tac_reduce, dim3(EWSJF_MAX_QUEUES), dim3(kReduceThreads), 0, stream, w.part_cnt, w.part_head, G,
                     len, arrival, now, table, theta, cost, w.cnt, w.head, w.score);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(tac_plan, dim3(1), dim3(EWSJF_MAX_QUEUES), 0, stream, table, w.cnt, w.score, B, empty_threshold,
                     empty_cnt, w.plan, q_prim, head_score);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if ((e = launch_fifo_select(len, arrival, n, table, w.plan, B, w.row_ids, w.row_top, w.row_n, w.select_ws,
                              stream)) != hipSuccess)
    return e;
  hipLaunchKernelGGL(tac_finish, dim3(1), dim3(kBlock), 0, stream, w.plan, w.row_ids, B, tomb_len, ids, n_sel, table,
                     w.cnt, empty_threshold, empty_cnt, eps, removed);
  return hipGetLastError();
}

}  // namespace ewsjf
