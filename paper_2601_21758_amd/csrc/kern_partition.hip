// Refine-and-Prune (Section 4.2) on the GPU.
//
// The paper sorts the window (the O(N log N) step of the strategic loop).
// Prompt lengths are bounded integers, so a length histogram carries exactly
// the information of the sorted window: the distinct values in order and
// their multiplicities.  Kernels:
//
//   window_hist      LDS-privatized histogram of clamped window lengths, one
//                    partial histogram per workgroup (no global atomics).
//   hist_reduce      column sums of the partial histograms.
//   hist_clear /     the same histogram into a caller-owned array (of a
//   window_hist_add  window kept as a range of a ring of recent lengths),
//                    flushed with one global atomic per non-empty bin per
//                    workgroup; the partition can start from it.
//   window_hist_move the window moved forward by n entries: the counts of
//                    the lengths that leave it go to the ones that join it.
//   rp_distinct      one workgroup: distinct values v[], counts c[] and exact
//                    int64 prefix sums of counts and of count * value.
//   rp_kmeans3 /     the exact 1-D 3-means initializer: every split (i, j) of
//   rp_kmeans3_pick  the distinct values, binary64 objective, ties to the
//                    smallest (i, j).
//   rp_refine_prune  one workgroup: Stage 1 cluster starts, Stage 2 as
//                    level-synchronous passes (every significant gap of every
//                    current cluster is cut in the same pass; a pass without a
//                    new cut ends the recursion), Stage 3 greedy merges of the
//                    lowest-utility adjacent pair, then the queue table.
//
// Every binary64 expression is evaluated in the same order as the oracle's
// definition and the library is built without floating-point contraction, so
// boundaries, counts, sums and means agree bit for bit.
#include <hip/hip_runtime.h>

#include "ewsjf_device.h"
#include "ewsjf_launch.h"

namespace ewsjf {

namespace {

constexpr int kHistPerBlock = 16384;   // window entries per histogram workgroup
constexpr int kMaxHistBlocks = 64;
constexpr int kKmeansBlocks = 256;
constexpr int kLeafLds = 2048;         // Stage-3 leaves kept in LDS
constexpr uint64_t kInfBits = 0x7FF0000000000000ull;  // +inf as binary64 bits
constexpr int kBinsPerThread = EWSJF_MAX_LEN / kBlock;  // 32

// A Stage-3 leaf with its neighbours' links and the density and mean of the
// leaf after it (so one merge needs two rounds of LDS reads).  48 bytes.
struct alignas(16) Leaf {
  int64_t n, S;
  double rho, mean;      // n / (hi - lo + 1), S / n
  double rho_n, mean_n;  // the same of the next leaf (unused when nxt < 0)
  int32_t lo, hi;
  int32_t nxt, prv;      // -1: none; prv == -2 marks a merged-away leaf
};

struct PartWs {
  uint32_t* partial;  // [Gh][L+1]
  uint32_t* hist_buf; // [L+1] the window's histogram when the partition builds it
  const uint32_t* hist;  // the histogram the partition reads: hist_buf or the caller's
  int32_t* v;         // [L] distinct values
  uint32_t* c;        // [L] multiplicities
  int64_t* PN;        // [L+1] prefix sums of c
  int64_t* PS;        // [L+1] prefix sums of c * v
  int32_t* meta;      // [16]: 0 V, 1 km_i, 2 km_j
  double* km_F;       // [kKmeansBlocks]
  int32_t* km_ij;     // [kKmeansBlocks][2]
  int64_t* gn;        // [L] Stage-3 leaves (global mode)
  int64_t* gS;
  int32_t* glo;
  int32_t* ghi;
  Leaf* grec;         // [L] Stage-3 records when the leaves exceed LDS
  uint64_t* gU;       // [L]
  int Gh;
};

size_t up256(size_t x) { return (x + 255) & ~(size_t)255; }

int hist_blocks(int64_t n) {
  int64_t g = (n + kHistPerBlock - 1) / kHistPerBlock;
  if (g < 1) g = 1;
  if (g > kMaxHistBlocks) g = kMaxHistBlocks;
  return (int)g;
}

PartWs carve_part(void* ws, int64_t n, int L) {
  PartWs w;
  w.Gh = hist_blocks(n);
  char* b = static_cast<char*>(ws);
  size_t o = 0;
  auto take = [&](size_t bytes) {
    char* p = b + o;
    o += up256(bytes);
    return p;
  };
  w.partial = reinterpret_cast<uint32_t*>(take((size_t)w.Gh * (L + 1) * 4));
  w.hist_buf = reinterpret_cast<uint32_t*>(take((size_t)(L + 1) * 4));
  w.hist = w.hist_buf;
  w.v = reinterpret_cast<int32_t*>(take((size_t)L * 4));
  w.c = reinterpret_cast<uint32_t*>(take((size_t)L * 4));
  w.PN = reinterpret_cast<int64_t*>(take((size_t)(L + 1) * 8));
  w.PS = reinterpret_cast<int64_t*>(take((size_t)(L + 1) * 8));
  w.meta = reinterpret_cast<int32_t*>(take(16 * 4));
  w.km_F = reinterpret_cast<double*>(take(kKmeansBlocks * 8));
  w.km_ij = reinterpret_cast<int32_t*>(take(kKmeansBlocks * 8));
  w.gn = reinterpret_cast<int64_t*>(take((size_t)L * 8));
  w.gS = reinterpret_cast<int64_t*>(take((size_t)L * 8));
  w.glo = reinterpret_cast<int32_t*>(take((size_t)L * 4));
  w.ghi = reinterpret_cast<int32_t*>(take((size_t)L * 4));
  w.grec = reinterpret_cast<Leaf*>(take((size_t)L * sizeof(Leaf)));
  w.gU = reinterpret_cast<uint64_t*>(take((size_t)L * 8));
  return w;
}

size_t carve_size(int64_t n, int L) {
  PartWs w = carve_part(nullptr, n, L);
  return reinterpret_cast<size_t>(w.gU) + up256((size_t)L * 8);
}

// ---------------------------------------------------------------------------
// A window length as the partition counts it: clamped to [1, L].
__device__ __forceinline__ int clamp_len(int32_t b, int L) { return b < 1 ? 1 : (b > L ? L : b); }

// The entry i < n of a window kept as ring[(begin + i) mod cap] (begin < cap,
// n <= cap, so one subtraction wraps it).
__device__ __forceinline__ int32_t ring_at(const int32_t* __restrict__ ring, int64_t cap, int64_t begin, int64_t i) {
  int64_t j = begin + i;
  if (j >= cap) j -= cap;
  return ring[j];
}

// This workgroup's share of the n window entries counted into h[0..L] (LDS).
__device__ void lds_window_hist(const int32_t* __restrict__ ring, int64_t cap, int64_t begin, int64_t n, int L,
                                uint32_t* h) {
  for (int b = threadIdx.x; b <= L; b += kBlock) h[b] = 0u;
  __syncthreads();
  const int64_t per = (n + gridDim.x - 1) / gridDim.x;
  const int64_t beg = per * blockIdx.x;
  const int64_t end = beg + per < n ? beg + per : n;
  for (int64_t i = beg + threadIdx.x; i < end; i += kBlock)
    atomicAdd(&h[clamp_len(ring_at(ring, cap, begin, i), L)], 1u);
  __syncthreads();
}

__global__ __launch_bounds__(kBlock) void window_hist(const int32_t* __restrict__ win, int64_t n, int L,
                                                      uint32_t* __restrict__ partial) {
  __shared__ uint32_t h[EWSJF_MAX_LEN + 1];
  lds_window_hist(win, n, 0, n, L, h);
  uint32_t* out = partial + (size_t)blockIdx.x * (L + 1);
  for (int b = threadIdx.x; b <= L; b += kBlock) out[b] = h[b];
}

__global__ void hist_clear(uint32_t* __restrict__ hist, int L) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b <= L) hist[b] = 0u;
}

__global__ __launch_bounds__(kBlock) void window_hist_add(const int32_t* __restrict__ ring, int64_t cap,
                                                          int64_t begin, int64_t n, int L,
                                                          uint32_t* __restrict__ hist) {
  __shared__ uint32_t h[EWSJF_MAX_LEN + 1];
  lds_window_hist(ring, cap, begin, n, L, h);
  for (int b = threadIdx.x; b <= L; b += kBlock)
    if (h[b]) atomicAdd(&hist[b], h[b]);
}

__global__ void hist_reduce(const uint32_t* __restrict__ partial, int Gh, int L, uint32_t* __restrict__ hist) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b > L) return;
  uint32_t s = 0;
  for (int g = 0; g < Gh; ++g) s += partial[(size_t)g * (L + 1) + b];
  hist[b] = s;
}

// The window moves forward by n entries: the counts of the n lengths that
// leave it (ring[(sub + i) mod cap]) move to the n that join it
// (ring[(add + i) mod cap]).  Per-workgroup signed deltas in LDS, flushed as
// modular uint32 adds: the final counts are exact in any flush order.
__global__ __launch_bounds__(kBlock) void window_hist_move(const int32_t* __restrict__ ring, int64_t cap, int64_t add,
                                                           int64_t sub, int64_t n, int L,
                                                           uint32_t* __restrict__ hist) {
  __shared__ int32_t d[EWSJF_MAX_LEN + 1];
  for (int b = threadIdx.x; b <= L; b += kBlock) d[b] = 0;
  __syncthreads();
  const int64_t per = (n + gridDim.x - 1) / gridDim.x;
  const int64_t beg = per * blockIdx.x;
  const int64_t end = beg + per < n ? beg + per : n;
  for (int64_t i = beg + threadIdx.x; i < end; i += kBlock) {
    const int ca = clamp_len(ring_at(ring, cap, add, i), L);
    const int cs = clamp_len(ring_at(ring, cap, sub, i), L);
    if (ca != cs) {
      atomicAdd(&d[ca], 1);
      atomicSub(&d[cs], 1);
    }
  }
  __syncthreads();
  for (int b = threadIdx.x; b <= L; b += kBlock)
    if (d[b]) atomicAdd(&hist[b], (uint32_t)d[b]);
}

// Exclusive int64 block scan (kBlock threads).
__device__ int64_t block_exclusive_scan64(int64_t x, int64_t* scratch, int64_t* total) {
  const int lane = threadIdx.x & (kWave - 1), wv = threadIdx.x / kWave;
  int64_t incl = x;
  for (int off = 1; off < kWave; off <<= 1) {
    const int64_t y = __shfl_up(incl, off);
    if (lane >= off) incl += y;
  }
  __syncthreads();
  if (lane == kWave - 1) scratch[wv] = incl;
  __syncthreads();
  int64_t base = 0, sum = 0;
  for (int i = 0; i < kWavesPerBlock; ++i) {
    if (i < wv) base += scratch[i];
    sum += scratch[i];
  }
  __syncthreads();
  *total = sum;
  return base + incl - x;
}

// Distinct values and exact prefix sums, one workgroup.  Wave w covers the
// bins [2048 w, 2048 w + 2048) and its lane l the 32 bins from
// 2048 w + 32 l (bin 0 is not a length; the last thread also takes bin
// 32768), so the distinct values come out in thread order.  The bins arrive
// by coalesced loads, 64 consecutive bins per load, all issued before any is
// used (bounded: past bin L they read 0), and are transposed through the
// wave's region of LDS, where each lane reads its 32 bins twice: for its
// totals, and after the scans for its outputs (nothing is held in registers
// across the scans).
constexpr int kDistinctRegion = kBinsPerThread * kWave + kWave;  // 2048 bins, one pad word per 32

__device__ __forceinline__ int pad32(int i) { return i + (i >> 5); }

__global__ __launch_bounds__(kBlock) void rp_distinct(PartWs w, int L) {
  static_assert(kBinsPerThread * kBlock == EWSJF_MAX_LEN, "every bin below the largest length has one owner");
  __shared__ uint32_t stage[kWavesPerBlock * kDistinctRegion];
  __shared__ int64_t scr[kWavesPerBlock];
  __shared__ int iscr[kWavesPerBlock];
  const int t = threadIdx.x, lane = t & (kWave - 1), wv = t / kWave;
  uint32_t* reg = stage + wv * kDistinctRegion;
  const int wbin = wv * kBinsPerThread * kWave;
  {
    const __amdgpu_buffer_rsrc_t rs =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<uint32_t*>(w.hist), (short)0, (L + 1) * 4, kBufferWord3);
    uint32_t x[kBinsPerThread];
#pragma unroll
    for (int q = 0; q < kBinsPerThread; ++q)
      x[q] = __builtin_amdgcn_raw_buffer_load_b32(rs, (wbin + q * kWave + lane) * 4, 0, 0);
#pragma unroll
    for (int q = 0; q < kBinsPerThread; ++q) reg[pad32(q * kWave + lane)] = x[q];
    if (t == 0) reg[0] = 0u;  // bin 0 is not a length
  }
  // Bin EWSJF_MAX_LEN, the last thread's extra bin (read only when it is a length).
  const uint32_t hx = (t == kBlock - 1 && L >= EWSJF_MAX_LEN) ? w.hist[EWSJF_MAX_LEN] : 0u;
  __syncthreads();
  const int b0 = wbin + lane * kBinsPerThread;  // this thread's first bin
  const uint32_t* mine = reg + pad32(lane * kBinsPerThread);  // its 32 bins, contiguous after padding
  int nz = hx != 0u;
  int64_t cn = hx, cs = (int64_t)hx * EWSJF_MAX_LEN;
#pragma unroll
  for (int k = 0; k < kBinsPerThread; ++k) {
    const uint32_t h = mine[k];
    nz += h != 0u;
    cn += h;
    cs += (int64_t)h * (b0 + k);
  }
  int V = 0;
  int64_t totN = 0, totS = 0;
  int pos = block_exclusive_scan(nz, iscr, &V);
  int64_t pn = block_exclusive_scan64(cn, scr, &totN);
  int64_t ps = block_exclusive_scan64(cs, scr, &totS);
  // Outputs, each lane's run of positions in bin order.
  auto put = [&](uint32_t h, int b) {
    if (h != 0u) {
      w.v[pos] = b;
      w.c[pos] = h;
      w.PN[pos] = pn;
      w.PS[pos] = ps;
      pn += h;
      ps += (int64_t)h * b;
      ++pos;
    }
  };
#pragma unroll
  for (int k = 0; k < kBinsPerThread; ++k) put(mine[k], b0 + k);
  put(hx, EWSJF_MAX_LEN);
  if (t == 0) {
    w.PN[V] = totN;
    w.PS[V] = totS;
    w.meta[0] = V;
    w.meta[1] = -1;
    w.meta[2] = -1;
  }
}

// Exact 1-D 3-means over splits 1 <= i < j <= V-1 of the distinct values.
__device__ __forceinline__ bool km_better(double F, int i, int j, double bF, int bi, int bj) {
  if (F > bF) return true;
  if (F < bF) return false;
  return i < bi || (i == bi && j < bj);
}

__global__ __launch_bounds__(kBlock) void rp_kmeans3(PartWs w) {
  __shared__ double sF[kWavesPerBlock];
  __shared__ int si[kWavesPerBlock], sj[kWavesPerBlock];
  const int V = w.meta[0];
  double bF = -1.0;
  int bi = 0x7fffffff, bj = 0x7fffffff;
  if (V > 3) {
    const double nV = (double)w.PN[V], sV = (double)w.PS[V];
    (void)nV;
    (void)sV;
    for (int i = 1 + blockIdx.x; i <= V - 2; i += gridDim.x) {
      const int64_t Ni = w.PN[i], Si = w.PS[i];
      for (int j = i + 1 + threadIdx.x; j <= V - 1; j += kBlock) {
        const int64_t Nj = w.PN[j], Sj = w.PS[j];
        const double n1 = (double)Ni, s1 = (double)Si;
        const double n2 = (double)(Nj - Ni), s2 = (double)(Sj - Si);
        const double n3 = (double)(w.PN[V] - Nj), s3 = (double)(w.PS[V] - Sj);
        const double F = ((s1 * s1) / n1 + (s2 * s2) / n2) + (s3 * s3) / n3;
        if (km_better(F, i, j, bF, bi, bj)) {
          bF = F;
          bi = i;
          bj = j;
        }
      }
    }
  }
  // block argmax with the tie rule
  for (int off = 32; off > 0; off >>= 1) {
    const double oF = __shfl_xor(bF, off);
    const int oi = __shfl_xor(bi, off), oj = __shfl_xor(bj, off);
    if (km_better(oF, oi, oj, bF, bi, bj)) {
      bF = oF;
      bi = oi;
      bj = oj;
    }
  }
  const int lane = threadIdx.x & (kWave - 1), wv = threadIdx.x / kWave;
  if (lane == 0) {
    sF[wv] = bF;
    si[wv] = bi;
    sj[wv] = bj;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int q = 0; q < kWavesPerBlock; ++q)
      if (km_better(sF[q], si[q], sj[q], bF, bi, bj)) {
        bF = sF[q];
        bi = si[q];
        bj = sj[q];
      }
    w.km_F[blockIdx.x] = bF;
    w.km_ij[2 * blockIdx.x] = bi;
    w.km_ij[2 * blockIdx.x + 1] = bj;
  }
}

__global__ void rp_kmeans3_pick(PartWs w, int nblocks) {
  if (threadIdx.x != 0) return;
  double bF = -1.0;
  int bi = 0x7fffffff, bj = 0x7fffffff;
  for (int q = 0; q < nblocks; ++q)
    if (km_better(w.km_F[q], w.km_ij[2 * q], w.km_ij[2 * q + 1], bF, bi, bj)) {
      bF = w.km_F[q];
      bi = w.km_ij[2 * q];
      bj = w.km_ij[2 * q + 1];
    }
  w.meta[1] = bi;
  w.meta[2] = bj;
}

// ---------------------------------------------------------------------------
// Stage 3 utility of the adjacent pair (a, b), Eq. 3 with density = count per
// token of value span.  Same binary64 expression order as the definition.
// ---------------------------------------------------------------------------
__device__ __forceinline__ double utility(int64_t na, int64_t Sa, int32_t loa, int32_t hia, int64_t nb, int64_t Sb,
                                          int32_t lob, int32_t hib, double eps) {
  const double rho_a = (double)na / (double)((int64_t)hia - (int64_t)loa + 1);
  const double rho_b = (double)nb / (double)((int64_t)hib - (int64_t)lob + 1);
  const double m_a = (double)Sa / (double)na;
  const double m_b = (double)Sb / (double)nb;
  return (rho_a + rho_b) / (fabs(m_b - m_a) + eps);
}

// The same expression on per-leaf densities and means computed once (the
// division results are identical to recomputing them).
__device__ __forceinline__ double utility_cached(double rho_a, double m_a, double rho_b, double m_b, double eps) {
  return (rho_a + rho_b) / (fabs(m_b - m_a) + eps);
}

__device__ __forceinline__ uint64_t dbits(double x) { return (uint64_t)__double_as_longlong(x); }


struct ArgMin {
  double u;
  int i;
};

__device__ __forceinline__ ArgMin argmin_pick(ArgMin a, ArgMin b) {
  if (b.u < a.u || (b.u == a.u && b.i < a.i)) return b;
  return a;
}

__device__ ArgMin block_argmin(ArgMin x, double* su, int* si) {
  for (int off = 32; off > 0; off >>= 1) {
    ArgMin o;
    o.u = __shfl_xor(x.u, off);
    o.i = __shfl_xor(x.i, off);
    x = argmin_pick(x, o);
  }
  const int lane = threadIdx.x & (kWave - 1), wv = threadIdx.x / kWave;
  __syncthreads();
  if (lane == 0) {
    su[wv] = x.u;
    si[wv] = x.i;
  }
  __syncthreads();
  ArgMin r{su[0], si[0]};
  for (int q = 1; q < kWavesPerBlock; ++q) r = argmin_pick(r, ArgMin{su[q], si[q]});
  __syncthreads();
  return r;
}

// The distinct values and the cluster-start flags sit in LDS padded by 4
// bytes per 32 entries (vat / sat): a thread owns 32 consecutive entries,
// and without the padding the lanes of a wave read them 64 (values) or 32
// (flags) bytes apart, 16- and 8-way bank conflicts.
struct RpShared {
  union {
    struct {
      uint16_t v[EWSJF_MAX_LEN + 2 * (EWSJF_MAX_LEN / 32)];
      uint8_t start[EWSJF_MAX_LEN + 4 * (EWSJF_MAX_LEN / 32)];
    } a;
  } u;
  int64_t scr64[kWavesPerBlock];
  double su[kWavesPerBlock];
  int si[kWavesPerBlock];
  int iscr[kWavesPerBlock];
  int flag;
};

__device__ __forceinline__ uint16_t& vat(RpShared& sm, int j) { return sm.u.a.v[j + 2 * (j >> 5)]; }
__device__ __forceinline__ uint8_t& sat(RpShared& sm, int j) { return sm.u.a.start[j + 4 * (j >> 5)]; }

// For thread-owned index ranges [j0, j0 + 32): carry_s = the last segment
// start before j0 (-1 if none), carry_e = the first segment start after the
// range (V if none).
__device__ void segment_carries(RpShared& sm, int V, int j0, int* carry_s, int* carry_e) {
  const int tid = threadIdx.x;
  int last = -1, first = 0x7fffffff;
  for (int q = 0; q < kBinsPerThread; ++q) {
    const int j = j0 + q;
    if (j < V && sat(sm, j)) {
      last = j;
      if (first == 0x7fffffff) first = j;
    }
  }
  const int lane = tid & (kWave - 1), wv = tid / kWave;
  int incl = last;
  for (int off = 1; off < kWave; off <<= 1) {
    const int y = __shfl_up(incl, off);
    if (lane >= off) incl = incl > y ? incl : y;
  }
  int rincl = first;
  for (int off = 1; off < kWave; off <<= 1) {
    const int y = __shfl_down(rincl, off);
    if (lane + off < kWave) rincl = rincl < y ? rincl : y;
  }
  __syncthreads();
  if (lane == kWave - 1) sm.iscr[wv] = incl;
  if (lane == 0) sm.si[wv] = rincl;
  __syncthreads();
  int wmax = -1, wmin = 0x7fffffff;
  for (int q = 0; q < wv; ++q) wmax = sm.iscr[q] > wmax ? sm.iscr[q] : wmax;
  for (int q = wv + 1; q < kWavesPerBlock; ++q) wmin = sm.si[q] < wmin ? sm.si[q] : wmin;
  const int prev_in_wave = __shfl_up(incl, 1);
  const int next_in_wave = __shfl_down(rincl, 1);
  const int cs = lane > 0 ? (prev_in_wave > wmax ? prev_in_wave : wmax) : wmax;
  const int ce = lane < kWave - 1 ? (next_in_wave < wmin ? next_in_wave : wmin) : wmin;
  __syncthreads();
  *carry_s = cs;
  *carry_e = ce < V ? ce : V;
}

// The queue table from k queue aggregates in length order.
template <class N, class Lo>
__device__ void write_queues(ewsjf_queue_table* tab, int k, const N* n, const N* S, const Lo* lo, const Lo* hi,
                             int tid, int nthreads) {
  for (int i = tid; i < k; i += nthreads) {
    const int64_t cn = n[i], cs = S[i];
    const int32_t l = lo[i], h = hi[i];
    if (i > 0) tab->bounds[i - 1] = l;
    tab->lo[i] = l;
    tab->hi[i] = h;
    tab->count[i] = cn;
    tab->sum[i] = cs;
    tab->mean[i] = (double)cs / (double)cn;
  }
  if (tid == 0) tab->k = k;
}

__global__ __launch_bounds__(kBlock) void rp_refine_prune(PartWs w, ewsjf_partition_params p, int64_t n_window,
                                                          ewsjf_queue_table* tab) {
  __shared__ RpShared sm;
  const int tid = threadIdx.x;
  const int V = w.meta[0];
  const int L = p.max_len;
  if (V == 0) {
    // An empty histogram (only a caller-kept one can be empty): one queue
    // that holds nothing and covers every length.
    if (tid == 0) {
      w.meta[3] = 0;
      tab->k = 1;
      tab->max_len = L;
      tab->n_distinct = tab->n_coarse = tab->n_leaves = tab->gapped = 0;
      tab->n_window = 0;
      tab->lo[0] = tab->hi[0] = 0;
      tab->count[0] = tab->sum[0] = 0;
      tab->mean[0] = 0.0;
    }
    return;
  }

  // ---- Stage 1: coarse cluster starts -------------------------------------
  {
    // Every load is issued before the first store (bounded: past V they read 0).
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(w.v, (short)0, V * 4, kBufferWord3);
    uint32_t x[kBinsPerThread];
#pragma unroll
    for (int k = 0; k < kBinsPerThread; ++k)
      x[k] = __builtin_amdgcn_raw_buffer_load_b32(rs, (tid + k * kBlock) * 4, 0, 0);
#pragma unroll
    for (int k = 0; k < kBinsPerThread; ++k)
      if (tid + k * kBlock < V) vat(sm, tid + k * kBlock) = (uint16_t)x[k];
  }
  __syncthreads();
  const int64_t vlo = vat(sm, 0), vhi = vat(sm, V - 1);
  if (p.init_mode == EWSJF_INIT_EQUAL_WIDTH) {
    const int64_t width = vhi - vlo + 1;
    for (int j = tid; j < V; j += kBlock) {
      uint8_t s = 1;
      if (j > 0) {
        // (v - lo) K < 2^30 (values and K are at most 32768): the 32-bit
        // quotient is the exact floor of the int64 definition.
        const uint32_t b1 = (uint32_t)(vat(sm, j) - vlo) * (uint32_t)p.init_queues / (uint32_t)width;
        const uint32_t b0 = (uint32_t)(vat(sm, j - 1) - vlo) * (uint32_t)p.init_queues / (uint32_t)width;
        s = b1 != b0;
      }
      sat(sm, j) = s;
    }
  } else {
    const int ki = w.meta[1], kj = w.meta[2];
    for (int j = tid; j < V; j += kBlock) {
      uint8_t s;
      if (V <= 3) s = 1;
      else s = (j == 0 || j == ki || j == kj) ? 1 : 0;
      sat(sm, j) = s;
    }
  }
  __syncthreads();
  int n_coarse = 0;
  {
    int cnt = 0;
    for (int j = tid; j < V; j += kBlock) cnt += sat(sm, j);
    int tot = 0;
    block_exclusive_scan(cnt, sm.iscr, &tot);
    n_coarse = tot;
  }

  // ---- Stage 2: level-synchronous refinement --------------------------------
  // Thread t owns distinct indices [32t, 32t + 32).
  const int j0 = tid * kBinsPerThread;
  const int min_distinct = p.gap_mode == EWSJF_GAPS_DISTINCT ? 3 : 2;
  int carry_s = -1, carry_e = V;
  for (;;) {
    segment_carries(sm, V, j0, &carry_s, &carry_e);
    // This thread's segment starts as a bit mask (bit q: index j0 + q); the
    // segment [s, e) holding index j0 + q starts at the highest set bit <= q
    // (else carry_s) and ends at the lowest set bit > q (else carry_e).
    // Branch-free and unrolled, so the LDS reads of all 32 gaps are issued
    // together; indices of gaps that are not tested are clamped to 0.
    uint32_t mask = 0u;
#pragma unroll
    for (int q = 0; q < kBinsPerThread; ++q) mask |= (uint32_t)(j0 + q < V && sat(sm, j0 + q)) << q;
    uint32_t newcuts = 0;
#pragma unroll
    for (int q = 0; q < kBinsPerThread; ++q) {
      const int j = j0 + q;
      const uint32_t below = mask & (0xFFFFFFFFu >> (31 - q));
      const int s = below ? j0 + 31 - __clz((int)below) : carry_s;
      const uint32_t above = q < 31 ? mask >> (q + 1) : 0u;
      const int e = above ? j + __ffs((int)above) : carry_e;
      // the gap between j and j+1 inside the segment [s, e)
      const bool gap = j + 1 < e;  // (e <= V, so j + 1 < V)
      const int VC = e - s;
      const int64_t span = (int64_t)vat(sm, gap ? e - 1 : 0) - (int64_t)vat(sm, gap ? s : 0);
      const bool test = gap && VC >= min_distinct && span >= (int64_t)p.min_width;
      // span, the gap and VC - 1 fit in int32 (values are at most 32768), so
      // they convert to binary64 in one exact step; the count-mode m - 1 is
      // an int64 count.
      const double mm1 = p.gap_mode == EWSJF_GAPS_DISTINCT ? (double)(VC - 1)
                                                           : (double)(test ? (w.PN[e] - w.PN[s]) - 1 : 0);
      const double rhs = p.alpha * (double)(int)span;
      const double lhs = (double)((int)vat(sm, gap ? j + 1 : 0) - (int)vat(sm, gap ? j : 0)) * mm1;
      if (test && lhs > rhs) newcuts |= 1u << q;
    }
    const int any = __syncthreads_or(newcuts != 0);
    if (!any) break;
    for (int q = 0; q < kBinsPerThread; ++q)
      if (newcuts & (1u << q)) sat(sm, j0 + q + 1) = 1;
    __syncthreads();
  }

  // ---- Leaves: one per segment, aggregates from the exact prefix sums -------
  // The segment starts are listed in order (in the Stage-3 workspace, which
  // rp_merge rewrites later), then each thread builds whole leaves: four
  // independent prefix-sum loads per leaf instead of a chain per thread.
  int nl = 0;
  {
    int cnt = 0;
    for (int q = 0; q < kBinsPerThread; ++q) {
      const int j = j0 + q;
      if (j < V) cnt += sat(sm, j);
    }
    int tot = 0;
    int pos = block_exclusive_scan(cnt, sm.iscr, &tot);
    nl = tot;
    int32_t* starts = reinterpret_cast<int32_t*>(w.gU);
    for (int q = 0; q < kBinsPerThread; ++q) {
      const int j = j0 + q;
      if (j < V && sat(sm, j)) starts[pos++] = j;
    }
    __syncthreads();
    for (int i = tid; i < nl; i += kBlock) {
      const int s = starts[i];
      const int e = i + 1 < nl ? starts[i + 1] : V;
      w.gn[i] = w.PN[e] - w.PN[s];
      w.gS[i] = w.PS[e] - w.PS[s];
      w.glo[i] = vat(sm, s);
      w.ghi[i] = vat(sm, e - 1);
    }
  }
  __threadfence();
  __syncthreads();
  const int n_leaves = nl;
  if (tid == 0) {
    w.meta[3] = n_leaves;
    tab->max_len = L;
    tab->n_distinct = V;
    tab->n_coarse = n_coarse;
    tab->n_leaves = n_leaves;
    tab->gapped = 0;
    tab->n_window = n_window >= 0 ? n_window : w.PN[V];
  }
  // Within the queue budget: the leaves are the queues.  Otherwise Stage 3
  // (rp_merge) writes them.
  if (nl <= p.max_queues) write_queues(tab, nl, w.gn, w.gS, w.glo, w.ghi, tid, kBlock);
}

}  // namespace

// ---------------------------------------------------------------------------
// Stage 3: greedy merge of the adjacent pair with the smallest utility until
// at most max_queues remain (Section 4.2, "Stage 3", Eq. 3).
//
// The merge is sequential (each merge changes its neighbours' utilities), so
// one wave runs it.  Leaves keep their index (a linked list replaces
// shifting), and lane l caches the minimum utility over the pairs it owns
// (left-leaf indices [l*P, l*P + P)).  A merge costs a two-step wave
// reduction for the global minimum, two rounds of record reads and a rescan
// by the few lanes whose pairs changed.  Utilities are non-negative binary64
// values, so their bit patterns order like the values; ties go to the smaller
// leaf index, which is the smaller position in the list.  The records live in
// LDS, or in the workspace when there are more leaves than LDS holds.
// ---------------------------------------------------------------------------
constexpr int kMergeThreads = 256;

// Lowest lane holding the wave's minimum of x, and that minimum (*m).  The
// high words are reduced first, the low words only when several lanes share
// the smallest high word (utilities rarely do).
__device__ __forceinline__ int wave_argmin_u64(uint64_t x, uint64_t* m) {
  const uint32_t xh = (uint32_t)(x >> 32);
  const uint32_t mh = __ockl_wfred_min_u32(xh);
  uint64_t cand = __ballot(xh == mh);
  if (__popcll(cand) > 1) {
    const uint32_t ml = __ockl_wfred_min_u32(xh == mh ? (uint32_t)x : 0xFFFFFFFFu);
    cand = __ballot(xh == mh && (uint32_t)x == ml);
  }
  const int src = (int)__builtin_ctzll(cand);
  *m = ((uint64_t)mh << 32) | (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)x, src);
  return src;
}

template <bool kInLds>
__device__ __forceinline__ void stage3(Leaf* rec, uint64_t* U, const PartWs& w, int nl0,
                                       const ewsjf_partition_params& p, ewsjf_queue_table* tab, int* iscr) {
  const int tid = threadIdx.x;
  for (int i = tid; i < nl0; i += kMergeThreads) {
    Leaf r;
    r.n = w.gn[i];
    r.S = w.gS[i];
    r.lo = w.glo[i];
    r.hi = w.ghi[i];
    r.rho = (double)r.n / (double)((int64_t)r.hi - (int64_t)r.lo + 1);
    r.mean = (double)r.S / (double)r.n;
    r.nxt = i + 1 < nl0 ? i + 1 : -1;
    r.prv = i - 1;
    r.rho_n = r.mean_n = 0.0;
    if (i + 1 < nl0) {
      const int64_t n1 = w.gn[i + 1], S1 = w.gS[i + 1];
      r.rho_n = (double)n1 / (double)((int64_t)w.ghi[i + 1] - (int64_t)w.glo[i + 1] + 1);
      r.mean_n = (double)S1 / (double)n1;
    }
    rec[i] = r;
    U[i] = i + 1 < nl0 ? dbits(utility_cached(r.rho, r.mean, r.rho_n, r.mean_n, p.eps)) : kInfBits;
  }
  __syncthreads();
  if (tid < kWave) {
    const int lane = tid;
    // Each lane owns P slots, P the power of two >= nl0 / 64 (owners by shift).
    int lgP = 0;
    while ((kWave << lgP) < nl0) ++lgP;
    const int P = 1 << lgP;
    // This lane's minimum (first index on ties) over its P slots.
    auto scan_own = [&](uint64_t& mu, int& mi) {
      mu = kInfBits + 1;  // above every utility, +inf included
      mi = 0x7fffffff;
#pragma unroll 8
      for (int q = 0; q < P; ++q) {
        const int i = (lane << lgP) + q;
        const uint64_t u = i < nl0 ? U[i] : ~0ull;
        if (u < mu) {
          mu = u;
          mi = i;
        }
      }
    };
    uint64_t lane_u;
    int lane_i;
    scan_own(lane_u, lane_i);
    // Lane `owner`'s minimum recomputed by the whole wave, one slot per lane
    // (P <= kWave when the records are in LDS).
    auto rescan = [&](int owner) {
      if constexpr (kInLds) {
        const int i = (owner << lgP) + lane;
        const uint64_t u = (lane < P && i < nl0) ? U[i] : ~0ull;
        uint64_t m;
        const int src = wave_argmin_u64(u, &m);
        if (lane == owner) {
          lane_u = m == ~0ull ? kInfBits + 1 : m;
          lane_i = m == ~0ull ? 0x7fffffff : (owner << lgP) + src;
        }
      } else {
        if (lane == owner) scan_own(lane_u, lane_i);
      }
    };
    for (int alive = nl0; alive > p.max_queues; --alive) {
      uint64_t mu;
      const int a = __builtin_amdgcn_readlane(lane_i, wave_argmin_u64(lane_u, &mu));
      const int b = rec[a].nxt, pr = rec[a].prv;
      const int64_t na = rec[a].n + rec[b].n;
      const int64_t Sa = rec[a].S + rec[b].S;
      const int32_t hia = rec[b].hi;
      const int c = rec[b].nxt;
      const double rho_c = rec[b].rho_n, mean_c = rec[b].mean_n;
      const double rho_a = (double)na / (double)((int64_t)hia - (int64_t)rec[a].lo + 1);
      const double m_a = (double)Sa / (double)na;
      const uint64_t Ua = c >= 0 ? dbits(utility_cached(rho_a, m_a, rho_c, mean_c, p.eps)) : kInfBits;
      const uint64_t Upr = pr >= 0 ? dbits(utility_cached(rec[pr].rho, rec[pr].mean, rho_a, m_a, p.eps)) : kInfBits;
      if (lane == 0) {
        rec[a].n = na;
        rec[a].S = Sa;
        rec[a].hi = hia;
        rec[a].rho = rho_a;
        rec[a].mean = m_a;
        rec[a].rho_n = rho_c;
        rec[a].mean_n = mean_c;
        rec[a].nxt = c;
        rec[b].prv = -2;
        if (c >= 0) rec[c].prv = a;
        if (pr >= 0) {
          rec[pr].rho_n = rho_a;
          rec[pr].mean_n = m_a;
          U[pr] = Upr;
        }
        U[b] = kInfBits;
        U[a] = Ua;
      }
      // Lane 0's stores before anyone's next reads: LDS serves one wave in
      // order; the workspace needs a fence.
      if constexpr (!kInLds) __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");
      // Cached minima that may be stale: a's owner (its minimum was a, now
      // Ua), b's owner if its minimum was b (now removed), pr's owner if its
      // minimum was pr (now Upr).  A value that improves a minimum is taken
      // directly; otherwise the owner's slots are rescanned.
      const int oa = a >> lgP, ob = b >> lgP, op = pr >= 0 ? pr >> lgP : -1;
      const bool lower_a = Ua < mu;  // still the global minimum: a keeps it
      bool stale = false;
      if (lane == oa) {
        if (lower_a) lane_u = Ua;  // lane_i == a already
        else stale = true;
      }
      if (lane == ob && lane_i == b) stale = true;
      if (lane == op) {
        if (Upr < lane_u || (Upr == lane_u && pr < lane_i)) {
          lane_u = Upr;
          lane_i = pr;
        } else if (lane_i == pr) {
          stale = true;
        }
      }
      uint64_t todo = __ballot(stale);
      while (todo != 0ull) {
        const int owner = (int)__builtin_ctzll(todo);
        todo &= todo - 1;
        rescan(owner);
      }
    }
  }
  __syncthreads();
  // Survivors in index (= length) order are the queues.
  const int per = (nl0 + kMergeThreads - 1) / kMergeThreads;
  const int i0 = tid * per;
  int cnt = 0;
  for (int q = 0; q < per; ++q)
    if (i0 + q < nl0 && rec[i0 + q].prv != -2) ++cnt;
  int tot = 0;
  int pos = block_exclusive_scan_n(cnt, iscr, &tot, kMergeThreads);
  for (int q = 0; q < per; ++q) {
    const int i = i0 + q;
    if (i < nl0 && rec[i].prv != -2) {
      const Leaf& r = rec[i];
      if (pos > 0) tab->bounds[pos - 1] = r.lo;
      tab->lo[pos] = r.lo;
      tab->hi[pos] = r.hi;
      tab->count[pos] = r.n;
      tab->sum[pos] = r.S;
      tab->mean[pos] = (double)r.S / (double)r.n;
      ++pos;
    }
  }
  if (tid == 0) tab->k = tot;
}

__global__ __launch_bounds__(kMergeThreads) void rp_merge(PartWs w, ewsjf_partition_params p,
                                                          ewsjf_queue_table* tab) {
  __shared__ Leaf srec[kLeafLds];
  __shared__ uint64_t sU[kLeafLds];
  __shared__ int iscr[kMergeThreads / kWave];
  const int nl = w.meta[3];
  if (nl <= p.max_queues) return;  // rp_refine_prune wrote the queues
  if (nl <= kLeafLds)
    stage3<true>(srec, sU, w, nl, p, tab, iscr);
  else
    stage3<false>(w.grec, w.gU, w, nl, p, tab, iscr);
}

size_t partition_ws_bytes(int64_t n_window, const ewsjf_partition_params& p) {
  return carve_size(n_window, p.max_len);
}

namespace {

// Stages 1-3 and the routing lut from the histogram w.hist (n_window < 0:
// the table records the histogram's total as the window size).
hipError_t launch_stages(const PartWs& w, const ewsjf_partition_params& p, int64_t n_window, ewsjf_queue_table* table,
                         hipStream_t stream) {
  const int L = p.max_len;
  hipLaunchKernelGGL(rp_distinct, dim3(1), dim3(kBlock), 0, stream, w, L);
  if (p.init_mode == EWSJF_INIT_KMEANS3) {
    hipLaunchKernelGGL(rp_kmeans3, dim3(kKmeansBlocks), dim3(kBlock), 0, stream, w);
    hipLaunchKernelGGL(rp_kmeans3_pick, dim3(1), dim3(64), 0, stream, w, kKmeansBlocks);
  }
  hipLaunchKernelGGL(rp_refine_prune, dim3(1), dim3(kBlock), 0, stream, w, p, n_window, table);
  hipLaunchKernelGGL(rp_merge, dim3(1), dim3(kMergeThreads), 0, stream, w, p, table);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_build_lut(table, stream);
}

}  // namespace

hipError_t launch_partition(const int32_t* window, int64_t n_window, const ewsjf_partition_params& p,
                            ewsjf_queue_table* table, void* ws, hipStream_t stream) {
  const int L = p.max_len;
  PartWs w = carve_part(ws, n_window, L);
  hipLaunchKernelGGL(window_hist, dim3(w.Gh), dim3(kBlock), 0, stream, window, n_window, L, w.partial);
  hipLaunchKernelGGL(hist_reduce, dim3((L + 1 + 255) / 256), dim3(256), 0, stream, w.partial, w.Gh, L, w.hist_buf);
  return launch_stages(w, p, n_window, table, stream);
}

hipError_t launch_partition_hist(const uint32_t* hist, const ewsjf_partition_params& p, ewsjf_queue_table* table,
                                 void* ws, hipStream_t stream) {
  PartWs w = carve_part(ws, 0, p.max_len);
  w.hist = hist;
  return launch_stages(w, p, -1, table, stream);
}

hipError_t launch_window_histogram(const int32_t* ring, int64_t cap, int64_t begin, int64_t n, int L, uint32_t* hist,
                                   hipStream_t stream) {
  hipLaunchKernelGGL(hist_clear, dim3((L + 1 + 255) / 256), dim3(256), 0, stream, hist, L);
  if (n > 0)
    hipLaunchKernelGGL(window_hist_add, dim3(hist_blocks(n)), dim3(kBlock), 0, stream, ring, cap, begin, n, L, hist);
  return hipGetLastError();
}

hipError_t launch_window_advance(const int32_t* ring, int64_t cap, int64_t add, int64_t sub, int64_t n, int L,
                                 uint32_t* hist, hipStream_t stream) {
  hipLaunchKernelGGL(window_hist_move, dim3(hist_blocks(n)), dim3(kBlock), 0, stream, ring, cap, add, sub, n, L,
                     hist);
  return hipGetLastError();
}

}  // namespace ewsjf
