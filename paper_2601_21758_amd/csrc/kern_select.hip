// Top-B admission (fused with routing and scoring for ewsjf_step).
//
// Two kernels per call, no grid-wide synchronization:
//
//  local_candidates  (grid = G x n_theta workgroups of 1024 threads)
//    Each workgroup owns the 256-request chunks c with c % G == blockIdx.x, so
//    a run of old (high-scoring) requests with neighbouring ids is spread over
//    many workgroups.  Each lane holds 16 requests' 64-bit composite keys in
//    registers.  Every wave takes the m-th largest lane maximum as its bar,
//    the workgroup the largest bar t; every element with key >= t goes to an
//    LDS list, which is sorted and cut to at most M entries.  The workgroup
//    writes the list and a completeness bound T: every element of its share
//    whose composite is >= T is in the list.
//
//  merge_candidates  (grid = n_theta workgroups of 1024 threads)
//    Loads all lists into LDS and selects the exact top-B of their union.  If
//    some workgroup's bound T exceeds the B-th composite, elements of that
//    share could be missing; the merge kernel then re-reads exactly those
//    shares from the source and merges what it finds (the exact fallback).
//
// The composite key (score key << 32 | ~id) is unique per request, so the
// order (score desc, id asc) is total and the admitted set is unique.
#include <hip/hip_runtime.h>

#include "ewsjf_device.h"
#include "ewsjf_launch.h"

namespace ewsjf {

// ---------------------------------------------------------------------------
// Key sources.  load4 issues the loads of 4 consecutive requests; keys4
// turns them into composites (0 = no element).
// ---------------------------------------------------------------------------
struct PoolSource {
  const int32_t* len;
  const float* arrival;
  const ewsjf_queue_table* table;
  const ewsjf_theta* theta;  // [n_theta]
  float now;
  CostF cost;

  struct Raw {
    i32x4 l;
    f32x4 a;
  };
  struct Shared {
    uint8_t lut[kLutBytes];
    QParams qp[EWSJF_MAX_QUEUES];
    int L;
  };

  __device__ __forceinline__ void stage(Shared& sh, int t) const {
    stage_policy(table, theta + t, sh.lut, sh.qp);
    if (threadIdx.x == 0) sh.L = table->max_len;
  }

  __device__ __forceinline__ Raw load4(int64_t base, int64_t n) const {
    Raw r;
    if (base + 3 < n) {
      r.l = load_i32x4(len + base);
      r.a = load_f32x4(arrival + base);
    } else {
      r.l = i32x4{0, 0, 0, 0};
      r.a = f32x4{0.f, 0.f, 0.f, 0.f};
      if (base + 0 < n) { r.l.x = len[base + 0]; r.a.x = arrival[base + 0]; }
      if (base + 1 < n) { r.l.y = len[base + 1]; r.a.y = arrival[base + 1]; }
      if (base + 2 < n) { r.l.z = len[base + 2]; r.a.z = arrival[base + 2]; }
    }
    return r;
  }

  __device__ __forceinline__ uint64_t key1(int b, float a, uint32_t id, const Shared& sh) const {
    if (b <= 0) return 0ull;
    const int q = sh.lut[b < sh.L ? b : sh.L];
    const float phi = phi_f32(b, a, now, sh.qp[q], cost);
    return make_comp(ukey_of(phi), id);
  }

  __device__ __forceinline__ void keys4(const Raw& r, int64_t base, const Shared& sh, uint64_t out[4]) const {
    const uint32_t id = (uint32_t)base;
    out[0] = key1(r.l.x, r.a.x, id + 0, sh);
    out[1] = key1(r.l.y, r.a.y, id + 1, sh);
    out[2] = key1(r.l.z, r.a.z, id + 2, sh);
    out[3] = key1(r.l.w, r.a.w, id + 3, sh);
  }
};

struct ScoreSource {
  const float* score;  // [n_theta][n]
  int64_t n;

  struct Raw {
    f32x4 s;
  };
  struct Shared {
    int t;
  };

  __device__ __forceinline__ void stage(Shared& sh, int t) const {
    if (threadIdx.x == 0) sh.t = t;
  }

  __device__ __forceinline__ Raw load4(int64_t base, int64_t nn) const {
    Raw r;
    if (vec_ && base + 3 < nn) {
      r.s = load_f32x4(row_ + base);
    } else if (base + 3 < nn) {
      r.s = f32x4{row_[base + 0], row_[base + 1], row_[base + 2], row_[base + 3]};
    } else {
      const float nan = __builtin_nanf("");
      r.s = f32x4{nan, nan, nan, nan};
      if (base + 0 < nn) r.s.x = row_[base + 0];
      if (base + 1 < nn) r.s.y = row_[base + 1];
      if (base + 2 < nn) r.s.z = row_[base + 2];
    }
    return r;
  }

  __device__ __forceinline__ static uint64_t key1(float s, uint32_t id) {
    return (s != s) ? 0ull : make_comp(ukey_of(s), id);
  }

  __device__ __forceinline__ void keys4(const Raw& r, int64_t base, const Shared&, uint64_t out[4]) const {
    const uint32_t id = (uint32_t)base;
    out[0] = key1(r.s.x, id + 0);
    out[1] = key1(r.s.y, id + 1);
    out[2] = key1(r.s.z, id + 2);
    out[3] = key1(r.s.w, id + 3);
  }

  const float* row_ = nullptr;
  bool vec_ = false;  // the row is 16-byte aligned
  __device__ __forceinline__ ScoreSource for_theta(int t) const {
    ScoreSource s = *this;
    s.row_ = score + (int64_t)t * n;
    s.vec_ = (reinterpret_cast<uintptr_t>(s.row_) & 15) == 0;
    return s;
  }
};

template <class Src>
__device__ __forceinline__ Src bind_theta(const Src& s, int) {
  return s;
}
template <>
__device__ __forceinline__ ScoreSource bind_theta<ScoreSource>(const ScoreSource& s, int t) {
  return s.for_theta(t);
}

// ---------------------------------------------------------------------------
// Per-workgroup candidate list.
// ---------------------------------------------------------------------------
struct ListShared {
  uint64_t list[kListCap];
  uint64_t red[kWavesPerBlock];
  uint32_t bar[kWavesPerBlock];
  int cnt;
  int ovf;
};

// Chunk c of workgroup w at local index lc is c = w + G * lc.  Wave v of the
// block takes local indices lc = v + kWavesPerBlock * (j + kChunksPerPass * pass).
template <class Src>
__device__ __forceinline__ void load_pass(const Src& src, int64_t n, int64_t nchunks, int G, int pass,
                                          typename Src::Raw raw[kChunksPerPass], int64_t base[kChunksPerPass]) {
  const int lane = threadIdx.x & (kWave - 1), wv = threadIdx.x / kWave;
#pragma unroll
  for (int j = 0; j < kChunksPerPass; ++j) {
    const int64_t lc = (int64_t)wv + kWavesPerBlock * ((int64_t)j + (int64_t)kChunksPerPass * pass);
    const int64_t c = (int64_t)blockIdx.x + (int64_t)G * lc;
    base[j] = c < nchunks ? c * kChunk + (int64_t)lane * 4 : n;  // n = past the end
    raw[j] = src.load4(base[j], n);
  }
}

template <class Src>
__global__ __launch_bounds__(kBlock) void local_candidates(Src src0, int64_t n, int G, int m, int M,
                                                           uint64_t* __restrict__ lists,
                                                           uint32_t* __restrict__ counts,
                                                           uint64_t* __restrict__ bounds) {
  __shared__ typename Src::Shared sh;
  __shared__ ListShared ls;
  const int t = blockIdx.y;
  const Src src = bind_theta(src0, t);
  const int lane = threadIdx.x & (kWave - 1), wv = threadIdx.x / kWave;
  const int64_t nchunks = (n + kChunk - 1) / kChunk;
  const int64_t my_chunks = nchunks > blockIdx.x ? (nchunks - blockIdx.x + G - 1) / G : 0;
  const int passes = (int)((my_chunks + kWavesPerBlock * kChunksPerPass - 1) / (kWavesPerBlock * kChunksPerPass));

  // Issue the first pass's loads before staging the policy so the table
  // fetch overlaps the pool stream.
  typename Src::Raw raw[kChunksPerPass];
  int64_t base[kChunksPerPass];
  if (passes > 0) load_pass(src, n, nchunks, G, 0, raw, base);
  src.stage(sh, t);
  if (threadIdx.x == 0) {
    ls.cnt = 0;
    ls.ovf = 0;
  }
  __syncthreads();

  uint32_t T_bar = 0;  // every element with key >= T_bar (over all passes) is listed
  for (int pass = 0; pass < passes; ++pass) {
    if (pass > 0) load_pass(src, n, nchunks, G, pass, raw, base);
    uint64_t c[kElemsPerLane];
#pragma unroll
    for (int j = 0; j < kChunksPerPass; ++j) src.keys4(raw[j], base[j], sh, c + 4 * j);
    uint32_t lmax = 0;
#pragma unroll
    for (int e = 0; e < kElemsPerLane; ++e) {
      const uint32_t k = (uint32_t)(c[e] >> 32);
      lmax = k > lmax ? k : lmax;
    }
    const uint32_t bar = wave_mth_largest_u32(lmax, m);
    if (lane == 0) ls.bar[wv] = bar;
    __syncthreads();
    uint32_t tw = 0;
#pragma unroll
    for (int i = 0; i < kWavesPerBlock; ++i) tw = ls.bar[i] > tw ? ls.bar[i] : tw;
    T_bar = tw > T_bar ? tw : T_bar;
    // Append every element with key >= T_bar (and every element at all when
    // T_bar == 0, i.e. the share has few distinct keys).
    if (__ballot(lmax >= T_bar && lmax != 0u)) {
#pragma unroll
      for (int e = 0; e < kElemsPerLane; ++e) {
        const bool p = c[e] != 0ull && (uint32_t)(c[e] >> 32) >= T_bar;
        const uint64_t bal = __ballot(p);
        if (bal) {
          int b0 = 0;
          if (lane == 0) b0 = atomicAdd(&ls.cnt, __popcll(bal));
          b0 = __shfl(b0, 0);
          const int pos = b0 + __popcll(bal & lanemask_lt());
          if (p) {
            if (pos < kListCap) ls.list[pos] = c[e];
            else ls.ovf = 1;
          }
        }
      }
    }
    __syncthreads();
    if (passes > 1) {
      // Between passes drop entries below the running bar so the list holds
      // exactly the elements >= T_bar seen so far.
      const int cnt = ls.cnt < kListCap ? ls.cnt : kListCap;
      const uint64_t lowc = (uint64_t)T_bar << 32;
      __syncthreads();
      int keep = 0;
      uint64_t mine[1];
      // compaction through a scan (cnt <= kListCap = kBlock)
      mine[0] = (int)threadIdx.x < cnt ? ls.list[threadIdx.x] : 0ull;
      const int flag = mine[0] >= lowc && mine[0] != 0ull;
      int total = 0;
      const int pos = block_exclusive_scan(flag, reinterpret_cast<int*>(ls.red), &total);
      __syncthreads();
      if (flag) ls.list[pos] = mine[0];
      keep = total;
      if (threadIdx.x == 0) ls.cnt = keep;
      __syncthreads();
    }
  }

  // Sort, cut to M and publish.
  const int cnt_all = ls.cnt;
  const bool ovf = ls.ovf != 0;
  const size_t slot = (size_t)t * G + blockIdx.x;
  if (ovf) {
    if (threadIdx.x == 0) {
      counts[slot] = 0u;
      bounds[slot] = ~0ull;  // nothing guaranteed: the merge re-reads this share
    }
    return;
  }
  const int cnt = cnt_all;
  const int P = pow2_ceil(cnt < 2 ? 2 : cnt);
  for (int i = cnt + (int)threadIdx.x; i < P; i += kBlock) ls.list[i] = 0ull;
  __syncthreads();
  block_bitonic_desc(ls.list, P);
  const uint64_t lowc = (uint64_t)T_bar << 32;
  // entries below lowc (from earlier passes with a lower bar) were removed above
  int out = cnt < M ? cnt : M;
  uint64_t T = lowc;
  if (cnt > M) {
    const uint64_t mth = ls.list[M - 1];
    T = mth > T ? mth : T;
  }
  for (int i = threadIdx.x; i < out; i += kBlock) lists[slot * (size_t)M + i] = ls.list[i];
  if (threadIdx.x == 0) {
    counts[slot] = (uint32_t)out;
    bounds[slot] = T;
  }
}

// ---------------------------------------------------------------------------
// Merge: exact top-B of the union of the lists, with re-reads of shares whose
// lists might be missing members of the top-B.
// ---------------------------------------------------------------------------
struct MergeShared {
  uint64_t X[kMergeCap];
  uint64_t S[kSortMax];
  uint32_t hist[256];
  uint64_t red[kWavesPerBlock];
  int iscan[kWavesPerBlock];
  int cntX;
  int cntS;
};

// Exact top-B of X[0..U) (distinct composites), sorted descending into
// X[0..min(U, B)).  Returns min(U, B).
__device__ inline int topb_inplace(MergeShared& ms, int U, int B) {
  const int tid = threadIdx.x;
  if (U <= kSortMax) {
    const int P = pow2_ceil(U < 2 ? 2 : U);
    for (int i = U + tid; i < P; i += kBlock) ms.X[i] = 0ull;
    __syncthreads();
    block_bitonic_desc(ms.X, P);
    return U < B ? U : B;
  }
  // Narrow a value range [lo, hi] until every element >= its cut fits the
  // sort buffer; `need` elements are still wanted from inside the range and
  // `above` elements lie above it.
  uint64_t mx = 0, mn = ~0ull;
  for (int i = tid; i < U; i += kBlock) {
    const uint64_t x = ms.X[i];
    mx = x > mx ? x : mx;
    mn = x < mn ? x : mn;
  }
  uint64_t hi = block_max_u64(mx, ms.red);
  uint64_t lo = block_min_u64(mn, ms.red);
  int need = B, above = 0;
  uint64_t cut = lo;
  for (;;) {
    const uint64_t diff = hi - lo;
    const int bits = diff == 0 ? 0 : 64 - __clzll((long long)diff);
    const int shift = bits > 8 ? bits - 8 : 0;
    for (int i = tid; i < 256; i += kBlock) ms.hist[i] = 0u;
    __syncthreads();
    for (int i = tid; i < U; i += kBlock) {
      const uint64_t x = ms.X[i];
      if (x >= lo && x <= hi) atomicAdd(&ms.hist[(int)((x - lo) >> shift)], 1u);
    }
    __syncthreads();
    // Find the bin where the running count from the top reaches `need`.
    int cstar = 0, cum_above = 0, cum_at = 0;
    if (tid < kWave) {
      // one wave: 4 bins per lane, suffix sums from the top
      const int b0 = 255 - 4 * tid;  // lane 0 holds bins 255..252
      int v[4], s = 0;
      for (int q = 0; q < 4; ++q) {
        v[q] = (int)ms.hist[b0 - q];
        s += v[q];
      }
      int incl = s;
      for (int off = 1; off < kWave; off <<= 1) {
        const int y = __shfl_up(incl, off);
        if (tid >= off) incl += y;
      }
      int run = incl - s;  // elements in bins above this lane's group
      int found = -1, fa = 0, fat = 0;
      for (int q = 0; q < 4; ++q) {
        if (found < 0 && run + v[q] >= need) {
          found = b0 - q;
          fa = run;
          fat = run + v[q];
        }
        run += v[q];
      }
      const uint64_t bal = __ballot(found >= 0);
      const int first = bal ? __ffsll((long long)bal) - 1 : 0;
      cstar = __shfl(found, first);
      cum_above = __shfl(fa, first);
      cum_at = __shfl(fat, first);
      if (tid == 0) {
        ms.iscan[0] = cstar;
        ms.iscan[1] = cum_above;
        ms.iscan[2] = cum_at;
      }
    }
    __syncthreads();
    cstar = ms.iscan[0];
    cum_above = ms.iscan[1];
    cum_at = ms.iscan[2];
    __syncthreads();
    const uint64_t bin_lo = lo + ((uint64_t)cstar << shift);
    if (above + cum_at <= kSortMax || shift == 0) {
      cut = bin_lo;
      break;
    }
    above += cum_above;
    need -= cum_above;
    lo = bin_lo;
    const uint64_t width = (shift >= 64) ? ~0ull : (((uint64_t)1 << shift) - 1);
    hi = (hi - lo > width) ? lo + width : hi;
  }
  // Gather everything >= cut, sort it, keep the first B.
  if (tid == 0) ms.cntS = 0;
  __syncthreads();
  for (int i = tid; i < U; i += kBlock) {
    const uint64_t x = ms.X[i];
    if (x >= cut) {
      const int p = atomicAdd(&ms.cntS, 1);
      if (p < kSortMax) ms.S[p] = x;
    }
  }
  __syncthreads();
  const int nS = ms.cntS < kSortMax ? ms.cntS : kSortMax;
  const int P = pow2_ceil(nS < 2 ? 2 : nS);
  for (int i = nS + tid; i < P; i += kBlock) ms.S[i] = 0ull;
  __syncthreads();
  block_bitonic_desc(ms.S, P);
  const int keep = nS < B ? nS : B;
  for (int i = tid; i < keep; i += kBlock) ms.X[i] = ms.S[i];
  __syncthreads();
  return keep;
}

template <class Src>
__global__ __launch_bounds__(kBlock) void merge_candidates(Src src0, int64_t n, int G, int M, int B,
                                                           const uint64_t* __restrict__ lists,
                                                           const uint32_t* __restrict__ counts,
                                                           const uint64_t* __restrict__ bounds,
                                                           int32_t* __restrict__ ids, float* __restrict__ top,
                                                           int32_t* __restrict__ n_sel, int32_t* tomb_len) {
  __shared__ MergeShared ms;
  __shared__ typename Src::Shared sh;
  __shared__ uint64_t sT[kMaxGrid];
  __shared__ int sOff[kMaxGrid];
  __shared__ int sCnt[kMaxGrid];
  const int t = blockIdx.x;
  const int tid = threadIdx.x;
  const Src src = bind_theta(src0, t);
  const size_t slot0 = (size_t)t * G;

  // Offsets of the lists (G <= kMaxGrid <= kBlock), then one flat, coalesced
  // copy of every list slot that holds an entry.
  int c = tid < G ? (int)counts[slot0 + tid] : 0;
  int total = 0;
  const int off = block_exclusive_scan(c, ms.iscan, &total);
  if (tid < G) {
    sOff[tid] = off;
    sCnt[tid] = c;
    sT[tid] = bounds[slot0 + tid];
  }
  __syncthreads();
  const uint64_t* lists_t = lists + slot0 * (size_t)M;
  for (int idx = tid; idx < G * M; idx += kBlock) {
    const int w = idx / M, i = idx - w * M;
    if (i < sCnt[w]) ms.X[sOff[w] + i] = lists_t[idx];
  }
  __syncthreads();
  int U = topb_inplace(ms, total, B);
  uint64_t tau = (U >= B) ? ms.X[B - 1] : 0ull;

  // Re-read shares whose lists could miss top-B members.
  bool staged = false;
  for (int w = 0; w < G; ++w) {
    const uint64_t thr = tau > 1ull ? tau : 1ull;
    if (!(sT[w] > thr)) continue;
    if (!staged) {
      src.stage(sh, t);
      __syncthreads();
      staged = true;
    }
    const uint64_t Tw = sT[w];
    const int64_t nchunks = (n + kChunk - 1) / kChunk;
    // All chunks of share w: c = w + G * lc, lc = 0, 1, ...; a chunk per wave,
    // 4 requests per lane.
    for (int64_t lc0 = 0;; lc0 += kWavesPerBlock) {
      const int64_t first_c = (int64_t)w + (int64_t)G * lc0;
      if (first_c >= nchunks) break;
      if (U + kBlock * 4 > kMergeCap) {
        U = topb_inplace(ms, U, B);
        tau = (U >= B) ? ms.X[B - 1] : 0ull;
      }
      if (tid == 0) ms.cntX = U;
      __syncthreads();
      const int lane = tid & (kWave - 1), wv = tid / kWave;
      const int64_t cidx = (int64_t)w + (int64_t)G * (lc0 + wv);
      const int64_t b0 = cidx < nchunks ? cidx * kChunk + (int64_t)lane * 4 : n;
      const typename Src::Raw r = src.load4(b0, n);
      uint64_t k4[4];
      src.keys4(r, b0, sh, k4);
      const uint64_t lowb = tau > 1ull ? tau : 1ull;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        if (b0 + e < n && k4[e] >= lowb && k4[e] < Tw) {
          const int p = atomicAdd(&ms.cntX, 1);
          ms.X[p] = k4[e];
        }
      }
      __syncthreads();
      U = ms.cntX;
      __syncthreads();
    }
  }
  if (staged) {
    U = topb_inplace(ms, U, B);
  }

  // Publish.
  const int sel = U < B ? U : B;
  int32_t* ids_t = ids + (size_t)t * B;
  float* top_t = top + (size_t)t * B;
  for (int r = tid; r < B; r += kBlock) {
    if (r < sel) {
      const uint64_t x = ms.X[r];
      ids_t[r] = (int32_t)comp_id(x);
      top_t[r] = float_of_ukey((uint32_t)(x >> 32));
    } else {
      ids_t[r] = -1;
      top_t[r] = __builtin_nanf("");
    }
  }
  if (tid == 0) n_sel[t] = sel;
  if (tomb_len != nullptr) {
    for (int r = tid; r < sel; r += kBlock) tomb_len[comp_id(ms.X[r])] = 0;
  }
}

// ---------------------------------------------------------------------------
// Host-side launch helpers.
// ---------------------------------------------------------------------------
SelectPlan plan_select(int64_t n, int32_t n_theta, int32_t B) {
  SelectPlan p;
  const int64_t nchunks = (n + kChunk - 1) / kChunk;
  int64_t G = (nchunks + kWavesPerBlock - 1) / kWavesPerBlock;
  if (G < 1) G = 1;
  if (G > kMaxGrid) G = kMaxGrid;
  p.G = (int)G;
  const int per = (int)((B + p.G - 1) / p.G);
  int m = (5 * per + 3) / 4;
  if (m < 4) m = 4;
  if (m > 64) m = 64;
  p.m = m;
  int M = pow2_ceil(8 * per);
  if (M < 16) M = 16;
  const int cap = kMergeCap / p.G;
  if (M > cap) M = cap;
  if (M > kListCap) M = kListCap;
  p.M = M;
  p.n_theta = n_theta;
  p.lists_bytes = (size_t)n_theta * p.G * p.M * sizeof(uint64_t);
  p.counts_bytes = (size_t)n_theta * p.G * sizeof(uint32_t);
  p.bounds_bytes = (size_t)n_theta * p.G * sizeof(uint64_t);
  auto up = [](size_t x) { return (x + 255) & ~(size_t)255; };
  p.ws_bytes = up(p.lists_bytes) + up(p.counts_bytes) + up(p.bounds_bytes);
  return p;
}

static void carve(const SelectPlan& p, void* ws, uint64_t** lists, uint32_t** counts, uint64_t** bounds) {
  auto up = [](size_t x) { return (x + 255) & ~(size_t)255; };
  char* b = static_cast<char*>(ws);
  *lists = reinterpret_cast<uint64_t*>(b);
  *counts = reinterpret_cast<uint32_t*>(b + up(p.lists_bytes));
  *bounds = reinterpret_cast<uint64_t*>(b + up(p.lists_bytes) + up(p.counts_bytes));
}

hipError_t launch_step(const int32_t* len, const float* arrival, int64_t n, float now,
                       const ewsjf_queue_table* table, const ewsjf_theta* theta, int32_t n_theta,
                       const ewsjf_cost& cost, int32_t B, int32_t* tomb_len, int32_t* ids, float* top,
                       int32_t* n_sel, void* ws, hipStream_t stream) {
  const SelectPlan p = plan_select(n, n_theta, B);
  uint64_t* lists;
  uint32_t* counts;
  uint64_t* bounds;
  carve(p, ws, &lists, &counts, &bounds);
  PoolSource src;
  src.len = len;
  src.arrival = arrival;
  src.table = table;
  src.theta = theta;
  src.now = now;
  src.cost = CostF{(float)cost.c0, (float)cost.c1, (float)cost.c2};
  hipLaunchKernelGGL(local_candidates<PoolSource>, dim3(p.G, n_theta), dim3(kBlock), 0, stream, src, n, p.G,
                     p.m, p.M, lists, counts, bounds);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(merge_candidates<PoolSource>, dim3(n_theta), dim3(kBlock), 0, stream, src, n, p.G, p.M,
                     B, lists, counts, bounds, ids, top, n_sel, tomb_len);
  return hipGetLastError();
}

hipError_t launch_select(const float* score, int64_t n, int32_t n_theta, int32_t B, int32_t* ids, float* top,
                         int32_t* n_sel, void* ws, hipStream_t stream) {
  const SelectPlan p = plan_select(n, n_theta, B);
  uint64_t* lists;
  uint32_t* counts;
  uint64_t* bounds;
  carve(p, ws, &lists, &counts, &bounds);
  ScoreSource src;
  src.score = score;
  src.n = n;
  hipLaunchKernelGGL(local_candidates<ScoreSource>, dim3(p.G, n_theta), dim3(kBlock), 0, stream, src, n, p.G,
                     p.m, p.M, lists, counts, bounds);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(merge_candidates<ScoreSource>, dim3(n_theta), dim3(kBlock), 0, stream, src, n, p.G, p.M,
                     B, lists, counts, bounds, ids, top, n_sel, nullptr);
  return hipGetLastError();
}

}  // namespace ewsjf
