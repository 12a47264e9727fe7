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
//    LDS list, which is ranked and cut to its M largest entries.  The workgroup
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
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <cmath>

#include "ewsjf_device.h"
#include "ewsjf_launch.h"
#include "ewsjf_stamps.h"

namespace ewsjf {

// ---------------------------------------------------------------------------
// Key sources.  stage_load issues the global loads of any per-workgroup
// tables; load4 issues the loads of 4 consecutive requests; stage_store
// (after both) moves the tables into LDS; keys4 turns the 4 requests into
// 32-bit order-preserving score keys (0 = no element).
// ---------------------------------------------------------------------------
struct PoolSource {
  const int32_t* len;
  const float* arrival;
  const ewsjf_queue_table* table;
  const ewsjf_theta* theta;  // [n_theta]
  float now;
  CostF cost;

  static constexpr int kRouteVecs = kRouteWords / 2;                                        // 513
  static constexpr int kRoutePerThread = (kRouteVecs + kStageThreads - 1) / kStageThreads;  // 3

  struct Raw {
    i32x4 l;
    f32x4 a;
  };
  struct Shared {
    // The routing map with each word's base queue scaled to its byte offset in
    // qp (16 q), so a request's weights are found with one add.
    uint64_t routeq[kRouteWords];
    QParams qp[EWSJF_MAX_QUEUES];
    uint8_t qpos[EWSJF_MAX_QUEUES];  // 1: the queue's three weights are all positive (or the queue is unused)
    int L;
  };
  struct Stage {
    i32x4 v[kRoutePerThread];
    double mean;
    i32x4 hdr;    // k, max_len, ...
    float th[6];  // the parameter vector
  };
  // How keys are formed (uniform; key_mode after the staging barrier).
  struct KeyMode {
    bool linear;    // c2 == 0
    bool positive;  // every weight positive: ukey_pos
  };

  // Run by the first kStageThreads threads, before any pool load is issued.
  // Branch-free on purpose: every load is issued unconditionally (the routing
  // map and the mean array are read whole, indices clamped into them).  The
  // table's header and the parameter vector are read with vector loads too
  // (opaque_zero): scalar loads, issued here or after the pool loads, put
  // their wait (which also covers LDS traffic) ahead of a barrier, or
  // queued behind the pool stream.
  __device__ __forceinline__ void stage_load(Stage& st, int t) const {
    const int z = opaque_zero();
    const i32x4* src = reinterpret_cast<const i32x4*>(table->route);
#pragma unroll
    for (int r = 0; r < kRoutePerThread; ++r) {
      const int i = threadIdx.x + r * kStageThreads;
      st.v[r] = src[i < kRouteVecs ? i : i - kStageThreads];  // a past-the-end slot reloads an earlier one
    }
    static_assert(EWSJF_MAX_QUEUES == kStageThreads, "one mean per staging thread");
    st.mean = table->mean[threadIdx.x];
    st.hdr = reinterpret_cast<const i32x4*>(table)[z];
    const float2* tp = reinterpret_cast<const float2*>(theta + t);
#pragma unroll
    for (int j = 0; j < 3; ++j) {
      const float2 w = tp[z + j];
      st.th[2 * j] = w.x;
      st.th[2 * j + 1] = w.y;
    }
  }

  __device__ __forceinline__ void stage_store(Shared& sh, const Stage& st0) const {
    // Pin the staged values here: the compiler would otherwise convert them
    // (binary32 -> binary64) right after their loads, waiting for them ahead
    // of the pool loads.
    Stage st = st0;
    pin(st.th[0], st.th[1], st.th[2], st.th[3], st.th[4], st.th[5], st.hdr, st.mean);
    static_assert(sizeof(QParams) == 16, "a queue's weights are 16 bytes");
    i32x4* dst = reinterpret_cast<i32x4*>(sh.routeq);
#pragma unroll
    for (int r = 0; r < kRoutePerThread; ++r) {
      const int i = threadIdx.x + r * kStageThreads;
      i32x4 v = st.v[r];  // two words: (mask, base) (mask, base)
      v.y <<= 4;
      v.w <<= 4;
      if (r + 1 < kRoutePerThread || i < kRouteVecs) dst[i] = v;
    }
    const ewsjf_theta th{st.th[0], st.th[1], st.th[2], st.th[3], st.th[4], st.th[5]};
    uint8_t pos = 1;
    if ((int)threadIdx.x < st.hdr.x) {
      const QParams q = make_qparams(th, st.mean, threadIdx.x);
      sh.qp[threadIdx.x] = q;
      pos = q.wb > 0.0f && q.wu > 0.0f && q.wf2 > 0.0f;
    }
    sh.qpos[threadIdx.x] = pos;
    if (threadIdx.x == 0) sh.L = st.hdr.y;
  }

  __device__ __forceinline__ KeyMode key_mode(const Shared& sh) const {
    static_assert(EWSJF_MAX_QUEUES == 4 * kWave, "one word of four flags per lane");
    const uint32_t w = reinterpret_cast<const uint32_t*>(sh.qpos)[threadIdx.x & (kWave - 1)];
    return KeyMode{cost.c2 == 0.0f, __ballot(w != 0x01010101u) == 0ull};
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

  // The 4 requests of this lane in chunk c (zeros past the end of the pool).
  __device__ __forceinline__ Raw load_chunk(int64_t c, int64_t n, int lane) const {
    const int64_t first = c * kChunk;
    Raw r;
    r.l = chunk_load_i32x4(chunk_rsrc(len + first, n - first), lane);
    const i32x4 a = chunk_load_i32x4(chunk_rsrc(arrival + first, n - first), lane);
    r.a = __builtin_bit_cast(f32x4, a);
    return r;
  }

  template <bool kLinear, bool kPositive>
  __device__ __forceinline__ uint32_t key1(int b, float a, const Shared& sh, int L) const {
    const int bc = clamp_len(b, L);
    const uint64_t w = sh.routeq[bc >> 5];
    const uint32_t off = (uint32_t)(w >> 32) + ((uint32_t)__builtin_popcount((uint32_t)w << (31 - (bc & 31))) << 4);
    const QParams& p = *reinterpret_cast<const QParams*>(reinterpret_cast<const uint8_t*>(sh.qp) + off);
    const float phi = phi_of(p, phi_terms<kLinear>(b, a, now, cost));
    return b > 0 ? (kPositive ? ukey_pos(phi) : ukey_fast(phi)) : 0u;
  }

  template <bool kLinear, bool kPositive>
  __device__ __forceinline__ void keys4_t(const Raw& r, const Shared& sh, uint32_t out[4]) const {
    const int L = __builtin_amdgcn_readfirstlane(sh.L);
    out[0] = key1<kLinear, kPositive>(r.l.x, r.a.x, sh, L);
    out[1] = key1<kLinear, kPositive>(r.l.y, r.a.y, sh, L);
    out[2] = key1<kLinear, kPositive>(r.l.z, r.a.z, sh, L);
    out[3] = key1<kLinear, kPositive>(r.l.w, r.a.w, sh, L);
  }

  // The key of each of 4 requests (0 for an empty slot); one uniform branch
  // picks the form.
  __device__ __forceinline__ void keys4(const Raw& r, const Shared& sh, const KeyMode& km, uint32_t out[4]) const {
    if (km.linear) {
      if (km.positive) keys4_t<true, true>(r, sh, out);
      else keys4_t<true, false>(r, sh, out);
    } else {
      if (km.positive) keys4_t<false, true>(r, sh, out);
      else keys4_t<false, false>(r, sh, out);
    }
  }

  __device__ __forceinline__ bool skip(int) const { return false; }
  static constexpr bool kClustered = false;
};

// Queue-order keys for the tactical step (Algorithm 1): row t of the grid
// selects the oldest requests of queue plan->q_sel[t] (FIFO order: arrival
// ascending, then id), so the composite (fifo key << 32 | ~id) is largest
// for the oldest request.  Rows t > 0 (the backfill queues) that the plan
// does not need are skipped before they read the pool.
struct FifoSource {
  const int32_t* len;
  const float* arrival;
  const ewsjf_queue_table* table;
  const TacticalPlan* plan;

  static constexpr int kRouteVecs = kRouteWords / 2;
  static constexpr int kRoutePerThread = (kRouteVecs + kStageThreads - 1) / kStageThreads;

  struct Raw {
    i32x4 l;
    f32x4 a;
  };
  struct Shared {
    uint64_t route[kRouteWords];
    int L;
    int qsel;
  };
  struct Stage {
    i32x4 v[kRoutePerThread];
    i32x4 hdr;  // k, max_len, ...
    int qsel;
  };

  // As PoolSource::stage_load: vector loads only, issued before the pool's.
  __device__ __forceinline__ void stage_load(Stage& st, int t) const {
    const int z = opaque_zero();
    const i32x4* src = reinterpret_cast<const i32x4*>(table->route);
#pragma unroll
    for (int r = 0; r < kRoutePerThread; ++r) {
      const int i = threadIdx.x + r * kStageThreads;
      st.v[r] = src[i < kRouteVecs ? i : i - kStageThreads];  // a past-the-end slot reloads an earlier one
    }
    st.hdr = reinterpret_cast<const i32x4*>(table)[z];
    st.qsel = plan->q_sel[t + z];
  }

  __device__ __forceinline__ void stage_store(Shared& sh, const Stage& st0) const {
    Stage st = st0;
    pin(st.hdr, st.qsel);
    i32x4* dst = reinterpret_cast<i32x4*>(sh.route);
#pragma unroll
    for (int r = 0; r < kRoutePerThread; ++r) {
      const int i = threadIdx.x + r * kStageThreads;
      if (r + 1 < kRoutePerThread || i < kRouteVecs) dst[i] = st.v[r];
    }
    if (threadIdx.x == 0) {
      sh.L = st.hdr.y;
      sh.qsel = st.qsel;
    }
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

  __device__ __forceinline__ Raw load_chunk(int64_t c, int64_t n, int lane) const {
    const int64_t first = c * kChunk;
    Raw r;
    r.l = chunk_load_i32x4(chunk_rsrc(len + first, n - first), lane);
    const i32x4 a = chunk_load_i32x4(chunk_rsrc(arrival + first, n - first), lane);
    r.a = __builtin_bit_cast(f32x4, a);
    return r;
  }

  struct KeyMode {};
  __device__ __forceinline__ KeyMode key_mode(const Shared&) const { return {}; }

  __device__ __forceinline__ uint32_t key1(int b, float a, const Shared& sh) const {
    const int bc = min(max(b, 1), sh.L);
    return (b > 0 && route_queue(sh.route, bc) == sh.qsel) ? fifo_key(a) : 0u;
  }

  __device__ __forceinline__ void keys4(const Raw& r, const Shared& sh, const KeyMode&, uint32_t out[4]) const {
    out[0] = key1(r.l.x, r.a.x, sh);
    out[1] = key1(r.l.y, r.a.y, sh);
    out[2] = key1(r.l.z, r.a.z, sh);
    out[3] = key1(r.l.w, r.a.w, sh);
  }

  __device__ __forceinline__ bool skip(int t) const { return t > 0 && plan->take[t] == 0; }
  // The oldest requests of a queue sit together in an arrival-ordered pool:
  // the streaming kernel keeps a spill list for full wave regions and lowers
  // the workgroup bound past a clustered wave (both cost the score sources
  // time and registers, so they are compiled in for this source only).
  static constexpr bool kClustered = true;
};

// The streaming pool with this step's arrivals (the streaming scheduler's
// per-step update fused into the step): a ring of request slots, of which
// the slots (pos + i) mod capacity, i < n_new, take new request i.  The
// streaming kernel substitutes the new requests for the loaded slots of the
// chunks that hold them and writes them to the ring (and their lengths to
// the partition window), so the step sees the pool after the insert and
// later steps find it stored.
struct RingSource : PoolSource {
  int32_t* ring_len;
  float* ring_arrival;
  int64_t capacity, pos;
  int32_t* window;
  int64_t window_cap, wpos;
  const int32_t* new_len;
  const float* new_arrival;
  int64_t n_new;

  __device__ __forceinline__ Raw load_chunk(int64_t c, int64_t n, int lane) const {
    Raw r = PoolSource::load_chunk(c, n, lane);
    const int64_t first = c * kChunk;
    if (first < n) {  // wave-uniform from here on
      int64_t d0 = first - pos;
      if (d0 < 0) d0 += capacity;
      int64_t d1 = pos - first;
      if (d1 < 0) d1 += capacity;
      if (d0 < n_new || d1 < kChunk) {  // the chunk holds new requests
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int64_t slot = first + 4 * lane + e;
          int64_t d = slot - pos;
          if (d < 0) d += capacity;
          if (slot < n && d < n_new) {
            const int32_t b = new_len[d];
            const float a = new_arrival[d];
            r.l[e] = b;
            r.a[e] = a;
            ring_len[slot] = b;
            ring_arrival[slot] = a;
            if (window_cap > 0) {
              int64_t w = wpos + d;
              if (w >= window_cap) w -= window_cap;
              window[w] = b;
            }
          }
        }
      }
    }
    return r;
  }
};

// Trials of scoring-parameter proposals: row t of the grid is proposal t
// with its own pool, the t-th block of `stride` slots of every pool array,
// and every pool takes the same arrivals (bind_theta moves the pointers).
struct TrialSource : RingSource {
  int64_t stride;
};

struct ScoreSource {
  const float* score;  // [n_theta][n]
  int64_t n;

  struct Raw {
    f32x4 s;
  };
  struct Shared {
    int unused;
  };
  struct Stage {};

  __device__ __forceinline__ void stage_load(Stage&, int) const {}
  __device__ __forceinline__ void stage_store(Shared&, const Stage&) const {}

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

  // A chunk beyond the row's end reads zeros, which are marked empty below.
  __device__ __forceinline__ Raw load_chunk(int64_t c, int64_t nn, int lane) const {
    const int64_t first = c * kChunk;
    Raw r;
    const i32x4 v = chunk_load_i32x4(chunk_rsrc(row_ + first, nn - first), lane);
    r.s = __builtin_bit_cast(f32x4, v);
    const int64_t i0 = first + 4 * lane;
    const float nan = __builtin_nanf("");
    if (i0 + 0 >= nn) r.s.x = nan;
    if (i0 + 1 >= nn) r.s.y = nan;
    if (i0 + 2 >= nn) r.s.z = nan;
    if (i0 + 3 >= nn) r.s.w = nan;
    return r;
  }

  // A NaN score marks an element that is not admissible.
  __device__ __forceinline__ static uint32_t key1(float s) { return (s != s) ? 0u : ukey_of(s); }

  struct KeyMode {};
  __device__ __forceinline__ KeyMode key_mode(const Shared&) const { return {}; }

  __device__ __forceinline__ void keys4(const Raw& r, const Shared&, const KeyMode&, uint32_t out[4]) const {
    out[0] = key1(r.s.x);
    out[1] = key1(r.s.y);
    out[2] = key1(r.s.z);
    out[3] = key1(r.s.w);
  }

  __device__ __forceinline__ bool skip(int) const { return false; }
  static constexpr bool kClustered = false;

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
__device__ __forceinline__ TrialSource bind_theta<TrialSource>(const TrialSource& s, int t) {
  TrialSource r = s;
  const int64_t o = (int64_t)t * s.stride;
  r.len += o;
  r.arrival += o;
  r.ring_len += o;
  r.ring_arrival += o;
  return r;
}
template <>
__device__ __forceinline__ ScoreSource bind_theta<ScoreSource>(const ScoreSource& s, int t) {
  return s.for_theta(t);
}

// ---------------------------------------------------------------------------
// Per-workgroup candidate list.
// ---------------------------------------------------------------------------
struct ListShared {
  uint64_t list[kListCap];  // kWavesPerBlock regions of kWaveCap entries
  uint64_t list2[kListCap];
  uint64_t spill[kListCap];  // entries of waves whose region is full (0 = unused)
  uint32_t hist[256];
  uint64_t red[kWavesPerBlock];
  int iscan[kWavesPerBlock];
  int rank[kShortList];  // ranks of a short list, summed over the waves
  uint32_t bar[kWavesPerBlock];
  int wcnt[kWavesPerBlock];
  int wkeep[kWavesPerBlock];
  int ovf;
  int nout;
  int nspill;
  uint32_t lowbar;  // the lowered workgroup bound (0: not lowered)
};
static_assert(kWaveCap == kWave, "the final filter maps one region slot to one lane");

// Chunk c of workgroup w at local index lc is c = w + G * lc.  Wave v of the
// block takes local indices lc = v + kWavesPerBlock * (j + kChunksPerPass * pass).
// Chunks past the end of the pool read as empty (bounded buffer loads), so
// the loads are issued without a branch.
__device__ __forceinline__ int64_t chunk_of(int G, int pass, int j) {
  const int wv = __builtin_amdgcn_readfirstlane((int)(threadIdx.x / kWave));
  const int64_t lc = (int64_t)wv + kWavesPerBlock * ((int64_t)j + (int64_t)kChunksPerPass * pass);
  return (int64_t)blockIdx.x + (int64_t)G * lc;
}

template <class Src>
__device__ __forceinline__ void load_one(const Src& src, int64_t n, int G, int pass, int j, typename Src::Raw& raw) {
  raw = src.load_chunk(chunk_of(G, pass, j), n, threadIdx.x & (kWave - 1));
}

// Keeps the compiler from moving memory operations or arithmetic across this
// point, so the load/score interleaving below stays as written.
__device__ __forceinline__ void sched_fence() { __builtin_amdgcn_sched_barrier(0); }

// Publishes a workgroup's filtered list list2[0..cnt) (every element of the
// share >= lowc) into its M slots, overflow list and bounds.  Called by the
// whole block (cnt is uniform).  kClearRank: leave the rank sums at zero for
// another list in the same kernel.
template <bool kClearRank>
__device__ __forceinline__ void publish_list(ListShared& ls, int cnt, uint64_t lowc, int M, size_t slot,
                                             const CandBufs& cb) {
  const int lane = threadIdx.x & (kWave - 1), wv = threadIdx.x / kWave;
  uint64_t* out_list = cb.lists + slot * (size_t)M;
  uint64_t* over_list = cb.over + slot * (size_t)kOverCap;
  if (cnt > kListCap) {
    for (int i = threadIdx.x; i < M; i += kBlock) out_list[i] = 0ull;
    if (threadIdx.x == 0) {
      cb.counts[slot] = 0u;
      cb.bounds[slot] = ~0ull;
      cb.bounds2[slot] = ~0ull;
      cb.over_cnt[slot] = 0u;
    }
    return;
  }
  if (cnt <= M) {
    for (int i = threadIdx.x; i < M; i += kBlock) out_list[i] = i < cnt ? ls.list2[i] : 0ull;
    if (threadIdx.x == 0) {
      cb.counts[slot] = (uint32_t)cnt;
      cb.bounds[slot] = lowc;
      cb.bounds2[slot] = lowc;
      cb.over_cnt[slot] = 0u;
    }
    return;
  }
  // Keep exactly the M largest: every element >= the M-th largest is listed.
  // Each element's rank is the number of larger entries (composites are
  // distinct, so ranks are 0..cnt-1).  The entries ranked below the M slots
  // go to the overflow list (up to kOverCap of them), which the merge reads
  // before it would re-read the share from the pool.
  const int listed = min(cnt, M + kOverCap);
  auto place = [&](uint64_t x, int rank) {
    if (rank < M) out_list[rank] = x;
    else if (rank < listed) over_list[rank - M] = x;
    if (rank == M - 1) {
      cb.counts[slot] = (uint32_t)M;
      cb.bounds[slot] = x > lowc ? x : lowc;
    }
    if (rank == listed - 1) cb.bounds2[slot] = (cnt <= M + kOverCap || x < lowc) ? lowc : x;
  };
  if (cnt <= 2 * kWave) {
    // The usual length: every wave holds entries lane and 64 + lane and
    // compares them with its own kSmallPer entries (read as broadcasts,
    // entries past the list masked to 0, which is never larger); the counts
    // add up in LDS, and after one barrier the first two waves place the
    // entries.  Straight-line code: no loop and no per-entry branch.
    constexpr int kSmallPer = 2 * kWave / kWavesPerBlock;
    static_assert(kSmallPer * kWavesPerBlock == 2 * kWave && 2 * kWave <= kShortList, "one slice per wave");
    const uint64_t x0 = lane < cnt ? ls.list2[lane] : 0ull;
    const uint64_t x1 = kWave + lane < cnt ? ls.list2[kWave + lane] : 0ull;
    const int j0 = kSmallPer * wv;
    if (j0 < cnt) {  // uniform
      int r0 = 0, r1 = 0;
      if (cnt > kWave) {  // uniform: entries 64.. exist
#pragma unroll
        for (int u = 0; u < kSmallPer; ++u) {
          const uint64_t y0 = ls.list2[j0 + u];  // in the array for every wave (j0 + u < 2 kWave)
          const uint64_t y = j0 + u < cnt ? y0 : 0ull;
          r0 += y > x0;
          r1 += y > x1;
        }
      } else {
#pragma unroll
        for (int u = 0; u < kSmallPer; ++u) {
          const uint64_t y0 = ls.list2[j0 + u];
          r0 += (j0 + u < cnt ? y0 : 0ull) > x0;
        }
      }
      if (lane < cnt && r0 != 0) atomicAdd(&ls.rank[lane], r0);
      if (kWave + lane < cnt && r1 != 0) atomicAdd(&ls.rank[kWave + lane], r1);
    }
    __syncthreads();
    if ((int)threadIdx.x < cnt) {
      place(ls.list2[threadIdx.x], ls.rank[threadIdx.x]);
      if (kClearRank) ls.rank[threadIdx.x] = 0;  // ready for the next list
    }
    if (threadIdx.x == 0) cb.over_cnt[slot] = (uint32_t)(listed - M);
    return;
  }
  if (cnt <= kShortList) {
    // Longer lists: every wave holds all entries (up to 8 per lane),
    // compares them with its own few (entries w, w + 16, ...) and adds its
    // counts into LDS, so no wave runs a long serial chain.
    constexpr int kG = kShortList / kWave;
    const int ng = (cnt + kWave - 1) / kWave;  // entries per lane in use
    uint64_t x[kG];
    int part[kG];
#pragma unroll
    for (int g = 0; g < kG; ++g) {
      x[g] = g < ng && g * kWave + lane < cnt ? ls.list2[g * kWave + lane] : 0ull;
      part[g] = 0;
    }
    // This wave's entries j = wv + 16 i, four reads at a time (an entry past
    // the list reads as 0, which is never larger).
    for (int j0 = wv; j0 < cnt; j0 += 4 * kWavesPerBlock) {
      uint64_t y[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int j = j0 + u * kWavesPerBlock;
        y[u] = j < cnt ? ls.list2[j] : 0ull;
      }
#pragma unroll
      for (int g = 0; g < kG; ++g)
        if (g < ng) {
#pragma unroll
          for (int u = 0; u < 4; ++u) part[g] += y[u] > x[g];
        }
    }
#pragma unroll
    for (int g = 0; g < kG; ++g)
      if (g < ng && g * kWave + lane < cnt && part[g] != 0) atomicAdd(&ls.rank[g * kWave + lane], part[g]);
    __syncthreads();
    if (wv < kG && threadIdx.x < cnt) {
      place(ls.list2[threadIdx.x], ls.rank[threadIdx.x]);
      if (kClearRank) ls.rank[threadIdx.x] = 0;  // ready for the next list
    }
    if (threadIdx.x == 0) cb.over_cnt[slot] = (uint32_t)(listed - M);
    return;
  }
  // Longer lists: tpe consecutive lanes count each element's rank, each over
  // a slice of the list, and sum with lane exchanges.
  int tpe = 1;
  if (cnt > 128)
    while (tpe < kWave && 2 * tpe * cnt <= kBlock) tpe *= 2;
  const int e = threadIdx.x / tpe, part = threadIdx.x & (tpe - 1);
  const int per = (cnt + tpe - 1) / tpe;
  uint64_t x = 0;
  int rank = 0;
  if (e < cnt) {
    x = ls.list2[e];
    const int j0 = part * per, j1 = min(cnt, j0 + per);
#pragma unroll 8
    for (int j = j0; j < j1; ++j) rank += ls.list2[j] > x;
  }
  for (int o = 1; o < tpe; o <<= 1) rank += (int)xor_lane_u32_dyn((uint32_t)rank, o);
  if (e < cnt && part == 0) place(x, rank);
  if (threadIdx.x == 0) cb.over_cnt[slot] = (uint32_t)(listed - M);
}

// Chunks each wave has in flight when it starts scoring (2, 3 or 4).
constexpr int kAhead = 2;
// Stage the table before the first pool load is issued.
constexpr bool kTableFirst = false;
static_assert(kAhead >= 2 && kAhead <= kChunksPerPass, "chunks in flight");

template <class Src>
__global__ __launch_bounds__(kBlock) void local_candidates(Src src0, int64_t n, int G, int lg, int M, CandBufs cb) {
  __shared__ typename Src::Shared sh;
  __shared__ ListShared ls;
  const int t = blockIdx.y;
  const Src src = bind_theta(src0, t);
  if (src.skip(t)) {  // a row with nothing to select: an empty, complete list
    const size_t slot = (size_t)t * G + blockIdx.x;
    for (int i = threadIdx.x; i < M; i += kBlock) cb.lists[slot * (size_t)M + i] = 0ull;
    if (threadIdx.x == 0) {
      cb.counts[slot] = 0u;
      cb.bounds[slot] = 0ull;
      cb.bounds2[slot] = 0ull;
      cb.over_cnt[slot] = 0u;
    }
    return;
  }
  EWSJF_STAMP(kStampLocal, 0);
  const int lane = threadIdx.x & (kWave - 1), wv = threadIdx.x / kWave;
  const int64_t nchunks = (n + kChunk - 1) / kChunk;
  const int64_t my_chunks = nchunks > blockIdx.x ? (nchunks - blockIdx.x + G - 1) / G : 0;
  const int passes = (int)((my_chunks + kWavesPerBlock * kChunksPerPass - 1) / (kWavesPerBlock * kChunksPerPass));

  // A wave stalls at a vector load while the compute unit's memory pipeline
  // is full, so a wave that issued all of its loads before scoring would
  // score only once nearly the whole stream had arrived.  Instead each wave
  // keeps two chunks in flight and scores one chunk per chunk it issues.
  // The tables go first (loaded by the first kStageWaves waves); the
  // barrier before scoring then waits only for them and for the first two
  // chunk loads of every wave.
  const bool stager = wv < kStageWaves;  // wave-uniform
  typename Src::Stage st;
  if (stager) src.stage_load(st, t);
  typename Src::Raw raw[kChunksPerPass];
  auto init_list = [&]() {
    if (threadIdx.x == 0) {
      ls.ovf = 0;
      ls.nout = 0;
      ls.nspill = 0;
      ls.lowbar = 0u;
    }
    if (threadIdx.x < kShortList) ls.rank[threadIdx.x] = 0;
    static_assert(kListCap == kBlock, "one spill entry per thread");
    if constexpr (Src::kClustered) ls.spill[threadIdx.x] = 0ull;
  };
  if constexpr (kTableFirst) {
    // The table lands in LDS before any pool load is issued, and the only
    // barrier before scoring comes first too: a wave stalls at a vector load
    // while the compute unit's memory queue is full, so a barrier behind pool
    // loads waits until most of them have been served.
    if (stager) src.stage_store(sh, st);
    init_list();
    __syncthreads();
    EWSJF_STAMP(kStampLocal, 1);
    load_one(src, n, G, 0, 0, raw[0]);
    load_one(src, n, G, 0, 1, raw[1]);
    if constexpr (kAhead >= 3) load_one(src, n, G, 0, 2, raw[2]);
    if constexpr (kAhead >= 4) load_one(src, n, G, 0, 3, raw[3]);
  } else {
    // The compute unit serves a workgroup's loads roughly in issue order; this
    // barrier (which does not wait for the loads) puts every table load ahead
    // of every pool load.
    __builtin_amdgcn_s_barrier();
    load_one(src, n, G, 0, 0, raw[0]);
    load_one(src, n, G, 0, 1, raw[1]);
    if constexpr (kAhead >= 3) load_one(src, n, G, 0, 2, raw[2]);
    if constexpr (kAhead >= 4) load_one(src, n, G, 0, 3, raw[3]);
    if (stager) src.stage_store(sh, st);
    init_list();
    __syncthreads();
    EWSJF_STAMP(kStampLocal, 1);
  }
  const auto km = src.key_mode(sh);

  // Each wave writes every element whose key is >= its bar into its own
  // region of the list.  The bar (wave_group_bar over the lane maxima of the
  // first three chunks) leaves at least 2^lg elements of the wave at or
  // above it.  The workgroup's completeness bound is the largest bar of any
  // wave and pass; entries below it are dropped at the end.
  static_assert(kChunksPerPass == 4, "the pipeline below is written for 4 chunks per pass");
  uint64_t* const region = ls.list + wv * kWaveCap;
  uint32_t my_bar = 0;  // this wave's largest bar over the passes
  int wcnt = 0;         // entries of this wave's region (wave-uniform)
  bool wovf = false;    // the region overflowed: elements were lost
  uint32_t key[kElemsPerLane];  // the last pass's keys stay live for the bound lowering below
  for (int pass = 0; pass < passes; ++pass) {
    // A wave stalls at a load while the memory pipeline is full, so it
    // scores a chunk that has arrived before it issues the next load; the
    // other waves keep the pipeline full meanwhile.
    // Chunk j >= kAhead is issued once chunk j - kAhead is scored.
    sched_fence();
    src.keys4(raw[0], sh, km, key + 0);
    sched_fence();
    if constexpr (kAhead == 2) load_one(src, n, G, pass, 2, raw[2]);
    if constexpr (kAhead == 3) load_one(src, n, G, pass, 3, raw[3]);
    sched_fence();
    src.keys4(raw[1], sh, km, key + 4);
    sched_fence();
    if constexpr (kAhead == 2) load_one(src, n, G, pass, 3, raw[3]);
    sched_fence();
    src.keys4(raw[2], sh, km, key + 8);
    // The bar comes from the first three chunks, so it is ready while the
    // last chunk is still in flight; every element (the last chunk's too)
    // at or above it is written.
    uint32_t lmax = 0;
#pragma unroll
    for (int e = 0; e < 12; ++e) lmax = key[e] > lmax ? key[e] : lmax;
    const uint32_t bar = wave_group_bar(lmax, lg);
    src.keys4(raw[3], sh, km, key + 12);
    sched_fence();
    // The next pass's first chunks, if there is a next pass (uniform): after
    // the last pass, loads of chunks past the pool would still queue behind
    // the wave's real ones before the list work can wait them out.
    if (pass + 1 < passes) {
      load_one(src, n, G, pass + 1, 0, raw[0]);
      load_one(src, n, G, pass + 1, 1, raw[1]);
      if constexpr (kAhead >= 3) load_one(src, n, G, pass + 1, 2, raw[2]);
      if constexpr (kAhead >= 4) load_one(src, n, G, pass + 1, 3, raw[3]);
    }
    sched_fence();
    my_bar = bar > my_bar ? bar : my_bar;
    // Per element slot: one compare; the wave's mask of qualifying lanes
    // gives each lane its position, and the wave-uniform count advances.
    const int wcnt0 = wcnt;
    auto emit = [&](uint32_t thr) {
#pragma unroll
      for (int e = 0; e < kElemsPerLane; ++e) {
        const bool p = key[e] >= thr;
        const uint64_t sm = __ballot(p);
        if (sm != 0ull) {
          const int pos = wcnt + lanes_below(sm);
          if (p && pos < kWaveCap)
            region[pos] = make_comp(key[e], (uint32_t)(chunk_of(G, pass, e / 4) * kChunk + lane * 4 + (e & 3)));
          wcnt += __popcll(sm);
        }
      }
    };
    const uint32_t thr = my_bar > 1u ? my_bar : 1u;
    emit(thr);
    if (Src::kClustered && wcnt > kWaveCap) {
      // Too many keys at or above the bar for the wave's region (data whose
      // high keys cluster in this wave): the rest goes to the workgroup's
      // spill list if it has room (one reservation per wave; a reservation
      // that does not fit is left as zeros, which mean "no entry").
      const int need = wcnt - kWaveCap;
      int base = 0;
      if (lane == 0) base = atomicAdd(&ls.nspill, need);
      base = __builtin_amdgcn_readfirstlane(base);  // lane 0 (the whole wave is active)
      if (base + need <= kListCap) {
        int c = wcnt0;
#pragma unroll
        for (int e = 0; e < kElemsPerLane; ++e) {
          const bool p = key[e] >= thr;
          const uint64_t sm = __ballot(p);
          const int pos = c + lanes_below(sm);
          if (p && pos >= kWaveCap)
            ls.spill[base + pos - kWaveCap] =
                make_comp(key[e], (uint32_t)(chunk_of(G, pass, e / 4) * kChunk + lane * 4 + (e & 3)));
          c += __popcll(sm);
        }
        wcnt = kWaveCap;
      }
    }
    if (wcnt > kWaveCap) {
      // No spill room either: raise the bar just above the (room)-th largest
      // key, so fewer than `room` keys qualify, and emit again.  Only equal
      // keys beyond the room can still overflow (then the list is marked
      // incomplete and the merge re-reads the share).
      const int room = kWaveCap - wcnt0;
      if (room > 0) {
        const uint32_t kth = wave_kth_largest(key, room);
        if (kth != 0xFFFFFFFFu) {
          my_bar = kth + 1u > my_bar ? kth + 1u : my_bar;
          wcnt = wcnt0;
          emit(my_bar);
        }
      }
    }
    if (wcnt > kWaveCap) {
      wovf = true;
      wcnt = kWaveCap;
    }
    if (passes > 1) {
      // Keep the regions bounded between passes: drop entries below the
      // largest bar published so far (never above the final bound, since
      // every bar only grows).
      if (lane == 0) ls.bar[wv] = my_bar;
      __syncthreads();
      uint32_t tb = 0;
#pragma unroll
      for (int i = 0; i < kWavesPerBlock; ++i) tb = ls.bar[i] > tb ? ls.bar[i] : tb;
      const uint64_t lowc = (uint64_t)tb << 32;
      const uint64_t x = lane < wcnt ? region[lane] : 0ull;
      const bool keep = x >= lowc && x != 0ull;
      const uint64_t km = __ballot(keep);
      if (keep) region[lanes_below(km)] = x;
      wcnt = __popcll(km);
    }
  }
  EWSJF_STAMP(kStampLocal, 2);
  if (lane == 0) {
    ls.bar[wv] = my_bar;
    ls.wcnt[wv] = wcnt;
    if (wovf) ls.ovf = 1;
  }
  __syncthreads();
  EWSJF_STAMP(kStampLocal, 3);

  // Publish into the workgroup's M fixed slots (unused slots hold 0).
  const size_t slot = (size_t)t * G + blockIdx.x;
  uint64_t* out_list = cb.lists + slot * (size_t)M;
  // The overflow flag, the wave bars (lane i reads wave i's) and this wave's
  // region entry are read together: one LDS round trip.
  const int any_ovf = ls.ovf;
  const uint32_t bar_l = ls.bar[lane & (kWavesPerBlock - 1)];
  const uint64_t reg_l = region[lane];  // the wave's region entry (valid for lane < wcnt)
  if (any_ovf != 0) {
    for (int i = threadIdx.x; i < M; i += kBlock) out_list[i] = 0ull;
    if (threadIdx.x == 0) {
      cb.counts[slot] = 0u;
      cb.bounds[slot] = ~0ull;  // nothing guaranteed: the merge re-reads this share
      cb.bounds2[slot] = ~0ull;
      cb.over_cnt[slot] = 0u;
    }
    EWSJF_STAMP_FLUSH(kStampLocal);
    return;
  }
  if constexpr (!Src::kClustered) {
    // The workgroup's bound would be the largest wave bar t1 (lane i < 16
    // reads wave i's).  One wave holding a few high keys in each of its lane
    // groups sets t1 alone, and t1 can then exceed the B-th key of the whole
    // pool, which sends the merge back to the share.  So in a single pass
    // (the keys are still in registers) the wave holding t1 also lists its
    // keys in [t2, t1), t2 the second largest bar, and the bound drops to t2.
    // Each wave keeps its entries at or above the bound; a scan of the kept
    // counts over the waves places them in list2.
    const uint32_t b = lane < kWavesPerBlock ? bar_l : 0u;
    const uint32_t t1 = wave_max_u32(b);
    const int v1 = (int)__builtin_ctzll(__ballot(lane < kWavesPerBlock && b == t1));
    const uint32_t t2 = wave_max_u32(lane != v1 ? b : 0u);
    const bool lower = passes == 1 && t2 != 0u && t2 < t1;  // uniform
    const uint32_t T_bar = lower ? t2 : t1;
    const uint64_t lowc = (uint64_t)T_bar << 32;
    const uint64_t x = lane < wcnt ? reg_l : 0ull;
    const bool keep = x >= lowc && x != 0ull;
    const uint64_t km = __ballot(keep);
    if (lane == 0) ls.wkeep[wv] = __popcll(km);
    // The wave holding t1 hands its keys to the workgroup (key e of lane l
    // at e * kWave + l); after the barrier wave w filters keys e = w, so the
    // extra keys cost every wave a few instructions rather than one wave a
    // long serial run.
    uint32_t* const held = reinterpret_cast<uint32_t*>(ls.spill);
    static_assert(kElemsPerLane == kWavesPerBlock && kElemsPerLane * kWave * 4 <= sizeof(ls.spill),
                  "one handed-over key per wave and lane");
    if (lower && wv == v1) {  // uniform
#pragma unroll
      for (int e = 0; e < kElemsPerLane; ++e) held[e * kWave + lane] = key[e];
    }
    __syncthreads();
    const int kc = lane < kWavesPerBlock ? ls.wkeep[lane] : 0;
    const int incl = wave_incl_scan_add(kc);
    const int nreg = __builtin_amdgcn_readlane(incl, kWavesPerBlock - 1);
    const int off = __builtin_amdgcn_readlane(incl - kc, wv);
    if (keep) ls.list2[off + lanes_below(km)] = x;  // nreg <= kListCap: at most kWave per wave
    if (lower) {  // uniform
      // Keys of wave v1 in [t2, t1) go after the regions' entries, in any
      // order (the list is ranked by value when published).
      const uint32_t k = held[wv * kWave + lane];
      const bool p = k >= t2 && k < t1;
      const uint64_t sm = __ballot(p);
      if (sm != 0ull) {
        int base = 0;
        if (lane == 0) base = atomicAdd(&ls.nout, __popcll(sm));
        base = __builtin_amdgcn_readfirstlane(base);  // lane 0 (the whole wave is active)
        const int at = nreg + base + lanes_below(sm);
        // the chunk that element e = wv of wave v1 came from (single pass)
        const int64_t c = (int64_t)blockIdx.x + (int64_t)G * (v1 + kWavesPerBlock * (wv / 4));
        if (p && at < kListCap) ls.list2[at] = make_comp(k, (uint32_t)(c * kChunk + lane * 4 + (wv & 3)));
      }
    }
    __syncthreads();
    // more than kListCap entries only with many extra keys: publish_list
    // then marks the list incomplete
    const int total = nreg + (lower ? ls.nout : 0);
    EWSJF_STAMP(kStampLocal, 4);
    EWSJF_STAMP_VALUE(kStampLocal, 6, total);
    publish_list<false>(ls, total, lowc, M, slot, cb);
    EWSJF_STAMP(kStampLocal, 5);
    EWSJF_STAMP_FLUSH(kStampLocal);
    return;
  }
  // The workgroup's bound: the largest wave bar t1.  When the wave holding
  // t1 is dense (a cluster of high keys, such as old requests in
  // neighbouring slots), it also lists its keys in [t2, t1), t2 the second
  // largest bar, so the bound drops to t2 and no longer sits far above the
  // rest of the share.  (Single pass only: the keys are still in registers.)
  uint32_t t1 = 0, t2 = 0;
  int v1 = 0;
#pragma unroll
  for (int i = 0; i < kWavesPerBlock; ++i) {
    const uint32_t b = ls.bar[i];
    if (b > t1) {
      t2 = t1;
      t1 = b;
      v1 = i;
    } else if (b > t2) {
      t2 = b;
    }
  }
  const uint32_t lo2 = t2 > 1u ? t2 : 1u;
  uint32_t T_bar = t1;
  if (Src::kClustered && passes == 1 && lo2 < t1 && ls.wcnt[v1] >= kDenseWave) {  // uniform
    if (wv == v1) {
      int need = 0;
#pragma unroll
      for (int e = 0; e < kElemsPerLane; ++e) need += __popcll(__ballot(key[e] >= lo2 && key[e] < t1));
      int base = 0;
      if (lane == 0) base = atomicAdd(&ls.nspill, need);
      base = __builtin_amdgcn_readfirstlane(base);  // lane 0 (the whole wave is active)
      if (base + need <= kListCap) {
        int c = base;
#pragma unroll
        for (int e = 0; e < kElemsPerLane; ++e) {
          const bool p = key[e] >= lo2 && key[e] < t1;
          const uint64_t sm = __ballot(p);
          if (p)
            ls.spill[c + lanes_below(sm)] =
                make_comp(key[e], (uint32_t)(chunk_of(G, 0, e / 4) * kChunk + lane * 4 + (e & 3)));
          c += __popcll(sm);
        }
        if (lane == 0) ls.lowbar = lo2;
      }
    }
    __syncthreads();
    if (ls.lowbar != 0u) T_bar = ls.lowbar;
  }
  const uint64_t lowc = (uint64_t)T_bar << 32;
  // Entries >= lowc (regions and spill) are exactly the share's elements >=
  // lowc.  More than kListCap of them: the list cannot hold the share's
  // candidates, so nothing is guaranteed (the merge re-reads the share).
  auto keep_into_list2 = [&](uint64_t x) {
    const bool keep = x >= lowc && x != 0ull;
    const uint64_t bal = __ballot(keep);
    if (bal) {
      int b0 = 0;
      if (lane == 0) b0 = atomicAdd(&ls.nout, __popcll(bal));
      b0 = __shfl(b0, 0);
      const int at = b0 + __popcll(bal & lanemask_lt());
      if (keep && at < kListCap) ls.list2[at] = x;
    }
  };
  keep_into_list2(lane < ls.wcnt[wv] ? ls.list[threadIdx.x] : 0ull);
  if (Src::kClustered && ls.nspill != 0) keep_into_list2(ls.spill[threadIdx.x]);  // uniform
  __syncthreads();
  EWSJF_STAMP(kStampLocal, 4);
  EWSJF_STAMP_VALUE(kStampLocal, 6, ls.nout);
  publish_list<false>(ls, ls.nout, lowc, M, slot, cb);
  EWSJF_STAMP(kStampLocal, 5);
  EWSJF_STAMP_FLUSH(kStampLocal);
}


// ---------------------------------------------------------------------------
// Many parameter vectors over one pool (ewsjf_step with n_theta > 1).  Each
// workgroup reads its share of the pool once (one pass: at most 64 chunks)
// and lists candidates for kThetaPerBlock vectors in turn.  Routing, the
// log, the reciprocal and the wait are the same for every vector, so they
// are computed once per request as three terms,
//   alpha = 1 / (b+1),  beta = W / ((b+1) C),  lg = log2(b+1),
// and a vector's score is Phi = ((q+1) w_b + (q+1) w_f ln2 lg) alpha +
// (q+1) w_u beta (Eq. 1 / Eq. 4 regrouped), three operations with the
// folded per-queue weights.  The list work per vector is as in
// local_candidates; the counters it uses alternate between two copies, so
// one vector's list can be published while the next vector's keys are
// formed, without a workgroup barrier in between.
// ---------------------------------------------------------------------------
constexpr int kThetaPerBlock = 16;

__global__ __launch_bounds__(kBlock) void local_candidates_multi(PoolSource src, int64_t n, int n_theta, int G,
                                                                 int lg, int M, CandBufs cb) {
  __shared__ uint64_t route[kRouteWords];
  __shared__ QParams qp[kThetaPerBlock][EWSJF_MAX_QUEUES];
  __shared__ ListShared ls;
  __shared__ int s_ovf[2], s_nout[2];
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wv = tid / kWave;
  const int t0 = blockIdx.y * kThetaPerBlock;
  const int nt = n_theta - t0 < kThetaPerBlock ? n_theta - t0 : kThetaPerBlock;

  // This wave's four chunks first (the longest wait), then the table and the
  // block's parameter vectors into LDS.
  PoolSource::Raw raw[kChunksPerPass];
#pragma unroll
  for (int j = 0; j < kChunksPerPass; ++j) raw[j] = src.load_chunk(chunk_of(G, 0, j), n, lane);
  {
    const i32x4* lsrc = reinterpret_cast<const i32x4*>(src.table->route);
    i32x4* ldst = reinterpret_cast<i32x4*>(route);
    for (int i = tid; i < kRouteWords / 2; i += kBlock) ldst[i] = lsrc[i];
    const int k = src.table->k;
    for (int i = tid; i < nt * EWSJF_MAX_QUEUES; i += kBlock) {
      const int tt = i / EWSJF_MAX_QUEUES, q = i % EWSJF_MAX_QUEUES;
      if (q < k) qp[tt][q] = make_qparams(src.theta[t0 + tt], src.table->mean[q], q);
    }
  }
  const int L = src.table->max_len;
  if (tid < 2) {
    s_ovf[tid] = 0;
    s_nout[tid] = 0;
  }
  if (tid < kShortList) ls.rank[tid] = 0;
  __syncthreads();

  // Per request: queue (-1 for an empty slot) and the three terms.
  int qv[kElemsPerLane];
  PhiTerms tm[kElemsPerLane];
#pragma unroll
  for (int e = 0; e < kElemsPerLane; ++e) {
    const int b = raw[e / 4].l[e & 3];
    qv[e] = b > 0 ? route_queue(route, min(b, L)) : -1;
    tm[e] = phi_terms(b, raw[e / 4].a[e & 3], src.now, src.cost);
  }

  uint64_t* const region = ls.list + wv * kWaveCap;
  for (int tt = 0; tt < nt; ++tt) {
    const int t = t0 + tt, pb = tt & 1;
    uint32_t key[kElemsPerLane];
#pragma unroll
    for (int e = 0; e < kElemsPerLane; ++e) {
      const float phi = phi_of(qp[tt][qv[e] < 0 ? 0 : qv[e]], tm[e]);
      key[e] = qv[e] >= 0 ? ukey_fast(phi) : 0u;
    }
    uint32_t lmax = 0;
#pragma unroll
    for (int e = 0; e < 12; ++e) lmax = key[e] > lmax ? key[e] : lmax;
    uint32_t my_bar = wave_group_bar(lmax, lg);
    int wcnt = 0;
    auto emit = [&](uint32_t thr) {
#pragma unroll
      for (int e = 0; e < kElemsPerLane; ++e) {
        const bool p = key[e] >= thr;
        const uint64_t sm = __ballot(p);
        if (sm != 0ull) {
          const int pos = wcnt + lanes_below(sm);
          if (p && pos < kWaveCap)
            region[pos] = make_comp(key[e], (uint32_t)(chunk_of(G, 0, e / 4) * kChunk + lane * 4 + (e & 3)));
          wcnt += __popcll(sm);
        }
      }
    };
    emit(my_bar > 1u ? my_bar : 1u);
    if (wcnt > kWaveCap) {  // as in local_candidates: raise the bar to fit the region
      const uint32_t kth = wave_kth_largest(key, kWaveCap);
      if (kth != 0xFFFFFFFFu) {
        my_bar = kth + 1u > my_bar ? kth + 1u : my_bar;
        wcnt = 0;
        emit(my_bar);
      }
    }
    if (lane == 0) {
      ls.bar[wv] = my_bar;
      ls.wcnt[wv] = wcnt < kWaveCap ? wcnt : kWaveCap;
      if (wcnt > kWaveCap) s_ovf[pb] = 1;
    }
    __syncthreads();
    // Every wave is past the previous vector now: clear its counters.
    if (tid == 0) {
      s_ovf[pb ^ 1] = 0;
      s_nout[pb ^ 1] = 0;
    }
    const size_t slot = (size_t)t * G + blockIdx.x;
    if (s_ovf[pb] != 0) {  // uniform
      for (int i = tid; i < M; i += kBlock) cb.lists[slot * (size_t)M + i] = 0ull;
      if (tid == 0) {
        cb.counts[slot] = 0u;
        cb.bounds[slot] = ~0ull;  // nothing guaranteed: the merge re-reads this share
        cb.bounds2[slot] = ~0ull;
        cb.over_cnt[slot] = 0u;
      }
      continue;
    }
    uint32_t T_bar = 0;
#pragma unroll
    for (int i = 0; i < kWavesPerBlock; ++i) T_bar = ls.bar[i] > T_bar ? ls.bar[i] : T_bar;
    const uint64_t lowc = (uint64_t)T_bar << 32;
    {
      const uint64_t x = lane < ls.wcnt[wv] ? ls.list[tid] : 0ull;
      const bool keep = x >= lowc && x != 0ull;
      const uint64_t bal = __ballot(keep);
      if (bal) {
        int b0 = 0;
        if (lane == 0) b0 = atomicAdd(&s_nout[pb], __popcll(bal));
        b0 = __shfl(b0, 0);
        if (keep) ls.list2[b0 + __popcll(bal & lanemask_lt())] = x;
      }
    }
    __syncthreads();
    publish_list<true>(ls, s_nout[pb], lowc, M, slot, cb);
  }
}

// ---------------------------------------------------------------------------
// Merge: exact top-B of the union of the lists, with re-reads of shares whose
// lists might be missing members of the top-B.
// ---------------------------------------------------------------------------
struct MergeShared {
  uint64_t X[kMergeCap];
  uint64_t S[kSortMax];
  uint32_t cnt[4096];
  uint64_t red[kWavesPerBlock];
  uint64_t wmax[kWavesPerBlock];
  uint64_t wmin[kWavesPerBlock];
  uint64_t wbound[kWavesPerBlock];  // largest completeness bound of each wave's shares
  int iscan[kWavesPerBlock];
  int wtot[kWavesPerBlock];
  int cntX;
  int cntS;
  int cut_bin;
  int cut_cnt;
};

// Exact top-B of the nonzero entries of X[0..U) (distinct composites; when
// U <= B every entry must be nonzero), sorted descending into X[0..min(U, B)).
// Returns the number selected.  When U > B the candidates at or above
// a histogram cut (between B and kSortMax of them) are gathered first; the
// gathered set is then ordered by a counting sort.
__device__ inline int select_top(MergeShared& ms, int U, int B) {
  const int tid = threadIdx.x, lane = tid & (kWave - 1);
  if (U == 0) return 0;
  const uint64_t* src = ms.X;
  int nS = U;
  if (U > B) {
    const uint64_t cut = find_cut(ms.X, U, B, kSortMax, ms.cnt, ms.iscan, ms.red);
    if (tid == 0) ms.cntS = 0;
    __syncthreads();
    for (int i0 = 0; i0 < U; i0 += kBlock) {
      const int i = i0 + tid;
      const uint64_t x = i < U ? ms.X[i] : 0ull;
      const bool p = x >= cut && x != 0ull;
      const uint64_t bal = __ballot(p);
      if (bal) {
        int b0 = 0;
        if (lane == 0) b0 = atomicAdd(&ms.cntS, __popcll(bal));
        b0 = __shfl(b0, 0);
        const int pos = b0 + __popcll(bal & lanemask_lt());
        if (p && pos < kSortMax) ms.S[pos] = x;
      }
    }
    __syncthreads();
    nS = ms.cntS < kSortMax ? ms.cntS : kSortMax;
    src = ms.S;
  }
  // X is free now: its upper part is the scatter buffer, its head the output.
  bucket_sort_desc(src, nS, ms.X + kSortMax, ms.X, ms.cnt, ms.iscan, ms.red);
  return nS < B ? nS : B;
}

// Count of entries greater than v in the descending array a[0..len).
__device__ __forceinline__ int count_greater_desc(const uint64_t* a, int len, uint64_t v) {
  int lo = 0, hi = len;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (a[mid] > v)
      lo = mid + 1;
    else
      hi = mid;
  }
  return lo;
}

// X[0..U0) holds the current top entries sorted descending, S[0..k) new
// entries (distinct from them).  Leaves the top min(B, U0 + k) of both
// sorted in X and returns that count.  A short S is sorted by rank counting
// and merged by binary searches; a long one goes through select_top.
constexpr int kMergeNewRank = 512;
__device__ inline int merge_new(MergeShared& ms, int U0, int k, int B) {
  const int tid = threadIdx.x;
  if (k == 0) return U0;
  if (k > kMergeNewRank || U0 + k > kMergeCap) {
    for (int i = tid; i < k; i += kBlock) ms.X[U0 + i] = ms.S[i];
    __syncthreads();
    return select_top(ms, U0 + k, B);
  }
  for (int e = tid; e < k; e += kBlock) {
    const uint64_t y = ms.S[e];
    int r = 0;
#pragma unroll 8
    for (int j = 0; j < k; ++j) r += ms.S[j] > y;
    ms.X[U0 + r] = y;
  }
  __syncthreads();
  const int total = U0 + k < B ? U0 + k : B;
  const uint64_t* N = ms.X + U0;
  for (int i = tid; i < U0; i += kBlock) {
    const uint64_t x = ms.X[i];
    const int r = i + count_greater_desc(N, k, x);
    if (r < total) ms.S[r] = x;
  }
  for (int j = tid; j < k; j += kBlock) {
    const uint64_t y = N[j];
    const int r = j + count_greater_desc(ms.X, U0, y);
    if (r < total) ms.S[r] = y;
  }
  __syncthreads();
  for (int i = tid; i < total; i += kBlock) ms.X[i] = ms.S[i];
  __syncthreads();
  return total;
}

// LDS of the exact merge.
template <class Src>
struct MergeLds {
  MergeShared ms;
  typename Src::Shared sh;
  uint64_t sT[kMaxGrid];
  uint64_t sT2[kMaxGrid];
};

// The exact top-B of row t (one workgroup): the union of the lists, then the
// recovery of shares whose lists could miss members of the top-B.
template <class Src>
__device__ void merge_exact(const Src& src0, int t, int64_t n, int G, int M, int B, const CandBufs& cb,
                            int32_t* __restrict__ ids, float* __restrict__ top, int32_t* __restrict__ n_sel,
                            int32_t* tomb_len, MergeLds<Src>& lds) {
  EWSJF_STAMP(kStampMergeExact, 0);
  MergeShared& ms = lds.ms;
  typename Src::Shared& sh = lds.sh;
  uint64_t* sT = lds.sT;
  uint64_t* sT2 = lds.sT2;
  const int tid = threadIdx.x;
  const Src src = bind_theta(src0, t);
  const size_t slot0 = (size_t)t * G;
  if (src.skip(t)) {
    for (int r = tid; r < B; r += kBlock) {
      ids[(size_t)t * B + r] = -1;
      top[(size_t)t * B + r] = __builtin_nanf("");
    }
    if (tid == 0) n_sel[t] = 0;
    EWSJF_STAMP_FLUSH(kStampMergeExact);
    return;
  }

  // One round trip: every list slot (G x M, empty slots hold 0) and the
  // completeness bounds, as bounded buffer loads (no branches, so the waits
  // below are exact).
  constexpr int kR = (kMergeCap + kBlock - 1) / kBlock;
  const int lane = tid & (kWave - 1), wv = tid / kWave;
  const int GM = G * M;
  const __amdgpu_buffer_rsrc_t lrs = __builtin_amdgcn_make_buffer_rsrc(
      cb.lists + slot0 * (size_t)M, (short)0, GM * 8, kBufferWord3);
  const uint64_t Tw = tid < G ? cb.bounds[slot0 + tid] : 0ull;
  const uint64_t Tw2 = tid < G ? cb.bounds2[slot0 + tid] : 0ull;
  uint64_t v[kR];
#pragma unroll
  for (int r = 0; r < kR; ++r) {
    const auto w = __builtin_amdgcn_raw_buffer_load_b64(lrs, (tid + r * kBlock) * 8, 0, kCachePolicyNT);
    v[r] = ((uint64_t)w[1] << 32) | w[0];
  }
  if (tid < G) {
    sT[tid] = Tw;
    sT2[tid] = Tw2;
  }
  // Exact range and count of the candidates (registers -> wave -> LDS)
  // while the slots go to LDS and the histogram is cleared.
  uint64_t mx = 0, mn = ~0ull;
  int nz = 0;
#pragma unroll
  for (int r = 0; r < kR; ++r) {
    const int idx = tid + r * kBlock;
    if (idx < GM) ms.X[idx] = v[r];
    mx = v[r] > mx ? v[r] : mx;
    mn = (v[r] != 0ull && v[r] < mn) ? v[r] : mn;
    nz += v[r] != 0ull;
  }
  mx = wave_max_u64(mx);
  mn = wave_min_u64(mn);
  nz = (int)__ockl_wfred_add_u32((uint32_t)nz);
  const uint64_t tb = wave_max_u64(Tw);
  for (int i = tid; i < 4096; i += kBlock) ms.cnt[i] = 0u;
  if (lane == 0) {
    ms.wmax[wv] = mx;
    ms.wmin[wv] = mn;
    ms.iscan[wv] = nz;
    ms.wbound[wv] = tb;
  }
  __syncthreads();
  // Every wave reduces the kWavesPerBlock partials itself, one per lane.
  static_assert(kWavesPerBlock <= kWave, "one partial per lane");
  const bool pl = lane < kWavesPerBlock;
  const int total = (int)__ockl_wfred_add_u32(pl ? (uint32_t)ms.iscan[lane] : 0u);
  // The largest bound of all shares: the recovery below runs only when it
  // lies above the cut (it usually does not).
  const uint64_t max_bound = wave_max_u64(pl ? ms.wbound[lane] : 0ull);
  int U = 0;
  if (total > 0) {
    const uint64_t hi = wave_max_u64(pl ? ms.wmax[lane] : 0ull);
    const uint64_t lo = wave_min_u64(pl ? ms.wmin[lane] : ~0ull);
    const uint64_t diff = hi - lo;
    const int bits = diff == 0 ? 0 : 64 - __clzll((long long)diff);
    const int shift = bits > 12 ? bits - 12 : 0;
#pragma unroll
    for (int r = 0; r < kR; ++r)
      if (v[r] != 0ull) atomicAdd(&ms.cnt[(int)((v[r] - lo) >> shift)], 1u);
    __syncthreads();
    // Bucket offsets from the top: this thread's 4 buckets, a wave scan, then
    // the waves' totals (one per lane) for the offset of this wave.
    const int want = B < total ? B : total;
    uint32_t cb[4];
    int s4 = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      cb[q] = ms.cnt[4095 - 4 * tid - q];
      s4 += (int)cb[q];
    }
    const int incl = wave_incl_scan_add(s4);
    if (lane == kWave - 1) ms.wtot[wv] = incl;
    __syncthreads();
    const int wt = pl ? ms.wtot[lane] : 0;
    const int wincl = wave_incl_scan_add(wt);
    const int before = __builtin_amdgcn_readlane(wincl - wt, wv);  // totals of the waves before this one
    int run = before + incl - s4;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int b = 4095 - 4 * tid - q;
      ms.cnt[b] = (uint32_t)run;  // bucket start, used as a cursor
      if (run < want && run + (int)cb[q] >= want) {
        ms.cut_bin = b;
        ms.cut_cnt = run + (int)cb[q];
      }
      run += (int)cb[q];
    }
    __syncthreads();
    const int cstar = ms.cut_bin, cum_at = ms.cut_cnt;
    if (cum_at <= kSortMax) {
#pragma unroll
      for (int r = 0; r < kR; ++r) {
        if (v[r] != 0ull) {
          const int b = (int)((v[r] - lo) >> shift);
          if (b >= cstar) ms.S[atomicAdd(&ms.cnt[b], 1u)] = v[r];
        }
      }
      __syncthreads();
      // ms.cnt[b] is now the end of bucket b, and the end of bucket b+1 is
      // its start: rank each element inside its bucket.
      for (int i = tid; i < cum_at; i += kBlock) {
        const uint64_t x = ms.S[i];
        const int b = (int)((x - lo) >> shift);
        const int start = b == 4095 ? 0 : (int)ms.cnt[b + 1];
        const int end = (int)ms.cnt[b];
        int rank = 0;
        for (int j = start; j < end; ++j) rank += ms.S[j] > x;
        ms.X[start + rank] = x;
      }
      __syncthreads();
      U = want;
    } else {
      U = select_top(ms, GM, B);  // X holds all G x M slots; empty slots are 0
    }
  }
  uint64_t tau = (U >= B) ? ms.X[B - 1] : 0ull;
  EWSJF_STAMP(kStampMergeExact, 1);

  // Shares whose slots could miss top-B members (rare), largest bound first:
  // each adds its entries in [cut, bound) -- from its overflow list when that
  // reaches down to the cut, else re-read from the pool -- and the cut is
  // raised right away, so later shares often drop out.  X[0..U) is sorted.
  bool staged = false;
  // The loop sits behind a test of the largest bound so that its set-up is
  // not paid when no share is at risk (the usual case).
  if (max_bound > (tau > 1ull ? tau : 1ull)) for (;;) {
    const uint64_t thr = tau > 1ull ? tau : 1ull;
    if (max_bound <= thr) break;  // bounds only fall and the cut only rises
    // The share with the largest bound; every wave finds it from LDS itself,
    // so the decision is uniform without a barrier.
    uint64_t bl = 0;
    int wl = 0x7fffffff;
    for (int w = lane; w < G; w += kWave)
      if (sT[w] > bl) {
        bl = sT[w];
        wl = w;
      }
    const uint64_t best = wave_max_u64(bl);
    if (best <= thr) break;
    const int wbest = __builtin_amdgcn_readlane(wl, (int)__builtin_ctzll(__ballot(bl == best)));
    if (tid == 0) ms.cntS = 0;
    __syncthreads();
    if (sT2[wbest] <= thr) {
      // The shares at risk whose overflow lists reach the cut contribute in
      // one round: the first kOverBatch of them (kOverBatch * kOverCap <=
      // kSortMax, so every reservation fits), the r-th handled by wave r mod
      // 16.  Every wave derives the same share order from LDS itself.
      constexpr int kOverBatch = kSortMax / kOverCap;
      static_assert(kMaxGrid % kWave == 0 && kOverBatch <= 2 * kWavesPerBlock, "two shares per wave at most");
      int mine0 = -1, mine1 = -1, r = 0;
      for (int q = 0; q < kMaxGrid / kWave && r < kOverBatch; ++q) {
        const int wq = q * kWave + lane;
        uint64_t m = __ballot(wq < G && sT[wq] > thr && sT2[wq] <= thr);
        while (m != 0ull && r < kOverBatch) {
          const int w = q * kWave + (int)__builtin_ctzll(m);
          m &= m - 1;
          if ((r & (kWavesPerBlock - 1)) == wv) {
            if (mine0 < 0) mine0 = w;
            else mine1 = w;
            const uint64_t* ov = cb.over + (slot0 + w) * (size_t)kOverCap;
            const int oc = (int)cb.over_cnt[slot0 + w];
            const uint64_t bw = sT[w];
            const uint64_t x0 = lane < oc ? ov[lane] : 0ull;
            const uint64_t x1 = lane + kWave < oc ? ov[lane + kWave] : 0ull;
            const bool p0 = x0 >= thr && x0 < bw, p1 = x1 >= thr && x1 < bw;
            const uint64_t m0 = __ballot(p0), m1 = __ballot(p1);
            int base = 0;
            if (lane == 0) base = atomicAdd(&ms.cntS, (int)(__popcll(m0) + __popcll(m1)));
            base = __builtin_amdgcn_readfirstlane(base);  // lane 0 (the whole wave is active)
            if (p0) ms.S[base + lanes_below(m0)] = x0;
            if (p1) ms.S[base + __popcll(m0) + lanes_below(m1)] = x1;
          }
          ++r;
        }
      }
      __syncthreads();
      U = merge_new(ms, U, ms.cntS, B);
      tau = (U >= B) ? ms.X[B - 1] : 0ull;
      if (lane == 0) {  // done
        if (mine0 >= 0) sT[mine0] = 0ull;
        if (mine1 >= 0) sT[mine1] = 0ull;
      }
      __syncthreads();
      continue;
    } else {
      if (!staged) {
        if (tid < kStageThreads) {
          typename Src::Stage st;
          src.stage_load(st, t);
          src.stage_store(sh, st);
        }
        __syncthreads();
        staged = true;
      }
      const int64_t nchunks = (n + kChunk - 1) / kChunk;
      // All chunks of share wbest: c = wbest + G * lc, lc = 0, 1, ...; a chunk
      // per wave, 4 requests per lane.
      for (int64_t lc0 = 0;; lc0 += kWavesPerBlock) {
        const int64_t first_c = (int64_t)wbest + (int64_t)G * lc0;
        if (first_c >= nchunks) break;
        if (lc0 > 0) {  // at most kBlock * 4 = kSortMax new entries per round
          U = merge_new(ms, U, ms.cntS, B);
          tau = (U >= B) ? ms.X[B - 1] : 0ull;
          if (tid == 0) ms.cntS = 0;
          __syncthreads();
        }
        const int64_t cidx = (int64_t)wbest + (int64_t)G * (lc0 + wv);
        const int64_t b0 = cidx < nchunks ? cidx * kChunk + (int64_t)lane * 4 : n;
        const typename Src::Raw r = src.load4(b0, n);
        uint32_t k4[4];
        src.keys4(r, sh, src.key_mode(sh), k4);
        const uint64_t lowb = tau > 1ull ? tau : 1ull;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          if (k4[e] != 0u && b0 + e < n) {
            const uint64_t x = make_comp(k4[e], (uint32_t)(b0 + e));
            if (x >= lowb && x < best) ms.S[atomicAdd(&ms.cntS, 1)] = x;
          }
        }
        __syncthreads();
      }
      U = merge_new(ms, U, ms.cntS, B);
    }
    tau = (U >= B) ? ms.X[B - 1] : 0ull;
    if (tid == 0) sT[wbest] = 0ull;  // done
    __syncthreads();
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
  EWSJF_STAMP(kStampMergeExact, 2);
  EWSJF_STAMP_FLUSH(kStampMergeExact);
}

template <class Src>
__global__ __launch_bounds__(kBlock) void merge_candidates(Src src0, int64_t n, int G, int M, int B, CandBufs cb,
                                                           int32_t* __restrict__ ids, float* __restrict__ top,
                                                           int32_t* __restrict__ n_sel, int32_t* tomb_len) {
  __shared__ MergeLds<Src> lds;
  merge_exact(src0, (int)blockIdx.x, n, G, M, B, cb, ids, top, n_sel, tomb_len, lds);
}

// ---------------------------------------------------------------------------
// Merge by rank counting (one parameter vector).  The lists hold distinct
// composites; when every share's completeness bound is at most the B-th
// largest listed composite tau, the top-B of the union is the exact top-B,
// and an entry's output position is the number of larger entries.  That
// holds when the largest bound T satisfies T <= 1 (every share listed all of
// its elements) or at least B entries are >= T.  Each workgroup ranks
// kRankPer own slots against all G x M slots, counting with wave ballots,
// and writes the entries of rank < B to their positions; no workgroup waits
// for another.  Only own slots at or above T are ranked (below T an entry
// has at least B entries above it), all in one pass; correctness needs no
// order in the lists (the order only balances the work).  Otherwise (a share could be missing
// members of the top-B) workgroup 0 runs the exact merge with its recovery
// and the others leave.  Every workgroup reaches the same decision from the
// same slots and bounds.
// ---------------------------------------------------------------------------
constexpr int kRankPer = 16;
constexpr int kRankR = (kMergeCap + kBlock - 1) / kBlock;  // most slots per thread

// NR: slots per thread, a compile-time bound >= ceil(G M / kBlock).
template <class Src, int NR>
__global__ __launch_bounds__(kBlock) void merge_rank(Src src, int64_t n, int G, int M, int B, CandBufs cb,
                                                     int32_t* __restrict__ ids, float* __restrict__ top,
                                                     int32_t* __restrict__ n_sel, int32_t* tomb_len) {
  __shared__ MergeLds<Src> lds;
  __shared__ uint64_t s_c[kRankPer];
  // per-wave partials, each reduced by every wave itself (no LDS atomics and
  // no barrier to clear them first): largest bound, nonzero slots, slots >= T
  __shared__ uint64_t s_wT[kWavesPerBlock];
  __shared__ int s_wnz[kWavesPerBlock], s_wge[kWavesPerBlock];
  __shared__ int s_rank[kRankPer];
  EWSJF_STAMP(kStampMergeRank, 0);
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wv = tid / kWave;
  const bool pl = lane < kWavesPerBlock;  // lane i reads wave i's partial
  const int GM = G * M;
  const int p0 = (int)blockIdx.x * kRankPer;

  // One round trip: the slots (slot tid + r kBlock in v[r]; past GM reads 0),
  // the bounds and this workgroup's own slots.
  const __amdgpu_buffer_rsrc_t lrs = __builtin_amdgcn_make_buffer_rsrc(cb.lists, (short)0, GM * 8, kBufferWord3);
  uint64_t v[NR];
#pragma unroll
  for (int r = 0; r < NR; ++r) {
    const auto w = __builtin_amdgcn_raw_buffer_load_b64(lrs, (tid + r * kBlock) * 8, 0, 0);
    v[r] = ((uint64_t)w[1] << 32) | w[0];
  }
  const uint64_t bnd = tid < G ? cb.bounds[tid] : 0ull;
  // Own slots: with M = kRankPer and G a multiple of it, workgroup w takes
  // entry k of list 16 (w / 16) + (w + k) % 16, one entry of each rank from
  // 16 lists (a bijection on each group of 16 lists).  Lists hold their
  // entries by rank, so every workgroup gets a similar number of slots at or
  // above T to count, rather than all of one list's.
  int os = p0 + tid;
  if (M == kRankPer && (G & (kRankPer - 1)) == 0) {
    const int w = (int)blockIdx.x;
    os = ((w & ~(kRankPer - 1)) | ((w + tid) & (kRankPer - 1))) * M + tid;
  }
  const uint64_t own = tid < kRankPer && os < GM ? cb.lists[os] : 0ull;
  if (tid < kRankPer) {
    s_c[tid] = own;
    s_rank[tid] = 0;
  }
  int nz = 0;
#pragma unroll
  for (int r = 0; r < NR; ++r) nz += __popcll(__ballot(v[r] != 0ull));
  const uint64_t wmax = wave_max_u64(bnd);
  if (lane == 0) {
    s_wT[wv] = wmax;
    s_wnz[wv] = nz;
  }
  __syncthreads();
  EWSJF_STAMP(kStampMergeRank, 1);
  const uint64_t T = wave_max_u64(pl ? s_wT[lane] : 0ull);
  int ge = 0;
#pragma unroll
  for (int r = 0; r < NR; ++r) ge += __popcll(__ballot(v[r] >= T));
  if (lane == 0) s_wge[wv] = ge;
  // This wave's count of slots larger than own slot p (wave-uniform: ballots
  // counted on the scalar unit, beside the compares on the vector unit),
  // summed over the waves in LDS.
  uint64_t c[kRankPer];
#pragma unroll
  for (int p = 0; p < kRankPer; ++p) c[p] = s_c[p];
  // When the merge is safe (below), an entry under T has at least B entries
  // above it, so own slots under T are not ranked (and not written); when it
  // is not, no count is used.
  const uint64_t below_T = T != 0ull ? T - 1ull : 0ull;
  {
    // Every own slot at or above T in one pass: lane p adds the count of slot
    // p (few own slots reach T).
    int mine = 0;
#pragma unroll
    for (int p = 0; p < kRankPer; ++p) {
      if (c[p] > below_T) {  // uniform
        int cnt = 0;
#pragma unroll
        for (int r = 0; r < NR; ++r) cnt += __popcll(__ballot(v[r] > c[p]));
        mine = lane == p ? cnt : mine;
      }
    }
    if (lane < kRankPer && mine != 0) atomicAdd(&s_rank[lane], mine);
  }
  __syncthreads();
  EWSJF_STAMP(kStampMergeRank, 2);
  const int n_ge = (int)__ockl_wfred_add_u32(pl ? (uint32_t)s_wge[lane] : 0u);
  const bool safe = T <= 1ull || n_ge >= B;
  if (!safe) {
    EWSJF_STAMP(kStampMergeRank, 7);
    if (blockIdx.x == 0) merge_exact(src, 0, n, G, M, B, cb, ids, top, n_sel, tomb_len, lds);
    EWSJF_STAMP_FLUSH(kStampMergeRank);
    return;
  }
  // own slots at or below T - 1 rank >= B
  const uint64_t out_bar = below_T;
  EWSJF_STAMP(kStampMergeRank, 3);
  const int nnz = (int)__ockl_wfred_add_u32(pl ? (uint32_t)s_wnz[lane] : 0u);
  const int sel = nnz < B ? nnz : B;
  if (tid < kRankPer) {
    const uint64_t x = s_c[tid];
    const int rank = s_rank[tid];
    if (x > out_bar && rank < B) {
      const uint32_t id = comp_id(x);
      ids[rank] = (int32_t)id;
      top[rank] = float_of_ukey((uint32_t)(x >> 32));
      if (tomb_len != nullptr) tomb_len[id] = 0;
    }
  }
  // Positions past the selection: every workgroup takes every gridDim-th.
  for (int r = (int)blockIdx.x + (int)gridDim.x * tid; r < B; r += (int)gridDim.x * kBlock) {
    if (r >= sel) {
      ids[r] = -1;
      top[r] = __builtin_nanf("");
    }
  }
  if (blockIdx.x == 0 && tid == 0) n_sel[0] = sel;
  EWSJF_STAMP(kStampMergeRank, 4);
  EWSJF_STAMP_FLUSH(kStampMergeRank);
}

// Launches merge_rank with the smallest compiled slots-per-thread bound.
template <class Src>
static void launch_merge_rank(const SelectPlan& p, hipStream_t stream, hipEvent_t e0, hipEvent_t e1, const Src& src,
                              int64_t n, int B, const CandBufs& cb, int32_t* ids, float* top, int32_t* n_sel,
                              int32_t* tomb_len) {
  const int nr = (p.G * p.M + kBlock - 1) / kBlock;
  const dim3 grid((p.G * p.M + kRankPer - 1) / kRankPer), block(kBlock);
  auto go = [&](auto kern) {
    if (e0 != nullptr)
      hipExtLaunchKernelGGL(kern, grid, block, 0, stream, e0, e1, 0, src, n, p.G, p.M, B, cb, ids, top, n_sel,
                            tomb_len);
    else
      hipLaunchKernelGGL(kern, grid, block, 0, stream, src, n, p.G, p.M, B, cb, ids, top, n_sel, tomb_len);
  };
  if (nr <= 1) go(merge_rank<Src, 1>);
  else if (nr <= 2) go(merge_rank<Src, 2>);
  else if (nr <= 4) go(merge_rank<Src, 4>);
  else go(merge_rank<Src, kRankR>);
}

// ---------------------------------------------------------------------------
// Host-side launch helpers.
// ---------------------------------------------------------------------------
// For a source whose highest keys fall anywhere in the pool (no cluster in
// one share): the smallest lg in [2, worst] for which bars above the pool's
// B-th key are rare.  A wave's bar (the least of 2^lg lane-group maxima
// over its first three chunks) lies above that key when every group holds
// one of the B; with the B spread at density d = B / n, a group of E / 2^lg
// keys holds one with probability 1 - exp(-d E / 2^lg).  In a single pass
// the workgroup's bound is its second largest bar, so two such waves in one
// workgroup are needed, else one wave anywhere; either must be expected in
// fewer than one step in a thousand.  Data that breaks the assumption only
// sends the merge back to the share (exact, slower).
static int spread_lg(int64_t n, int G, int B, int passes, int64_t chunks_per_wave, int worst) {
  const double d = (double)B / (double)n;
  const double E = (double)kChunk * (double)(chunks_per_wave < 3 ? chunks_per_wave : 3);
  const double waves = (double)G * kWavesPerBlock * passes;
  for (int lg = 2; lg < worst; ++lg) {
    const double g = (double)(1 << lg);
    const double pw = std::pow(-std::expm1(-d * E / g), g);  // one wave's bar above the B-th key
    const double fail = passes == 1 ? (double)G * (kWavesPerBlock * (kWavesPerBlock - 1) / 2) * pw * pw : waves * pw;
    if (fail <= 1e-3) return lg;
  }
  return worst;
}

SelectPlan plan_select(int64_t n, int32_t n_theta, int32_t B, bool packed, int max_grid, bool spread) {
  SelectPlan p;
  const int64_t nchunks = (n + kChunk - 1) / kChunk;
  // Packed: every wave holds all four chunks of its one pass.
  const int64_t per_wg = packed ? (int64_t)kWavesPerBlock * kChunksPerPass : (int64_t)kWavesPerBlock;
  int64_t G = (nchunks + per_wg - 1) / per_wg;
  if (G < 1) G = 1;
  const int gmax = max_grid > 0 ? max_grid : kMaxGrid;
  if (G > gmax) G = gmax;
  p.G = (int)G;
  const int per = (int)((B + p.G - 1) / p.G);
  // Each wave leaves at least 2^lg elements at or above its bar: the largest
  // power of two <= 5/4 of the workgroup's even share of the B, within [4, 64].
  int m = (5 * per + 3) / 4;
  if (m < 4) m = 4;
  if (m > 64) m = 64;
  int lg = 0;
  while ((2 << lg) <= m) ++lg;
  if (spread && !packed && n > 0) {
    const int64_t my_chunks = (nchunks + G - 1) / G;
    const int64_t per_pass = (int64_t)kWavesPerBlock * kChunksPerPass;
    const int passes = (int)((my_chunks + per_pass - 1) / per_pass);
    lg = spread_lg(n, p.G, B, passes, (my_chunks + kWavesPerBlock - 1) / kWavesPerBlock, lg);
  }
  p.lg = lg;
  int M = pow2_ceil(4 * per);
  if (M < 16) M = 16;
  const int cap = kMergeCap / p.G;
  if (M > cap) M = cap;
  if (M > kListCap) M = kListCap;
  p.M = M;
  p.n_theta = n_theta;
  p.lists_bytes = (size_t)n_theta * p.G * p.M * sizeof(uint64_t);
  p.counts_bytes = (size_t)n_theta * p.G * sizeof(uint32_t);
  p.bounds_bytes = (size_t)n_theta * p.G * sizeof(uint64_t);
  p.over_bytes = (size_t)n_theta * p.G * kOverCap * sizeof(uint64_t);
  p.over_cnt_bytes = (size_t)n_theta * p.G * sizeof(uint32_t);
  p.bounds2_bytes = (size_t)n_theta * p.G * sizeof(uint64_t);
  auto up = [](size_t x) { return (x + 255) & ~(size_t)255; };
  p.ws_bytes = up(p.lists_bytes) + up(p.counts_bytes) + up(p.bounds_bytes) + up(p.over_bytes) +
               up(p.over_cnt_bytes) + up(p.bounds2_bytes);
  return p;
}

static CandBufs carve(const SelectPlan& p, void* ws) {
  auto up = [](size_t x) { return (x + 255) & ~(size_t)255; };
  char* b = static_cast<char*>(ws);
  CandBufs c;
  size_t o = 0;
  c.lists = reinterpret_cast<uint64_t*>(b + o);
  o += up(p.lists_bytes);
  c.counts = reinterpret_cast<uint32_t*>(b + o);
  o += up(p.counts_bytes);
  c.bounds = reinterpret_cast<uint64_t*>(b + o);
  o += up(p.bounds_bytes);
  c.over = reinterpret_cast<uint64_t*>(b + o);
  o += up(p.over_bytes);
  c.over_cnt = reinterpret_cast<uint32_t*>(b + o);
  o += up(p.over_cnt_bytes);
  c.bounds2 = reinterpret_cast<uint64_t*>(b + o);
  return c;
}

static bool step_packed(int64_t n, int32_t n_theta) {
  const int64_t nchunks = (n + kChunk - 1) / kChunk;
  return n_theta > 1 && nchunks <= (int64_t)kMaxGrid * kWavesPerBlock * kChunksPerPass;
}

SelectPlan plan_step(int64_t n, int32_t n_theta, int32_t B) {
  return plan_select(n, n_theta, B, step_packed(n, n_theta));
}

// Trials: each pool gets the workgroups that give every wave one full pass
// (four chunks in flight), the shape of the 4M-pool step, rather than one per
// CU and row: a workgroup's table staging and list publication are then paid
// once per 16,384 requests.
SelectPlan plan_trial(int64_t capacity, int32_t n_pools, int32_t B) {
  return plan_select(capacity, n_pools, B, true);
}

hipError_t launch_step(const int32_t* len, const float* arrival, int64_t n, float now,
                       const ewsjf_queue_table* table, const ewsjf_theta* theta, int32_t n_theta,
                       const ewsjf_cost& cost, int32_t B, int32_t* tomb_len, int32_t* ids, float* top,
                       int32_t* n_sel, void* ws, hipStream_t stream, hipEvent_t* marks) {
  const bool packed = step_packed(n, n_theta);
  const SelectPlan p = plan_select(n, n_theta, B, packed, 0, true);
  const CandBufs cb = carve(p, ws);
  PoolSource src;
  src.len = len;
  src.arrival = arrival;
  src.table = table;
  src.theta = theta;
  src.now = now;
  src.cost = CostF{(float)cost.c0, (float)cost.c1, (float)cost.c2};
  const dim3 multi_grid(p.G, (n_theta + kThetaPerBlock - 1) / kThetaPerBlock);
  if (marks == nullptr) {
    if (packed)
      hipLaunchKernelGGL(local_candidates_multi, multi_grid, dim3(kBlock), 0, stream, src, n, n_theta, p.G, p.lg,
                         p.M, cb);
    else
      hipLaunchKernelGGL(local_candidates<PoolSource>, dim3(p.G, n_theta), dim3(kBlock), 0, stream, src, n, p.G,
                         p.lg, p.M, cb);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (n_theta == 1)
      launch_merge_rank(p, stream, nullptr, nullptr, src, n, B, cb, ids, top, n_sel, tomb_len);
    else
      hipLaunchKernelGGL(merge_candidates<PoolSource>, dim3(n_theta), dim3(kBlock), 0, stream, src, n, p.G, p.M,
                         B, cb, ids, top, n_sel, tomb_len);
    return hipGetLastError();
  }
  // The events take the start and end timestamps of each kernel's own
  // dispatch.
  if (packed)
    hipExtLaunchKernelGGL(local_candidates_multi, multi_grid, dim3(kBlock), 0, stream, marks[0], marks[1], 0, src, n,
                          n_theta, p.G, p.lg, p.M, cb);
  else
    hipExtLaunchKernelGGL(local_candidates<PoolSource>, dim3(p.G, n_theta), dim3(kBlock), 0, stream, marks[0],
                          marks[1], 0, src, n, p.G, p.lg, p.M, cb);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (n_theta == 1)
    launch_merge_rank(p, stream, marks[2], marks[3], src, n, B, cb, ids, top, n_sel, tomb_len);
  else
    hipExtLaunchKernelGGL(merge_candidates<PoolSource>, dim3(n_theta), dim3(kBlock), 0, stream, marks[2], marks[3],
                          0, src, n, p.G, p.M, B, cb, ids, top, n_sel, tomb_len);
  return hipGetLastError();
}

hipError_t launch_ring_step(int32_t* ring_len, float* ring_arrival, int64_t capacity, int64_t pos, int32_t* window,
                            int64_t window_cap, int64_t wpos, const int32_t* new_len, const float* new_arrival,
                            int64_t n_new, float now, const ewsjf_queue_table* table, const ewsjf_theta* theta,
                            const ewsjf_cost& cost, int32_t B, int32_t* tomb_len, int32_t* ids, float* top,
                            int32_t* n_sel, void* ws, hipStream_t stream) {
  const SelectPlan p = plan_select(capacity, 1, B, false, 0, true);
  const CandBufs cb = carve(p, ws);
  RingSource src;
  src.len = ring_len;
  src.arrival = ring_arrival;
  src.table = table;
  src.theta = theta;
  src.now = now;
  src.cost = CostF{(float)cost.c0, (float)cost.c1, (float)cost.c2};
  src.ring_len = ring_len;
  src.ring_arrival = ring_arrival;
  src.capacity = capacity;
  src.pos = pos;
  src.window = window;
  src.window_cap = window_cap;
  src.wpos = wpos;
  src.new_len = new_len;
  src.new_arrival = new_arrival;
  src.n_new = n_new;
  hipLaunchKernelGGL(local_candidates<RingSource>, dim3(p.G, 1), dim3(kBlock), 0, stream, src, capacity, p.G, p.lg,
                     p.M, cb);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  launch_merge_rank(p, stream, nullptr, nullptr, src, capacity, B, cb, ids, top, n_sel, tomb_len);
  return hipGetLastError();
}

hipError_t launch_trial_select(int32_t* len, float* arrival, int64_t capacity, int32_t n_pools, int64_t pos,
                               const int32_t* new_len, const float* new_arrival, int64_t n_new, float now,
                               const ewsjf_queue_table* table, const ewsjf_theta* theta, const ewsjf_cost& cost,
                               int32_t B, int32_t* ids, float* top, int32_t* n_sel, void* ws, hipStream_t stream) {
  const SelectPlan p = plan_trial(capacity, n_pools, B);
  const CandBufs cb = carve(p, ws);
  TrialSource src;
  src.len = len;
  src.arrival = arrival;
  src.table = table;
  src.theta = theta;
  src.now = now;
  src.cost = CostF{(float)cost.c0, (float)cost.c1, (float)cost.c2};
  src.ring_len = len;
  src.ring_arrival = arrival;
  src.capacity = capacity;
  src.pos = pos;
  src.window = nullptr;
  src.window_cap = 0;
  src.wpos = 0;
  src.new_len = new_len;
  src.new_arrival = new_arrival;
  src.n_new = n_new;
  src.stride = capacity;
  hipLaunchKernelGGL(local_candidates<TrialSource>, dim3(p.G, n_pools), dim3(kBlock), 0, stream, src, capacity, p.G,
                     p.lg, p.M, cb);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(merge_candidates<TrialSource>, dim3(n_pools), dim3(kBlock), 0, stream, src, capacity, p.G, p.M,
                     B, cb, ids, top, n_sel, nullptr);
  return hipGetLastError();
}

hipError_t launch_fifo_select(const int32_t* len, const float* arrival, int64_t n, const ewsjf_queue_table* table,
                              const TacticalPlan* plan, int32_t B, int32_t* ids, float* top, int32_t* n_sel, void* ws,
                              hipStream_t stream) {
  const SelectPlan p = plan_select(n, kTacticalRows, B);
  const CandBufs cb = carve(p, ws);
  FifoSource src;
  src.len = len;
  src.arrival = arrival;
  src.table = table;
  src.plan = plan;
  hipLaunchKernelGGL(local_candidates<FifoSource>, dim3(p.G, kTacticalRows), dim3(kBlock), 0, stream, src, n, p.G,
                     p.lg, p.M, cb);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(merge_candidates<FifoSource>, dim3(kTacticalRows), dim3(kBlock), 0, stream, src, n, p.G, p.M,
                     B, cb, ids, top, n_sel, nullptr);
  return hipGetLastError();
}

hipError_t launch_select(const float* score, int64_t n, int32_t n_theta, int32_t B, int32_t* ids, float* top,
                         int32_t* n_sel, void* ws, hipStream_t stream) {
  const SelectPlan p = plan_select(n, n_theta, B);
  const CandBufs cb = carve(p, ws);
  ScoreSource src;
  src.score = score;
  src.n = n;
  hipLaunchKernelGGL(local_candidates<ScoreSource>, dim3(p.G, n_theta), dim3(kBlock), 0, stream, src, n, p.G,
                     p.lg, p.M, cb);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (n_theta == 1)
    launch_merge_rank(p, stream, nullptr, nullptr, src, n, B, cb, ids, top, n_sel, nullptr);
  else
    hipLaunchKernelGGL(merge_candidates<ScoreSource>, dim3(n_theta), dim3(kBlock), 0, stream, src, n, p.G, p.M,
                       B, cb, ids, top, n_sel, nullptr);
  return hipGetLastError();
}

}  // namespace ewsjf

#ifdef EWSJF_STAMPS
// Instrumented build only: copy the phase stamps to the host (count <=
// kStampSlots words) or clear them.
extern "C" int ewsjf_debug_stamps(uint64_t* host, size_t count) {
  if (count > (size_t)ewsjf::kStampSlots) count = ewsjf::kStampSlots;
  return (int)hipMemcpyFromSymbol(host, HIP_SYMBOL(ewsjf::g_stamps), count * sizeof(uint64_t), 0,
                                  hipMemcpyDeviceToHost);
}
extern "C" int ewsjf_debug_stamps_clear(void) {
  static uint64_t zeros[ewsjf::kStampSlots];
  return (int)hipMemcpyToSymbol(HIP_SYMBOL(ewsjf::g_stamps), zeros, sizeof(zeros), 0, hipMemcpyHostToDevice);
}
#endif
