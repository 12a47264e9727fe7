// Device-side building blocks shared by the EWSJF kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "ewsjf.h"

namespace ewsjf {

constexpr int kWave = 64;
constexpr int kBlock = 1024;                 // threads per streaming workgroup
constexpr int kWavesPerBlock = kBlock / kWave;
constexpr int kChunk = 256;                  // requests per wave chunk: 64 lanes x 4
constexpr int kChunksPerPass = 4;            // chunks a wave holds in registers at once
constexpr int kElemsPerLane = 4 * kChunksPerPass;
constexpr int kMaxGrid = 256;                // streaming workgroups (one per CU)
constexpr int kListCap = 1024;               // per-workgroup candidate list in LDS
constexpr int kShortList = 512;              // lists ranked by all waves at once (up to 8 entries per lane)
constexpr int kWaveCap = kListCap / (kBlock / kWave);  // one region of the list per wave
constexpr int kOverCap = 128;                // overflow entries kept per workgroup
constexpr int kDenseWave = 32;              // region entries that mark a wave holding a cluster of high keys
constexpr int kStageWaves = 4;                // waves that stage the per-workgroup tables
constexpr int kStageThreads = kStageWaves * kWave;
constexpr int kMergeCap = 9088;              // merge kernel candidate capacity (LDS, >= 2 * kSortMax)
constexpr int kSortMax = 4096;               // largest bitonic sort in LDS
constexpr int kLutBytes = EWSJF_MAX_LEN + 16;

// Native 16-byte vectors for coalesced pool loads and stores.
typedef int32_t i32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ i32x4 load_i32x4(const int32_t* p) { return *reinterpret_cast<const i32x4*>(p); }
__device__ __forceinline__ f32x4 load_f32x4(const float* p) { return *reinterpret_cast<const f32x4*>(p); }

// Buffer-resource loads of one 256-element chunk: the resource covers only the
// chunk's in-range part, so lanes past the end of the array read zeros
// instead of faulting, and every chunk costs exactly one load instruction
// per array (no branches, so the wait counters track each chunk).
constexpr int kBufferWord3 = 0x00020000;  // raw buffer, 32-bit data (gfx9 family)
constexpr int kCachePolicyNT = 2;         // streaming (non-temporal) hint

__device__ __forceinline__ __amdgpu_buffer_rsrc_t chunk_rsrc(const void* chunk_base, int64_t remaining_elems) {
  const int64_t r = remaining_elems < 0 ? 0 : (remaining_elems > kChunk ? kChunk : remaining_elems);
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(chunk_base), (short)0, (int)(r * 4), kBufferWord3);
}

__device__ __forceinline__ i32x4 chunk_load_i32x4(__amdgpu_buffer_rsrc_t rs, int lane) {
  return __builtin_amdgcn_raw_buffer_load_b128(rs, lane * 16, 0, kCachePolicyNT);
}

// A zero held in a vector register that the compiler cannot see through.
// Loads indexed by it stay vector loads, counted in issue order with the
// pool loads, instead of becoming scalar loads, whose waits also cover LDS
// traffic.
__device__ __forceinline__ int opaque_zero() {
  int z;
  asm volatile("v_mov_b32 %0, 0" : "=v"(z));
  return z;
}

// Values the compiler must treat as produced at this point (an empty asm
// that "modifies" them), so no computation on them moves above it.
__device__ __forceinline__ void pin_one(float& x) { asm volatile("" : "+v"(x)); }
__device__ __forceinline__ void pin_one(int& x) { asm volatile("" : "+v"(x)); }
__device__ __forceinline__ void pin_one(double& x) { asm volatile("" : "+v"(x)); }
__device__ __forceinline__ void pin_one(i32x4& x) { asm volatile("" : "+v"(x)); }
template <class... T>
__device__ __forceinline__ void pin(T&... x) {
  (pin_one(x), ...);
}

// Per-queue scoring constants derived from one parameter vector, each already
// multiplied by the queue's density factor q + 1: (q+1) w_base, (q+1) w_urg
// and (q+1) w_fair ln 2 (so the fairness term takes a log2).  16 bytes, so a
// lookup is one LDS read.
struct alignas(16) QParams {
  float wb, wu, wf2, pad;
};

// The weights are affine in the queue's mean length (Section 4.1); they and the
// (q + 1) factor are formed in double and rounded once.
__device__ __forceinline__ QParams make_qparams(const ewsjf_theta& th, double mean, int q) {
  const double f = (double)(q + 1);
  const double wb = ((double)th.a_base * mean + (double)th.b_base) * f;
  const double wu = ((double)th.a_urg * mean + (double)th.b_urg) * f;
  const double wf = ((double)th.a_fair * mean + (double)th.b_fair) * f * 0.69314718055994530942;
  return QParams{(float)wb, (float)wu, (float)wf, 0.0f};
}

// ---------------------------------------------------------------------------
// Order-preserving keys.  A float score maps to a 32-bit unsigned key whose
// unsigned order equals the float order (NaN -> -inf, -0 -> +0).  The 64-bit
// composite (key << 32) | (0xFFFFFFFF - id) orders by (score desc, id asc)
// when compared as larger-is-better.  0 is reserved for "no element".
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t ukey_of(float f) {
  uint32_t u = __float_as_uint(f);
  if (f != f) u = 0xFF800000u;           // NaN -> -inf
  if (u == 0x80000000u) u = 0u;          // -0 -> +0
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float float_of_ukey(uint32_t k) {
  uint32_t u = (k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k;
  return __uint_as_float(u);
}

__device__ __forceinline__ uint64_t make_comp(uint32_t ukey, uint32_t id) {
  return ((uint64_t)ukey << 32) | (uint64_t)(0xFFFFFFFFu - id);
}

__device__ __forceinline__ uint32_t comp_id(uint64_t c) { return 0xFFFFFFFFu - (uint32_t)c; }

// Queue (FIFO) order of the tactical step: arrival ascending, a NaN arrival
// counted as +inf and -0 as +0.  arrival_key is ascending in that order;
// fifo_key is its complement, so the oldest request has the largest key
// (always >= 0x007FFFFF, never the reserved 0).
__device__ __forceinline__ uint32_t arrival_key(float a) {
  uint32_t u = __float_as_uint(a);
  if (a != a) u = 0x7F800000u;     // NaN -> +inf
  if (u == 0x80000000u) u = 0u;    // -0 -> +0
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ uint32_t fifo_key(float a) { return ~arrival_key(a); }

// ---------------------------------------------------------------------------
// Wave and block reductions.
// ---------------------------------------------------------------------------
// Wave reductions from the device library (DPP-based).
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t x) { return __ockl_wfred_max_u32(x); }

__device__ __forceinline__ uint64_t wave_max_u64(uint64_t x) {
  const uint32_t mh = __ockl_wfred_max_u32((uint32_t)(x >> 32));
  const uint32_t ml = __ockl_wfred_max_u32((uint32_t)(x >> 32) == mh ? (uint32_t)x : 0u);
  return ((uint64_t)mh << 32) | ml;
}

__device__ __forceinline__ uint64_t wave_min_u64(uint64_t x) {
  const uint32_t mh = __ockl_wfred_min_u32((uint32_t)(x >> 32));
  const uint32_t ml = __ockl_wfred_min_u32((uint32_t)(x >> 32) == mh ? (uint32_t)x : 0xFFFFFFFFu);
  return ((uint64_t)mh << 32) | ml;
}

__device__ __forceinline__ int wave_sum_i32(int x) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) x += __shfl_xor(x, off);
  return x;
}

__device__ __forceinline__ uint64_t lanemask_lt() {
  const int lane = threadIdx.x & (kWave - 1);
  return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

// Block-wide reductions over kBlock threads using a 16-entry LDS scratch.
__device__ __forceinline__ uint64_t block_max_u64(uint64_t x, uint64_t* scratch) {
  const int lane = threadIdx.x & (kWave - 1), wv = threadIdx.x / kWave;
  x = wave_max_u64(x);
  __syncthreads();
  if (lane == 0) scratch[wv] = x;
  __syncthreads();
  uint64_t r = 0;
  for (int i = 0; i < kWavesPerBlock; ++i) r = scratch[i] > r ? scratch[i] : r;
  __syncthreads();
  return r;
}

__device__ __forceinline__ uint64_t block_min_u64(uint64_t x, uint64_t* scratch) {
  const int lane = threadIdx.x & (kWave - 1), wv = threadIdx.x / kWave;
  x = wave_min_u64(x);
  __syncthreads();
  if (lane == 0) scratch[wv] = x;
  __syncthreads();
  uint64_t r = ~0ull;
  for (int i = 0; i < kWavesPerBlock; ++i) r = scratch[i] < r ? scratch[i] : r;
  __syncthreads();
  return r;
}

// Inclusive wave prefix sum with DPP: shifts by 1, 2, 4, 8 inside each row of
// 16 lanes, then the row totals are carried with the row broadcasts of
// lane 15 (to rows 1, 3) and lane 31 (to rows 2, 3).
__device__ __forceinline__ int wave_incl_scan_add(int v) {
  v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xF, 0xF, false);  // row_shr:1
  v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xF, 0xF, false);  // row_shr:2
  v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xF, 0xF, false);  // row_shr:4
  v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xF, 0xF, false);  // row_shr:8
  v += __builtin_amdgcn_update_dpp(0, v, 0x142, 0xA, 0xF, false);  // row_bcast:15
  v += __builtin_amdgcn_update_dpp(0, v, 0x143, 0xC, 0xF, false);  // row_bcast:31
  return v;
}

// Exclusive prefix sum over kBlock threads; returns this thread's prefix and
// writes the total to *total.  scratch holds >= kWavesPerBlock ints.
// The same over a block of nthreads threads (a multiple of kWave).
__device__ __forceinline__ int block_exclusive_scan_n(int x, int* scratch, int* total, int nthreads) {
  const int lane = threadIdx.x & (kWave - 1), wv = threadIdx.x / kWave;
  const int nw = nthreads / kWave;
  const int incl = wave_incl_scan_add(x);
  if (lane == kWave - 1) scratch[wv] = incl;
  __syncthreads();
  int wave_base = 0, sum = 0;
  for (int i = 0; i < nw; ++i) {
    const int si = scratch[i];
    wave_base += i < wv ? si : 0;
    sum += si;
  }
  __syncthreads();
  *total = sum;
  return wave_base + incl - x;
}

__device__ __forceinline__ int block_exclusive_scan(int x, int* scratch, int* total) {
  const int lane = threadIdx.x & (kWave - 1), wv = threadIdx.x / kWave;
  const int incl = wave_incl_scan_add(x);
  if (lane == kWave - 1) scratch[wv] = incl;
  __syncthreads();
  int wave_base = 0, sum = 0;
#pragma unroll
  for (int i = 0; i < kWavesPerBlock; ++i) {
    const int si = scratch[i];
    wave_base += i < wv ? si : 0;
    sum += si;
  }
  __syncthreads();
  *total = sum;
  return wave_base + incl - x;
}

// ---------------------------------------------------------------------------
// Lane exchange x -> x of lane (lane ^ J) without LDS traffic where the
// hardware allows it: DPP quad permutes for J = 1, 2, a half-row mirror
// followed by a quad reversal for J = 4, a row rotation by 8 for J = 8, a
// bit-mode swizzle within 32 lanes for J = 16, a permute for J = 32.
// ---------------------------------------------------------------------------
template <int J>
__device__ __forceinline__ uint32_t xor_lane_u32(uint32_t x) {
  const int v = (int)x;
  if constexpr (J == 1) {
    return (uint32_t)__builtin_amdgcn_update_dpp(0, v, 0xB1, 0xF, 0xF, false);  // quad_perm [1,0,3,2]
  } else if constexpr (J == 2) {
    return (uint32_t)__builtin_amdgcn_update_dpp(0, v, 0x4E, 0xF, 0xF, false);  // quad_perm [2,3,0,1]
  } else if constexpr (J == 4) {
    const int y = __builtin_amdgcn_update_dpp(0, v, 0x141, 0xF, 0xF, false);    // row_half_mirror
    return (uint32_t)__builtin_amdgcn_update_dpp(0, y, 0x1B, 0xF, 0xF, false);  // quad_perm [3,2,1,0]
  } else if constexpr (J == 8) {
    return (uint32_t)__builtin_amdgcn_update_dpp(0, v, 0x128, 0xF, 0xF, false);  // row_ror:8
  } else {
    // Rows of 16 lanes (J = 16) or halves of the wave (J = 32) trade places
    // in registers: swapping x with a copy of itself leaves the partner's
    // value in the first result on the lanes with bit J set, in the second
    // on the others.
    static_assert(J == 16 || J == 32, "xor distances 1 to 32");
    const int lane = (int)(threadIdx.x & 63u);
    const auto r = J == 16 ? __builtin_amdgcn_permlane16_swap(x, x, true, false)
                           : __builtin_amdgcn_permlane32_swap(x, x, true, false);
    return (lane & J) ? r[0] : r[1];
  }
}

// Bar of a wave over its lane values x (0 = no element): the lanes form
// 2^lg groups of 64 >> lg consecutive lanes; the bar is the smallest group
// maximum over the groups holding an element (0 when no lane holds one).  At
// least one element per such group is >= the bar.  Six butterfly max steps:
// the steps inside a group take the group maximum, then the values are
// negated (so 0 stays 0 and the smallest nonzero maximum becomes the largest)
// and the remaining steps take the maximum across groups.
__device__ __forceinline__ uint32_t wave_group_bar(uint32_t x, int lg) {
  const int s = 6 - lg;  // steps that stay inside a group
  if (s == 0) x = 0u - x;
  x = max(x, xor_lane_u32<1>(x));
  if (s == 1) x = 0u - x;
  x = max(x, xor_lane_u32<2>(x));
  if (s == 2) x = 0u - x;
  x = max(x, xor_lane_u32<4>(x));
  if (s == 3) x = 0u - x;
  x = max(x, xor_lane_u32<8>(x));
  if (s == 4) x = 0u - x;
  x = max(x, xor_lane_u32<16>(x));
  if (s == 5) x = 0u - x;
  x = max(x, xor_lane_u32<32>(x));
  if (s == 6) x = 0u - x;
  return 0u - x;
}

// The k-th largest (k >= 1) of the wave's kElemsPerLane * 64 keys (0 when
// fewer than k keys are nonzero): the largest v with at least k keys >= v,
// found bit by bit from the top with wave-wide counts.
__device__ inline uint32_t wave_kth_largest(const uint32_t* key, int k) {
  uint32_t prefix = 0;
  for (int bit = 31; bit >= 0; --bit) {
    const uint32_t cand = prefix | (1u << bit);
    uint32_t c = 0;
#pragma unroll
    for (int e = 0; e < kElemsPerLane; ++e) c += key[e] >= cand ? 1u : 0u;
    if ((int)__ockl_wfred_add_u32(c) >= k) prefix = cand;
  }
  return prefix;
}

// Number of lanes below this one whose bit is set in the wave mask sm.
__device__ __forceinline__ int lanes_below(uint64_t sm) {
  return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(sm >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)sm, 0u));
}

// xor_lane_u32 for a wave-uniform distance j in {1, 2, 4, 8, 16, 32}.
__device__ __forceinline__ uint32_t xor_lane_u32_dyn(uint32_t x, int j) {
  switch (j) {
    case 1: return xor_lane_u32<1>(x);
    case 2: return xor_lane_u32<2>(x);
    case 4: return xor_lane_u32<4>(x);
    case 8: return xor_lane_u32<8>(x);
    case 16: return xor_lane_u32<16>(x);
    default: return xor_lane_u32<32>(x);
  }
}

template <int J>
__device__ __forceinline__ uint64_t xor_lane_u64(uint64_t x) {
  const uint32_t lo = xor_lane_u32<J>((uint32_t)x);
  const uint32_t hi = xor_lane_u32<J>((uint32_t)(x >> 32));
  return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t xor_lane_u64_dyn(uint64_t x, int j) {
  switch (j) {
    case 1: return xor_lane_u64<1>(x);
    case 2: return xor_lane_u64<2>(x);
    case 4: return xor_lane_u64<4>(x);
    case 8: return xor_lane_u64<8>(x);
    case 16: return xor_lane_u64<16>(x);
    default: return xor_lane_u64<32>(x);
  }
}

__device__ __forceinline__ void cmpx_desc(uint64_t& a, uint64_t& b, bool desc) {
  const uint64_t hi = a > b ? a : b, lo = a > b ? b : a;
  a = desc ? hi : lo;
  b = desc ? lo : hi;
}

// Descending bitonic sort of s[0..P) in LDS, all kBlock threads participating,
// P a power of two with 64 <= P <= 64 * kWavesPerBlock * EPT.  Each wave owns
// EPT consecutive 64-element blocks (one element per lane per block):
// partners closer than 64 are reached by lane exchanges, partners in another
// block of the same wave in registers, and only partners held by another wave
// go through LDS (two barriers per such stage).
template <int EPT>
__device__ void block_sort_desc_t(uint64_t* s, int P) {
  const int lane = threadIdx.x & (kWave - 1), wv = threadIdx.x / kWave;
  const int nblk = P / kWave;
  const bool active = EPT * wv < nblk;
  const int i0 = EPT * wv * kWave + lane;  // index of x[0]
  uint64_t x[EPT];
#pragma unroll
  for (int q = 0; q < EPT; ++q) x[q] = active ? s[i0 + q * kWave] : 0ull;
  for (int k = 2; k <= P; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      if (j >= kWave * EPT) {
        __syncthreads();
        if (active) {
#pragma unroll
          for (int q = 0; q < EPT; ++q) s[i0 + q * kWave] = x[q];
        }
        __syncthreads();
        if (active) {
#pragma unroll
          for (int q = 0; q < EPT; ++q) {
            const int i = i0 + q * kWave;
            const uint64_t y = s[i ^ j];
            const bool keep_max = ((i & j) == 0) == ((i & k) == 0);
            x[q] = keep_max ? (x[q] > y ? x[q] : y) : (x[q] < y ? x[q] : y);
          }
        }
      } else if (j >= kWave) {
        if constexpr (EPT == 2) {
          cmpx_desc(x[0], x[1], (i0 & k) == 0);
        } else if constexpr (EPT == 4) {
          if (j == kWave) {
            cmpx_desc(x[0], x[1], (i0 & k) == 0);
            cmpx_desc(x[2], x[3], ((i0 + 2 * kWave) & k) == 0);
          } else {
            cmpx_desc(x[0], x[2], (i0 & k) == 0);
            cmpx_desc(x[1], x[3], ((i0 + kWave) & k) == 0);
          }
        }
      } else {
        const bool lower = (lane & j) == 0;
#pragma unroll
        for (int q = 0; q < EPT; ++q) {
          const uint64_t y = xor_lane_u64_dyn(x[q], j);
          const bool keep_max = lower == (((i0 + q * kWave) & k) == 0);
          x[q] = keep_max ? (x[q] > y ? x[q] : y) : (x[q] < y ? x[q] : y);
        }
      }
    }
  }
  __syncthreads();
  if (active) {
#pragma unroll
    for (int q = 0; q < EPT; ++q) s[i0 + q * kWave] = x[q];
  }
  __syncthreads();
}

// Descending sort of s[0..P), P a power of two in [1, kSortMax]; entries
// beyond the caller's data must already be 0.
__device__ inline void block_sort_desc(uint64_t* s, int P) {
  if (P < kWave) {
    for (int i = P + threadIdx.x; i < kWave; i += kBlock) s[i] = 0ull;
    __syncthreads();
    P = kWave;
  }
  if (P <= kBlock) block_sort_desc_t<1>(s, P);
  else if (P <= 2 * kBlock) block_sort_desc_t<2>(s, P);
  else block_sort_desc_t<4>(s, P);
}

// ---------------------------------------------------------------------------
// Exact cut by histogram narrowing over LDS data X[0..U) of distinct 64-bit
// keys (0 = empty slot, never counted): returns `cut` such that exactly
// min(need, #nonzero) elements are >= cut when stop_at_most == 0, or such
// that at least `need` and at most `stop_at_most` elements are >= cut
// otherwise.  Each round bins the current value range [lo, hi] into 256
// linear bins and descends into the bin where the running count from the
// top reaches `need`; ranges shrink 256-fold per round.  All kBlock threads
// call it.  hist: 256 LDS words; iscan: >= 3 LDS ints; red: kWavesPerBlock
// LDS u64.
// ---------------------------------------------------------------------------
__device__ inline uint64_t find_cut(const uint64_t* X, int U, int need, int stop_at_most, uint32_t* hist, int* iscan,
                                    uint64_t* red) {
  const int tid = threadIdx.x;
  uint64_t mx = 0, mn = ~0ull;
  for (int i = tid; i < U; i += kBlock) {
    const uint64_t x = X[i];
    if (x != 0ull) {
      mx = x > mx ? x : mx;
      mn = x < mn ? x : mn;
    }
  }
  uint64_t hi = block_max_u64(mx, red);
  uint64_t lo = block_min_u64(mn, red);
  if (hi == 0ull) return ~0ull;  // nothing to select
  int above = 0;
  for (;;) {
    const uint64_t diff = hi - lo;
    const int bits = diff == 0 ? 0 : 64 - __clzll((long long)diff);
    const int shift = bits > 8 ? bits - 8 : 0;
    for (int i = tid; i < 256; i += kBlock) hist[i] = 0u;
    __syncthreads();
    for (int i = tid; i < U; i += kBlock) {
      const uint64_t x = X[i];
      if (x != 0ull && x >= lo && x <= hi) atomicAdd(&hist[(int)((x - lo) >> shift)], 1u);
    }
    __syncthreads();
    if (tid < kWave) {
      const int b0 = 255 - 4 * tid;  // lane 0 holds bins 255..252
      int v[4], s = 0;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        v[q] = (int)hist[b0 - q];
        s += v[q];
      }
      int incl = s;
#pragma unroll
      for (int off = 1; off < kWave; off <<= 1) {
        const int y = __shfl_up(incl, off);
        if (tid >= off) incl += y;
      }
      const int total = __shfl(incl, kWave - 1);
      int run = incl - s;
      int found = -1, fa = 0, fat = 0;
      const int want = need - above < total ? need - above : total;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        if (found < 0 && run + v[q] >= want) {
          found = b0 - q;
          fa = run;
          fat = run + v[q];
        }
        run += v[q];
      }
      const uint64_t bal = __ballot(found >= 0);
      const int first = bal ? __ffsll((long long)bal) - 1 : 0;
      const int f0 = __shfl(found, first), f1 = __shfl(fa, first), f2 = __shfl(fat, first);
      if (tid == 0) {
        iscan[0] = f0;
        iscan[1] = f1;
        iscan[2] = f2;
      }
    }
    __syncthreads();
    const int cstar = iscan[0], cum_above = iscan[1], cum_at = iscan[2];
    __syncthreads();
    const uint64_t bin_lo = lo + ((uint64_t)cstar << shift);
    const bool done = stop_at_most > 0 ? (above + cum_at <= stop_at_most) : (above + cum_at <= need);
    if (done || shift == 0) return bin_lo;
    above += cum_above;
    lo = bin_lo;
    const uint64_t width = (((uint64_t)1) << shift) - 1;
    hi = (hi - lo > width) ? lo + width : hi;
  }
}

// ---------------------------------------------------------------------------
// Descending counting sort of S[0..nS) (distinct nonzero keys, nS <= 4096)
// into O[0..nS): 4096 linear buckets over [min, max], bucket offsets from the
// top, scatter, then each element's rank inside its bucket.  Cost is linear
// in nS plus the squares of the bucket sizes.  cnt: 4096 LDS words.
// ---------------------------------------------------------------------------
__device__ inline void bucket_sort_desc(const uint64_t* S, int nS, uint64_t* T, uint64_t* O, uint32_t* cnt,
                                        int* iscan, uint64_t* red) {
  const int tid = threadIdx.x;
  constexpr int NB = 4096;
  uint64_t mx = 0, mn = ~0ull;
  for (int i = tid; i < nS; i += kBlock) {
    const uint64_t x = S[i];
    mx = x > mx ? x : mx;
    mn = x < mn ? x : mn;
  }
  const uint64_t hi = block_max_u64(mx, red);
  const uint64_t lo = block_min_u64(mn, red);
  const uint64_t diff = hi - lo;
  const int bits = diff == 0 ? 0 : 64 - __clzll((long long)diff);
  const int shift = bits > 12 ? bits - 12 : 0;
  for (int i = tid; i < NB; i += kBlock) cnt[i] = 0u;
  __syncthreads();
  for (int i = tid; i < nS; i += kBlock) atomicAdd(&cnt[(int)((S[i] - lo) >> shift)], 1u);
  __syncthreads();
  // exclusive offsets in descending bucket order: thread t owns buckets
  // NB-1-4t .. NB-4-4t
  {
    uint32_t v[4];
    int sum = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      v[q] = cnt[NB - 1 - 4 * tid - q];
      sum += (int)v[q];
    }
    int tot = 0;
    int run = block_exclusive_scan(sum, iscan, &tot);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      cnt[NB - 1 - 4 * tid - q] = (uint32_t)run;  // bucket start, reused as a cursor
      run += (int)v[q];
    }
  }
  __syncthreads();
  for (int i = tid; i < nS; i += kBlock) {
    const uint64_t x = S[i];
    const int b = (int)((x - lo) >> shift);
    const uint32_t pos = atomicAdd(&cnt[b], 1u);
    T[pos] = x;
  }
  __syncthreads();
  // cnt[b] is now the end of bucket b; its start is the end of bucket b+1.
  for (int i = tid; i < nS; i += kBlock) {
    const uint64_t x = T[i];
    const int b = (int)((x - lo) >> shift);
    const int start = b == NB - 1 ? 0 : (int)cnt[b + 1];
    const int end = (int)cnt[b];
    int rank = 0;
    for (int r = start; r < end; ++r) rank += T[r] > x;
    O[start + rank] = x;
  }
  __syncthreads();
}

__host__ __device__ inline int pow2_ceil(int x) {
  int p = 1;
  while (p < x) p <<= 1;
  return p;
}

// ---------------------------------------------------------------------------
// Scoring (Eq. 1 / Eq. 4) in binary32 for one request of prompt length b >= 1:
//   Phi = (q+1)/(b+1) * (w_base + w_urg * W/C(b) + w_fair * ln(b+1)),
// computed from one reciprocal of (b+1) C(b) and one log2 (below).  With the
// parameter ranges of the evaluation every term is positive, so the binary32
// result is within a few ulps of the exact value.
// ---------------------------------------------------------------------------
struct CostF {
  float c0, c1, c2;
};

// Phi (Eq. 1 / Eq. 4) regrouped as three per-request terms and the folded
// per-queue weights of one parameter vector:
//   Phi = ((q+1) w_b + (q+1) w_f ln2 lg) alpha + (q+1) w_u beta,
//   alpha = 1/(b+1), beta = W / ((b+1) C), lg = log2(b+1).
// Every kernel that forms a request's key uses these two functions, so a
// request gets the same key wherever it is scored (the merge's re-reads
// compare keys with the streaming kernel's).
struct PhiTerms {
  float al, be, lg;
};
// kLinear: the caller knows c2 == 0 and C is one FMA; the value is the same
// (fma(0, b, c1) = c1 exactly).
template <bool kLinear = false>
__device__ __forceinline__ PhiTerms phi_terms(int b, float arrival, float now, const CostF& c) {
  const float fb = (float)b;
  const float bp1 = fb + 1.0f;
  const float W = fmaxf(now - arrival, 0.0f);  // NaN arrival or future arrival -> 0
  const float C = kLinear ? __builtin_fmaf(c.c1, fb, c.c0) : __builtin_fmaf(__builtin_fmaf(c.c2, fb, c.c1), fb, c.c0);
  const float r = __builtin_amdgcn_rcpf(bp1 * C);
  return PhiTerms{C * r, W * r, __builtin_amdgcn_logf(bp1)};
}
__device__ __forceinline__ float phi_of(const QParams& p, const PhiTerms& t) {
  return __builtin_fmaf(__builtin_fmaf(p.wf2, t.lg, p.wb), t.al, p.wu * t.be);
}
__device__ __forceinline__ float phi_f32(int b, float arrival, float now, const QParams& p, const CostF& c) {
  return phi_of(p, phi_terms(b, arrival, now, c));
}

// Order-preserving key of a score computed in registers: NaN -> -inf,
// -0 -> +0, then the sign-magnitude flip.  Never 0 (0 marks "no element").
__device__ __forceinline__ uint32_t ukey_fast(float f) {
  f = fmaxf(f, -__builtin_inff());  // maxNum: a NaN operand yields -inf
  f = f + 0.0f;                     // -0 + 0 = +0
  const uint32_t u = __float_as_uint(f);
  return u ^ ((uint32_t)((int32_t)u >> 31) | 0x80000000u);
}

// The same key for a score known to be +0, positive or +inf: the bits with
// the sign bit set.  When every per-queue weight of the parameter vector is
// positive, every request of length >= 1 has such a score: its three terms
// are >= 0 and finite except beta (+inf for an arrival of -inf), and the
// reciprocal stays a normal number under the cost bounds the library
// enforces, so no product is NaN and no sum is -0.
__device__ __forceinline__ uint32_t ukey_pos(float f) { return __float_as_uint(f) | 0x80000000u; }

// min(max(b, 1), L) in one instruction.
__device__ __forceinline__ int clamp_len(int b, int L) {
  int r;
  asm("v_med3_i32 %0, %1, 1, %2" : "=v"(r) : "v"(b), "s"(L));
  return r;
}

// Stage the routing lut and per-queue constants of one parameter vector into
// LDS.  lut: kLutBytes bytes; qp: EWSJF_MAX_QUEUES entries.
__device__ inline void stage_policy(const ewsjf_queue_table* tab, const ewsjf_theta* theta, uint8_t* lut,
                                    QParams* qp) {
  const int L = tab->max_len;
  const int k = tab->k;
  const uint4* src = reinterpret_cast<const uint4*>(tab->lut);
  uint4* dst = reinterpret_cast<uint4*>(lut);
  const int nvec = (L + 1 + 15) / 16;
  for (int i = threadIdx.x; i < nvec; i += blockDim.x) dst[i] = src[i];
  if (theta != nullptr) {
    for (int q = threadIdx.x; q < k; q += blockDim.x) qp[q] = make_qparams(*theta, tab->mean[q], q);
  }
}

// Queue of length b in [1, L] from the table's compact routing map: the
// queue of length 32 (b / 32) - 1 plus the rises at lengths 32 (b / 32) .. b.
constexpr int kRouteWords = EWSJF_ROUTE_WORDS;
__device__ __forceinline__ int route_queue(const uint64_t* route, int b) {
  const uint64_t w = route[b >> 5];
  return (int)(uint32_t)(w >> 32) + __builtin_popcount((uint32_t)w << (31 - (b & 31)));
}

__device__ __forceinline__ int route_lut(int b, int L, const uint8_t* lut) {
  return b <= 0 ? -1 : (int)lut[b < L ? b : L];
}

}  // namespace ewsjf
