// Device-side building blocks shared by the EWSJF kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

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
constexpr int kMergeCap = 10240;             // merge kernel candidate capacity (LDS)
constexpr int kSortMax = 4096;               // largest bitonic sort in LDS
constexpr int kLutBytes = EWSJF_MAX_LEN + 16;

// Native 16-byte vectors for coalesced pool loads and stores.
typedef int32_t i32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ i32x4 load_i32x4(const int32_t* p) { return *reinterpret_cast<const i32x4*>(p); }
__device__ __forceinline__ f32x4 load_f32x4(const float* p) { return *reinterpret_cast<const f32x4*>(p); }

// Per-queue scoring constants derived from one parameter vector:
// w_base, w_urg, w_fair * ln 2 (so the fairness term uses log2), and q + 1.
struct QParams {
  float wb, wu, wf2, qn;
};

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

// ---------------------------------------------------------------------------
// Wave and block reductions.
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t x) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    uint32_t y = __shfl_xor(x, off);
    x = x > y ? x : y;
  }
  return x;
}

__device__ __forceinline__ uint64_t wave_max_u64(uint64_t x) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    uint64_t y = __shfl_xor(x, off);
    x = x > y ? x : y;
  }
  return x;
}

__device__ __forceinline__ uint64_t wave_min_u64(uint64_t x) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    uint64_t y = __shfl_xor(x, off);
    x = x < y ? x : y;
  }
  return x;
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

// The m-th largest of the 64 lane values (distinct values; ties removed
// together), or 0 when fewer than m distinct non-zero values exist.
__device__ __forceinline__ uint32_t wave_mth_largest_u32(uint32_t x, int m) {
  uint32_t t = 0;
  for (int r = 0; r < m; ++r) {
    const uint32_t mx = wave_max_u32(x);
    t = mx;
    if (mx == 0u) break;
    if (x == mx) x = 0u;
  }
  return t;
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

// Exclusive prefix sum over kBlock threads; returns this thread's prefix and
// writes the total to *total.  scratch holds >= kWavesPerBlock ints.
__device__ __forceinline__ int block_exclusive_scan(int x, int* scratch, int* total) {
  const int lane = threadIdx.x & (kWave - 1), wv = threadIdx.x / kWave;
  int incl = x;
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const int y = __shfl_up(incl, off);
    if (lane >= off) incl += y;
  }
  __syncthreads();
  if (lane == kWave - 1) scratch[wv] = incl;
  __syncthreads();
  int wave_base = 0, sum = 0;
  for (int i = 0; i < kWavesPerBlock; ++i) {
    if (i < wv) wave_base += scratch[i];
    sum += scratch[i];
  }
  __syncthreads();
  *total = sum;
  return wave_base + incl - x;
}

// Descending bitonic sort of s[0..P) in LDS (P a power of two <= kSortMax),
// all kBlock threads participating.
__device__ inline void block_bitonic_desc(uint64_t* s, int P) {
  for (int k = 2; k <= P; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      for (int i = threadIdx.x; i < P; i += kBlock) {
        const int ixj = i ^ j;
        if (ixj > i) {
          const uint64_t a = s[i], b = s[ixj];
          const bool desc = (i & k) == 0;
          if (desc ? (a < b) : (a > b)) {
            s[i] = b;
            s[ixj] = a;
          }
        }
      }
      __syncthreads();
    }
  }
}

__host__ __device__ inline int pow2_ceil(int x) {
  int p = 1;
  while (p < x) p <<= 1;
  return p;
}

// ---------------------------------------------------------------------------
// Scoring (Eq. 1 / Eq. 4) in binary32 for one request of prompt length b >= 1:
//   Phi = (q+1)/(b+1) * (w_base + w_urg * W/C(b) + w_fair * ln(b+1)).
// ---------------------------------------------------------------------------
struct CostF {
  float c0, c1, c2;
};

__device__ __forceinline__ float phi_f32(int b, float arrival, float now, const QParams& p, const CostF& c) {
  const float fb = (float)b;
  const float bp1 = fb + 1.0f;
  const float W = fmaxf(now - arrival, 0.0f);  // NaN arrival or future arrival -> 0
  const float C = __builtin_fmaf(__builtin_fmaf(c.c2, fb, c.c1), fb, c.c0);
  const float cs = W * __builtin_amdgcn_rcpf(C);
  const float lg = __builtin_amdgcn_logf(bp1);  // log2(b + 1)
  const float inner = __builtin_fmaf(p.wf2, lg, __builtin_fmaf(p.wu, cs, p.wb));
  return p.qn * inner * __builtin_amdgcn_rcpf(bp1);
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
    for (int q = threadIdx.x; q < k; q += blockDim.x) {
      const double m = tab->mean[q];
      const double wb = (double)theta->a_base * m + (double)theta->b_base;
      const double wu = (double)theta->a_urg * m + (double)theta->b_urg;
      const double wf = (double)theta->a_fair * m + (double)theta->b_fair;
      QParams p;
      p.wb = (float)wb;
      p.wu = (float)wu;
      p.wf2 = (float)(wf * 0.69314718055994530942);
      p.qn = (float)(q + 1);
      qp[q] = p;
    }
  }
}

__device__ __forceinline__ int route_lut(int b, int L, const uint8_t* lut) {
  return b <= 0 ? -1 : (int)lut[b < L ? b : L];
}

}  // namespace ewsjf
