// The routing rule that a queue table's lut encodes, for the kernels that
// (re)build the lut.  Two readings of the table:
//
//   contiguous  the queues cover the length axis: queue i holds
//               [bounds[i-1], bounds[i]), queue 0 is open below and the last
//               queue open above (Section 3.2, Dispatcher; Section 5).
//   gapped      queue i holds the lengths [lo_i, hi_i] and the gaps between
//               queues follow the Dispatcher's rule for gap-falling requests
//               (Section 4.3 and the appendix algorithm): a length L between
//               queues i and i+1 joins queue i when L <= 1.10 max_len_i
//               (max_len = hi + 1), queue i+1 when L >= 0.90 min_len_{i+1}
//               (min_len = lo), in exact integers; a true gap takes the
//               nearer neighbour (L - hi_i against lo_{i+1} - L, ties to the
//               lower) until a dispatched request puts a bubble queue there.
//               Below the first queue: queue 0; above the last: queue k-1.
#pragma once

#include <stdint.h>

namespace ewsjf {

// The number of entries of a[0..n) that are <= b (a ascending).
template <class P>
__device__ __forceinline__ int count_le(P a, int n, int b) {
  int lo = 0, hi = n;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (a[mid] <= b) lo = mid + 1;
    else hi = mid;
  }
  return lo;
}

// Algorithm 2's first two branches for b between queues i and i+1 (hi_i <
// b < lo_next): i, i + 1, or -1 for a true gap.
__device__ __forceinline__ int gap_tolerance(int b, int hi_i, int lo_next, int i) {
  if (10 * (int64_t)b <= 11 * ((int64_t)hi_i + 1)) return i;
  if (10 * (int64_t)b >= 9 * (int64_t)lo_next) return i + 1;
  return -1;
}

__device__ __forceinline__ int gap_nearer(int b, int hi_i, int lo_next, int i) {
  return b - hi_i <= lo_next - b ? i : i + 1;
}

// Queue of length b >= 1 in the gapped reading of lo/hi[0..k).
template <class P>
__device__ __forceinline__ int lut_gapped(int b, P lo, P hi, int k) {
  const int i = count_le(lo, k, b) - 1;
  if (i < 0) return 0;
  if (b <= hi[i] || i == k - 1) return i;
  const int t = gap_tolerance(b, hi[i], lo[i + 1], i);
  return t >= 0 ? t : gap_nearer(b, hi[i], lo[i + 1], i);
}

// lut entry of index e (lut[0] and entries past L are 0).
template <class P>
__device__ __forceinline__ uint8_t lut_entry(int e, int L, bool gapped, P bounds, P lo, P hi, int k) {
  if (e < 1 || e > L) return 0;
  return (uint8_t)(gapped ? lut_gapped(e, lo, hi, k) : count_le(bounds, k - 1, e));
}

constexpr int kLutWords = (EWSJF_MAX_LEN + 16) / 4;

// Thread t of nthreads writes its share of the lut's 32-bit words: one
// search places its first length, then the walk up the length axis moves to
// the next queue start (or bound) as it is passed, and four entries go out
// per store.  The same entries as lut_entry.
template <class P>
__device__ void lut_fill(uint8_t* lut, int t, int nthreads, int L, bool gapped, P bounds, P lo, P hi, int k) {
  const int per = (kLutWords + nthreads - 1) / nthreads;
  const int w0 = t * per, w1 = min(kLutWords, w0 + per);
  if (w0 >= w1) return;
  const int big = 0x7fffffff;
  const int b0 = max(4 * w0, 1);
  // gapped: i = last queue starting at or below the length, nxt = the next start;
  // contiguous: i = bounds passed, nxt = the next bound
  int i = gapped ? count_le(lo, k, b0) - 1 : count_le(bounds, k - 1, b0);
  int hi_i = gapped && i >= 0 ? hi[i] : 0;
  int nxt = gapped ? (i + 1 < k ? lo[i + 1] : big) : (i < k - 1 ? bounds[i] : big);
  for (int w = w0; w < w1; ++w) {
    uint32_t word = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int x = 4 * w + j;
      int q = 0;
      if (x >= 1 && x <= L) {
        if (x >= nxt) {  // starts and bounds strictly increase, so at most one per length
          ++i;
          if (gapped) {
            hi_i = hi[i];
            nxt = i + 1 < k ? lo[i + 1] : big;
          } else {
            nxt = i < k - 1 ? bounds[i] : big;
          }
        }
        if (!gapped || i < 0 || x <= hi_i || i == k - 1) {
          q = i < 0 ? 0 : i;
        } else {
          const int tq = gap_tolerance(x, hi_i, nxt, i);
          q = tq >= 0 ? tq : gap_nearer(x, hi_i, nxt, i);
        }
      }
      word |= (uint32_t)q << (8 * j);
    }
    *reinterpret_cast<uint32_t*>(lut + 4 * w) = word;
  }
}

}  // namespace ewsjf
