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

// A walk up the length axis that gives the queue of each length in turn
// (the same queue as lut_entry): one search places the walk's first
// length, then the walk moves to the next queue start (or bound) as it is
// passed.  Lengths must be visited one by one in increasing order from the
// first, all within [1, L].
template <class P>
struct QueueWalk {
  P bounds, lo, hi;
  int k;
  bool gapped;
  // gapped: i = last queue starting at or below the length, nxt = the next
  // start; contiguous: i = bounds passed, nxt = the next bound
  int i, hi_i, nxt;
  static constexpr int kBig = 0x7fffffff;

  __device__ __forceinline__ void start(int b0) {
    i = gapped ? count_le(lo, k, b0) - 1 : count_le(bounds, k - 1, b0);
    hi_i = gapped && i >= 0 ? hi[i] : 0;
    nxt = gapped ? (i + 1 < k ? lo[i + 1] : kBig) : (i < k - 1 ? bounds[i] : kBig);
  }

  __device__ __forceinline__ int at(int x) {
    if (x >= nxt) {  // starts and bounds strictly increase, so at most one per length
      ++i;
      if (gapped) {
        hi_i = hi[i];
        nxt = i + 1 < k ? lo[i + 1] : kBig;
      } else {
        nxt = i < k - 1 ? bounds[i] : kBig;
      }
    }
    if (!gapped || i < 0 || x <= hi_i || i == k - 1) return i < 0 ? 0 : i;
    const int tq = gap_tolerance(x, hi_i, nxt, i);
    return tq >= 0 ? tq : gap_nearer(x, hi_i, nxt, i);
  }
};

// Thread t of nthreads writes its share of the lut's 32-bit words, four
// entries per store.  The same entries as lut_entry.
template <class P>
__device__ void lut_fill(uint8_t* lut, int t, int nthreads, int L, bool gapped, P bounds, P lo, P hi, int k) {
  const int per = (kLutWords + nthreads - 1) / nthreads;
  const int w0 = t * per, w1 = min(kLutWords, w0 + per);
  if (w0 >= w1) return;
  QueueWalk<P> qw{bounds, lo, hi, k, gapped, 0, 0, 0};
  qw.start(max(4 * w0, 1));
  for (int w = w0; w < w1; ++w) {
    uint32_t word = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int x = 4 * w + j;
      const int q = (x >= 1 && x <= L) ? qw.at(x) : 0;
      word |= (uint32_t)q << (8 * j);
    }
    *reinterpret_cast<uint32_t*>(lut + 4 * w) = word;
  }
}

// Thread t of nthreads writes its share of the compact routing map (the
// table's route words): word w = (queue of length 32 w - 1) << 32 | the
// mask of lengths 32 w + j in [1, L] whose queue is one above the queue of
// the length before.  Under both readings the queue of a length never falls
// and rises by at most one per length (contiguous bounds strictly increase;
// in the gapped reading each gap is split once, lower part to the lower
// queue), so the mask and the base give every queue.  Lengths past L keep
// the queue of L.
template <class P>
__device__ void route_fill(uint64_t* route, int t, int nthreads, int L, bool gapped, P bounds, P lo, P hi, int k) {
  const int per = (kRouteWords + nthreads - 1) / nthreads;
  const int w0 = t * per, w1 = min(kRouteWords, w0 + per);
  if (w0 >= w1) return;
  QueueWalk<P> qw{bounds, lo, hi, k, gapped, 0, 0, 0};
  int prev = 0;  // queue of length 32 w0 - 1 (lengths <= 0 count as queue 0)
  if (w0 == 0) {
    qw.start(1);
  } else {
    const int x = min(32 * w0 - 1, L);
    qw.start(x);
    prev = qw.at(x);
  }
  for (int w = w0; w < w1; ++w) {
    const uint32_t base = (uint32_t)prev;
    uint32_t mask = 0;
    for (int j = 0; j < 32; ++j) {
      const int x = 32 * w + j;
      if (x < 1 || x > L) continue;
      const int q = qw.at(x);
      mask |= (uint32_t)(q != prev) << j;
      prev = q;
    }
    route[w] = ((uint64_t)base << 32) | mask;
  }
}

}  // namespace ewsjf
