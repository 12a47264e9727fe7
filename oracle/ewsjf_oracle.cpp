// EWSJF scheduler core -- CPU oracle.
//
// TEST INFRASTRUCTURE ONLY.  This file is the plain, slow, single-threaded
// definition that the HIP library is checked against.  Only the tests, the
// smoke check and the benchmark's CPU-baseline leg may load it; the product
// path never calls it.  It shares no code, header, table or helper with the
// HIP library.
//
// Every floating-point step is IEEE-754 binary64 in the order written here
// (built with -ffp-contract=off so no multiply-add is fused).
//
// What it computes (EWSJF, arXiv 2601.21758):
//   * Refine-and-Prune partitioning of an observation window of prompt
//     lengths into contiguous queue intervals (Section 4.2, Stages 1-3,
//     Eq. 2 and Eq. 3).
//   * Dynamic Queue Routing of each request to the one interval containing
//     its prompt length (Section 3.2 "Dispatcher"; Section 5 "Stability and
//     Correctness").
//   * Density-Weighted Scoring Phi(r, q) (Eq. 1 / Eq. 4) with the affine
//     context-aware weights of the meta-policy (Section 4.1, Section 4.4.1).
//   * Top-B admission ordered by (score desc, request id asc).
//
// Readings of passages the paper leaves open are listed next to the code
// that adopts them.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <limits>
#include <utility>
#include <vector>

namespace {

constexpr int kOk = 0;
constexpr int kErrArg = -2;

// ---------------------------------------------------------------------------
// Window: clamp to [1, L], sort, and list the distinct values with their
// multiplicities.  The paper's D is the sorted set of window prompt lengths
// (Section 4.2, "Formalism").
// ---------------------------------------------------------------------------
struct Distinct {
  std::vector<int32_t> v;  // strictly increasing
  std::vector<int64_t> c;  // multiplicity of v[j]
};

Distinct sorted_distinct(const int32_t* w, int64_t n, int32_t max_len) {
  std::vector<int32_t> d(w, w + n);
  for (auto& x : d) x = std::min(std::max(x, 1), max_len);
  std::sort(d.begin(), d.end());
  Distinct out;
  for (int64_t i = 0; i < n; ++i) {
    if (out.v.empty() || out.v.back() != d[i]) {
      out.v.push_back(d[i]);
      out.c.push_back(1);
    } else {
      out.c.back() += 1;
    }
  }
  return out;
}

// ---------------------------------------------------------------------------
// Stage 1: coarse partitioning (Section 4.2, "Stage 1").  Returns cluster
// start indices into the distinct-value list; cluster i is
// [start[i], start[i+1]).
//
// EQUAL_WIDTH(K): the workloads start from K equal-width queues over the
//   window's [min, max]; value v goes to bin floor((v - lo) * K / (hi-lo+1)),
//   non-empty bins in order.
// KMEANS3: the paper's k-means with k = 3, taken as the exact 1-D optimum
//   (minimum within-cluster sum of squares over the multiset).  In one
//   dimension optimal clusters are contiguous runs of the sorted values, so
//   every split (i, j) is tried; F = S1^2/N1 + S2^2/N2 + S3^2/N3 is maximal
//   exactly where the sum of squares is minimal.  Ties keep the
//   lexicographically smallest (i, j).
// ---------------------------------------------------------------------------
std::vector<int32_t> stage1_equal_width(const Distinct& d, int32_t K) {
  const int32_t V = (int32_t)d.v.size();
  std::vector<int32_t> starts;
  const int64_t lo = d.v[0], hi = d.v[V - 1];
  const int64_t width = hi - lo + 1;
  int64_t prev_bin = -1;
  for (int32_t j = 0; j < V; ++j) {
    const int64_t bin = ((int64_t)d.v[j] - lo) * (int64_t)K / width;
    if (j == 0 || bin != prev_bin) starts.push_back(j);
    prev_bin = bin;
  }
  return starts;
}

std::vector<int32_t> stage1_kmeans3(const Distinct& d) {
  const int32_t V = (int32_t)d.v.size();
  std::vector<int32_t> starts;
  if (V <= 3) {
    for (int32_t j = 0; j < V; ++j) starts.push_back(j);
    return starts;
  }
  // Exact integer prefix sums of counts and of count * value.
  std::vector<int64_t> N(V + 1, 0), S(V + 1, 0);
  for (int32_t j = 0; j < V; ++j) {
    N[j + 1] = N[j] + d.c[j];
    S[j + 1] = S[j] + d.c[j] * (int64_t)d.v[j];
  }
  double best = -1.0;
  int32_t bi = 1, bj = 2;
  for (int32_t i = 1; i <= V - 2; ++i) {
    for (int32_t j = i + 1; j <= V - 1; ++j) {
      const double n1 = (double)N[i], s1 = (double)S[i];
      const double n2 = (double)(N[j] - N[i]), s2 = (double)(S[j] - S[i]);
      const double n3 = (double)(N[V] - N[j]), s3 = (double)(S[V] - S[j]);
      const double F = ((s1 * s1) / n1 + (s2 * s2) / n2) + (s3 * s3) / n3;
      if (F > best) {
        best = F;
        bi = i;
        bj = j;
      }
    }
  }
  starts.push_back(0);
  starts.push_back(bi);
  starts.push_back(bj);
  return starts;
}

// ---------------------------------------------------------------------------
// Stage 2: recursive refinement (Section 4.2, "Stage 2", Eq. 2).
//
// A cluster is the distinct-value range [s, e).  G is the set of gaps
// between consecutive members; a gap is significant when it exceeds
// alpha * mean(G).
//   gap_mode 0 (default): G is taken over distinct values, so
//     mean(G) = span / (V_C - 1)  (the gaps telescope to the span);
//     the test is gap * (V_C - 1) > alpha * span.
//   gap_mode 1: G is taken over the multiset, zero gaps between duplicates
//     included, so mean(G) = span / (n_C - 1); test gap * (n_C-1) > alpha*span.
// The cluster is cut at every significant gap at once and each piece is
// refined again.  Recursion stops when no gap is significant, or when the
// value span (the cluster's width) is below min_width, or when the cluster
// has too few distinct values to hold a significant gap.
// ---------------------------------------------------------------------------
std::vector<int32_t> stage2(const Distinct& d, const std::vector<int32_t>& coarse_starts,
                            double alpha, int32_t min_width, int32_t gap_mode) {
  const int32_t V = (int32_t)d.v.size();
  std::vector<std::pair<int32_t, int32_t>> work, leaves;
  for (size_t i = 0; i < coarse_starts.size(); ++i) {
    const int32_t s = coarse_starts[i];
    const int32_t e = (i + 1 < coarse_starts.size()) ? coarse_starts[i + 1] : V;
    work.push_back({s, e});
  }
  const int32_t min_distinct = (gap_mode == 0) ? 3 : 2;
  while (!work.empty()) {
    const auto [s, e] = work.back();
    work.pop_back();
    const int32_t VC = e - s;
    const int64_t span = (int64_t)d.v[e - 1] - (int64_t)d.v[s];
    if (VC < min_distinct || span < (int64_t)min_width) {
      leaves.push_back({s, e});
      continue;
    }
    int64_t members_minus_one;
    if (gap_mode == 0) {
      members_minus_one = VC - 1;
    } else {
      int64_t nC = 0;
      for (int32_t j = s; j < e; ++j) nC += d.c[j];
      members_minus_one = nC - 1;
    }
    const double rhs = alpha * (double)span;
    std::vector<int32_t> cut_after;
    for (int32_t j = s; j < e - 1; ++j) {
      const double lhs = (double)((int64_t)d.v[j + 1] - (int64_t)d.v[j]) * (double)members_minus_one;
      if (lhs > rhs) cut_after.push_back(j);
    }
    if (cut_after.empty()) {
      leaves.push_back({s, e});
      continue;
    }
    int32_t piece_start = s;
    for (int32_t j : cut_after) {
      work.push_back({piece_start, j + 1});
      piece_start = j + 1;
    }
    work.push_back({piece_start, e});
  }
  std::sort(leaves.begin(), leaves.end());
  std::vector<int32_t> starts;
  for (auto& l : leaves) starts.push_back(l.first);
  return starts;
}

// ---------------------------------------------------------------------------
// Stage 3: intelligent pruning (Section 4.2, "Stage 3", Eq. 3).
//
// Adjacent queues are merged, lowest scheduling utility first, until at most
// max_queues remain.  Density rho(q) = n_q / (hi_q - lo_q + 1): window
// requests per token of the queue's value span.  Mean = S_q / n_q.
//   U_i = (rho_i + rho_{i+1}) / (|mean_{i+1} - mean_i| + eps).
// One merge at a time; U is recomputed from the current queues before every
// merge; ties go to the leftmost pair.  A merged queue sums counts and
// length sums and spans both intervals.
// ---------------------------------------------------------------------------
struct Leaf {
  int64_t n, S;
  int32_t lo, hi;
};

std::vector<Leaf> stage3(std::vector<Leaf> q, int32_t max_queues, double eps) {
  while ((int32_t)q.size() > max_queues) {
    int32_t best_i = 0;
    double best_u = 0.0;
    for (int32_t i = 0; i + 1 < (int32_t)q.size(); ++i) {
      const double rho_a = (double)q[i].n / (double)((int64_t)q[i].hi - (int64_t)q[i].lo + 1);
      const double rho_b = (double)q[i + 1].n / (double)((int64_t)q[i + 1].hi - (int64_t)q[i + 1].lo + 1);
      const double m_a = (double)q[i].S / (double)q[i].n;
      const double m_b = (double)q[i + 1].S / (double)q[i + 1].n;
      const double u = (rho_a + rho_b) / (std::fabs(m_b - m_a) + eps);
      if (i == 0 || u < best_u) {
        best_u = u;
        best_i = i;
      }
    }
    Leaf merged{q[best_i].n + q[best_i + 1].n, q[best_i].S + q[best_i + 1].S, q[best_i].lo,
                q[best_i + 1].hi};
    q[best_i] = merged;
    q.erase(q.begin() + best_i + 1);
  }
  return q;
}

std::vector<Leaf> leaves_from_starts(const Distinct& d, const std::vector<int32_t>& starts) {
  const int32_t V = (int32_t)d.v.size();
  std::vector<Leaf> out;
  for (size_t i = 0; i < starts.size(); ++i) {
    const int32_t s = starts[i];
    const int32_t e = (i + 1 < starts.size()) ? starts[i + 1] : V;
    Leaf l{0, 0, d.v[s], d.v[e - 1]};
    for (int32_t j = s; j < e; ++j) {
      l.n += d.c[j];
      l.S += d.c[j] * (int64_t)d.v[j];
    }
    out.push_back(l);
  }
  return out;
}

bool params_ok(int64_t n, int32_t init_mode, int32_t init_queues, int32_t max_queues, int32_t min_width,
               int32_t max_len, double alpha, double eps, int32_t gap_mode) {
  if (n < 1) return false;
  if (init_mode != 0 && init_mode != 1) return false;
  if (init_mode == 0 && init_queues < 1) return false;
  if (max_queues < 1 || min_width < 0 || max_len < 1) return false;
  if (!(alpha > 1.0) || !std::isfinite(alpha)) return false;
  if (!(eps > 0.0) || !std::isfinite(eps)) return false;
  if (gap_mode != 0 && gap_mode != 1) return false;
  return true;
}

// Route one prompt length (Section 3.2 "Dispatcher").  The queues form a
// contiguous cover of the length axis: bounds[i] is the smallest window
// length of queue i+1, queue 0 extends down to 1 and the last queue up
// without limit, so each length b >= 1 lies in exactly one interval.
// Empty slots (b <= 0) route nowhere (-1).
int32_t route_one(int32_t b, const int32_t* bounds, int32_t k) {
  if (b <= 0) return -1;
  return (int32_t)(std::upper_bound(bounds, bounds + (k - 1), b) - bounds);
}

// ---------------------------------------------------------------------------
// Algorithm 2 (Section 4.3 and the appendix algorithm "On-Demand Bubble Queue
// Creation"): the Dispatcher's rule for a length that falls between two
// queues, and the gapped reading of a queue table that it needs.
//
// Readings (the paper leaves these open):
//   B1 Queue i holds the lengths [lo_i, hi_i]: for a partitioned table the
//      smallest and largest window length that fell in it, for a bubble its
//      interval.  In the algorithm's notation min_len = lo_i and max_len =
//      hi_i + 1 (the half-open [min_len, max_len) of Section 4.2).
//   B2 A length below the first queue goes to queue 0 and one above the last
//      to queue k-1: the algorithm covers gaps between two queues only.
//   B3 The tolerances in exact integer arithmetic: L <= 1.10 * max_len is
//      10 L <= 11 max_len, and L >= 0.90 * min_len is 10 L >= 9 min_len.
//   B4 range / 2 on integers: the bubble is [L - floor(range/2),
//      L - floor(range/2) + range) (range lengths, L inside), clipped to the
//      gap [max_len_i, min_len_{i+1}).
//   B5 A bubble's profile is the request that created it: count 1, sum L,
//      mean L; lo/hi are its interval (B1).
//   B6 Requests are dispatched one at a time in arrival order (T1's FIFO
//      order), each against the queue set the earlier ones left; empty slots
//      (len <= 0) are not dispatched (qid -1).  A request's queue index is its
//      queue's place in the final set (a bubble shifts the queues above it).
//   B7 The set holds at most max_queues queues.  Once it is full, a request
//      that would create a bubble joins the nearer neighbour (L - hi_i
//      against lo_{i+1} - L; equal distances: the lower).
//   B8 A length routed without being dispatched (a request already pending
//      when the queue set changes) takes the algorithm's first two branches,
//      and B7's nearer neighbour in place of a bubble.
// ---------------------------------------------------------------------------

// Where length b >= 1 lies: returns false with *q its queue (inside one, or
// below the first / above the last, B2), or true with *q the queue below the
// gap that holds b.
bool in_gap(int32_t b, const int32_t* lo, const int32_t* hi, int32_t k, int32_t* q) {
  const int32_t i = (int32_t)(std::upper_bound(lo, lo + k, b) - lo) - 1;  // last queue with lo <= b
  if (i < 0) {
    *q = 0;
    return false;
  }
  *q = i;
  return !(b <= hi[i] || i == k - 1);
}

// Algorithm 2's first two branches (B3) for b between queues i and i+1:
// i, i + 1, or -1 for a true gap.
int32_t tolerance(int64_t b, int64_t max_len_i, int64_t min_len_next, int32_t i) {
  if (10 * b <= 11 * max_len_i) return i;
  if (10 * b >= 9 * min_len_next) return i + 1;
  return -1;
}

// B7: the nearer of queues i and i+1.
int32_t nearer(int64_t b, int64_t hi_i, int64_t lo_next, int32_t i) { return b - hi_i <= lo_next - b ? i : i + 1; }

// B8: the queue of length b in the gapped reading, without dispatch.
int32_t route_gapped(int32_t b, const int32_t* lo, const int32_t* hi, int32_t k) {
  if (b <= 0) return -1;
  int32_t i;
  if (!in_gap(b, lo, hi, k, &i)) return i;
  const int32_t t = tolerance(b, (int64_t)hi[i] + 1, lo[i + 1], i);
  return t >= 0 ? t : nearer(b, hi[i], lo[i + 1], i);
}

// The queue of length b under the table's reading: the contiguous cover of
// bounds, or the gapped reading of lo/hi.
int32_t route_table(int32_t b, const int32_t* bounds, const int32_t* lo, const int32_t* hi, int32_t k,
                    int32_t gapped) {
  return gapped ? route_gapped(b, lo, hi, k) : route_one(b, bounds, k);
}


// ---------------------------------------------------------------------------
// Algorithm 1 (Section 3.2, "Tactical Loop"): the paper's own batch rule
// over per-queue FIFOs.
//
// Readings (the paper leaves these open):
//   T1 Each queue is a FIFO of its pending requests in arrival order; equal
//      arrivals keep request-id order, a NaN arrival counts as +inf and -0
//      as +0.  peek() is the oldest request.
//   T2 CalculateScore is Phi (Eq. 1 / Eq. 4) of the head request with the
//      queue's profile, evaluated exactly as in the per-request scoring
//      below and rounded once to binary32 (NaN -> -inf).
//   T3 ArgMax over the non-empty queues; equal scores go to the lower queue
//      index.
//   T4 GreedyFill pulls q_prim's requests oldest first until the batch
//      holds B requests or q_prim is empty.
//   T5 GetAdjacent(q_prim) = the queues directly below and above q_prim in
//      length order that are non-empty; Backfill drains them oldest first,
//      the one with the higher head score first (equal scores: lower index
//      first), until the batch is full.
//   T6 empty_cnt counts consecutive steps a queue was empty (a non-empty
//      step resets it).  Removals are applied after the batch is built
//      (scores of this step use the queue indices at its start).  The
//      lowest-index queue past the threshold goes first; it is re-absorbed
//      by the neighbour whose pair has the lower utility U of Eq. 3 (the
//      Stage-3 merge rule; equal U: the lower neighbour): the boundary
//      between the two disappears, aggregates add up, lo/hi span both, and
//      the merged queue keeps the absorber's empty_cnt.  The last remaining
//      queue is never removed.
// ---------------------------------------------------------------------------
struct FifoKey {
  float arrival;  // canonical: NaN -> +inf, -0 -> +0
  int64_t id;
};

float canonical_arrival(float a) {
  if (std::isnan(a)) return std::numeric_limits<float>::infinity();
  if (a == 0.0f) return 0.0f;
  return a;
}

bool older(const FifoKey& x, const FifoKey& y) {
  return x.arrival < y.arrival || (x.arrival == y.arrival && x.id < y.id);
}

// Density-Weighted Scoring, Eq. 1 / Eq. 4, of one request of queue q:
//   Phi = qf * ((w_base + w_urg * cs) + w_fair * ln(b + 1))
//   qf  = q_i / (b + 1) with q_i the 1-based queue index in length order,
//   cs  = W_t / C_prefill(b), W_t = max(0, now - arrival) seconds,
//   C_prefill(b) = c0 + c1*b + c2*b*b seconds,
//   w_x = a_x * mean_q + b_x (the affine meta-policy of Section 4.1 applied
//   to all three weights), mean_q the queue's window mean length;
//   th = (a_base, b_base, a_urg, b_urg, a_fair, b_fair).
// Returned rounded once to binary32, NaN mapped to -inf.
float phi_key(int32_t len, float arrival, float now, int32_t q, double mean_q, const float* th, double c0,
              double c1, double c2) {
  const double m = mean_q;
  const double w_base = (double)th[0] * m + (double)th[1];
  const double w_urg = (double)th[2] * m + (double)th[3];
  const double w_fair = (double)th[4] * m + (double)th[5];
  double W = (double)now - (double)arrival;
  if (!(W > 0.0)) W = 0.0;
  const double b = (double)len;
  const double C = c0 + c1 * b + c2 * b * b;
  const double cs = W / C;
  const double qf = (double)(q + 1) / (b + 1.0);
  const double phi = qf * ((w_base + w_urg * cs) + w_fair * std::log(b + 1.0));
  float key = (float)phi;
  if (std::isnan(key)) key = -std::numeric_limits<float>::infinity();
  return key;
}

double utility(const Leaf& a, const Leaf& b, double eps) {
  const double rho_a = (double)a.n / (double)((int64_t)a.hi - (int64_t)a.lo + 1);
  const double rho_b = (double)b.n / (double)((int64_t)b.hi - (int64_t)b.lo + 1);
  const double m_a = (double)a.S / (double)a.n;
  const double m_b = (double)b.S / (double)b.n;
  return (rho_a + rho_b) / (std::fabs(m_b - m_a) + eps);
}

}  // namespace

extern "C" {

int oracle_version(void) { return 1; }

// Distinct clamped window values; returns V (v_out/c_out need n entries).
int64_t oracle_distinct(const int32_t* window, int64_t n, int32_t max_len, int32_t* v_out,
                        int64_t* c_out) {
  if (n < 0 || max_len < 1) return kErrArg;
  Distinct d = sorted_distinct(window, n, max_len);
  for (size_t j = 0; j < d.v.size(); ++j) {
    v_out[j] = d.v[j];
    c_out[j] = d.c[j];
  }
  return (int64_t)d.v.size();
}

// Stage 1 over a distinct list; writes cluster starts, returns their count.
int32_t oracle_stage1(const int32_t* v, const int64_t* c, int32_t V, int32_t init_mode,
                      int32_t init_queues, int32_t* starts_out) {
  if (V < 1) return kErrArg;
  Distinct d{std::vector<int32_t>(v, v + V), std::vector<int64_t>(c, c + V)};
  std::vector<int32_t> st = init_mode == 0 ? stage1_equal_width(d, init_queues) : stage1_kmeans3(d);
  for (size_t i = 0; i < st.size(); ++i) starts_out[i] = st[i];
  return (int32_t)st.size();
}

// Stage 2 from given coarse starts; writes leaf starts, returns their count.
int32_t oracle_stage2(const int32_t* v, const int64_t* c, int32_t V, const int32_t* coarse_starts,
                      int32_t n_coarse, double alpha, int32_t min_width, int32_t gap_mode,
                      int32_t* leaf_starts_out) {
  if (V < 1 || n_coarse < 1) return kErrArg;
  Distinct d{std::vector<int32_t>(v, v + V), std::vector<int64_t>(c, c + V)};
  std::vector<int32_t> cs(coarse_starts, coarse_starts + n_coarse);
  std::vector<int32_t> st = stage2(d, cs, alpha, min_width, gap_mode);
  for (size_t i = 0; i < st.size(); ++i) leaf_starts_out[i] = st[i];
  return (int32_t)st.size();
}

// Stage 3 over explicit queues (n, S, lo, hi in length order); returns k.
int32_t oracle_stage3(const int64_t* n, const int64_t* S, const int32_t* lo, const int32_t* hi,
                      int32_t n_leaves, int32_t max_queues, double eps, int64_t* n_out, int64_t* S_out,
                      int32_t* lo_out, int32_t* hi_out) {
  if (n_leaves < 1 || max_queues < 1) return kErrArg;
  std::vector<Leaf> q;
  for (int32_t i = 0; i < n_leaves; ++i) q.push_back({n[i], S[i], lo[i], hi[i]});
  q = stage3(q, max_queues, eps);
  for (size_t i = 0; i < q.size(); ++i) {
    n_out[i] = q[i].n;
    S_out[i] = q[i].S;
    lo_out[i] = q[i].lo;
    hi_out[i] = q[i].hi;
  }
  return (int32_t)q.size();
}

// Full Refine-and-Prune.  Output arrays hold max_queues entries (bounds:
// max_queues - 1).  diag[0..2] = distinct values, coarse clusters, leaves.
int oracle_partition(const int32_t* window, int64_t n, int32_t init_mode, int32_t init_queues,
                     int32_t max_queues, int32_t min_width, int32_t max_len, double alpha, double eps,
                     int32_t gap_mode, int32_t* k_out, int32_t* bounds, int64_t* count, int64_t* sum,
                     int32_t* lo, int32_t* hi, double* mean, int32_t* diag) {
  if (!params_ok(n, init_mode, init_queues, max_queues, min_width, max_len, alpha, eps, gap_mode))
    return kErrArg;
  Distinct d = sorted_distinct(window, n, max_len);
  std::vector<int32_t> coarse =
      init_mode == 0 ? stage1_equal_width(d, init_queues) : stage1_kmeans3(d);
  std::vector<int32_t> leaf_starts = stage2(d, coarse, alpha, min_width, gap_mode);
  std::vector<Leaf> q = stage3(leaves_from_starts(d, leaf_starts), max_queues, eps);
  const int32_t k = (int32_t)q.size();
  *k_out = k;
  for (int32_t i = 0; i < k; ++i) {
    if (i > 0) bounds[i - 1] = q[i].lo;
    count[i] = q[i].n;
    sum[i] = q[i].S;
    lo[i] = q[i].lo;
    hi[i] = q[i].hi;
    mean[i] = (double)q[i].S / (double)q[i].n;
  }
  if (diag) {
    diag[0] = (int32_t)d.v.size();
    diag[1] = (int32_t)coarse.size();
    diag[2] = (int32_t)leaf_starts.size();
  }
  return kOk;
}

void oracle_route(const int32_t* len, int64_t n, const int32_t* bounds, int32_t k, int32_t* qid) {
  for (int64_t i = 0; i < n; ++i) qid[i] = route_one(len[i], bounds, k);
}

void oracle_route_gapped(const int32_t* len, int64_t n, const int32_t* lo, const int32_t* hi, int32_t k,
                         int32_t* qid) {
  for (int64_t i = 0; i < n; ++i) qid[i] = route_gapped(len[i], lo, hi, k);
}

// The Dispatcher with on-demand bubble queues (Algorithm 2, readings B1-B7)
// over the requests with len > 0, in arrival order.  The queue set (k,
// bounds, count, sum, lo, hi, mean; arrays of max_queues entries) is read in
// its gapped reading and updated in place: bubbles are inserted in length
// order, bounds[i-1] = lo_i.  qid[i] = request i's queue in the final set.
int oracle_dispatch(const int32_t* len, const float* arrival, int64_t n, int32_t* k_io, int32_t* bounds,
                    int64_t* count, int64_t* sum, int32_t* lo, int32_t* hi, double* mean, int32_t bubble_width,
                    int32_t max_queues, int32_t* qid) {
  const int32_t k = *k_io;
  if (k < 1 || n < 0 || bubble_width < 1 || max_queues < k) return kErrArg;
  struct Q {
    int32_t lo, hi;
    int64_t n, S;
    double mean;
    int32_t ident;  // stable name of the queue while others are inserted
  };
  std::vector<Q> qs(k);
  for (int32_t q = 0; q < k; ++q) qs[q] = {lo[q], hi[q], count[q], sum[q], mean[q], q};
  std::vector<FifoKey> order;
  for (int64_t i = 0; i < n; ++i)
    if (len[i] > 0) order.push_back({canonical_arrival(arrival[i]), i});
  std::stable_sort(order.begin(), order.end(), older);
  std::vector<int32_t> who(n, -1);  // ident of each request's queue
  int32_t next_ident = k;
  for (const FifoKey& r : order) {
    const int64_t b = len[r.id];
    const int32_t m = (int32_t)qs.size();
    std::vector<int32_t> clo(m), chi(m);
    for (int32_t q = 0; q < m; ++q) {
      clo[q] = qs[q].lo;
      chi[q] = qs[q].hi;
    }
    int32_t i;
    if (!in_gap((int32_t)b, clo.data(), chi.data(), m, &i)) {
      who[r.id] = qs[i].ident;
      continue;
    }
    const int64_t max_len = (int64_t)chi[i] + 1, min_len = clo[i + 1];
    int32_t t = tolerance(b, max_len, min_len, i);
    if (t < 0 && m < max_queues) {  // a true gap: create a bubble queue
      const int64_t available = min_len - max_len;
      const int64_t range = std::min<int64_t>(bubble_width, available);
      const int64_t new_min = std::max(b - range / 2, max_len);
      const int64_t new_max = std::min(b - range / 2 + range, min_len);
      qs.insert(qs.begin() + i + 1, Q{(int32_t)new_min, (int32_t)(new_max - 1), 1, b, (double)b, next_ident});
      who[r.id] = next_ident++;
      continue;
    }
    if (t < 0) t = nearer(b, chi[i], clo[i + 1], i);
    who[r.id] = qs[t].ident;
  }
  const int32_t k2 = (int32_t)qs.size();
  std::vector<int32_t> place(next_ident);
  for (int32_t q = 0; q < k2; ++q) place[qs[q].ident] = q;
  for (int64_t i = 0; i < n; ++i) qid[i] = who[i] < 0 ? -1 : place[who[i]];
  *k_io = k2;
  for (int32_t q = 0; q < k2; ++q) {
    if (q > 0) bounds[q - 1] = qs[q].lo;
    count[q] = qs[q].n;
    sum[q] = qs[q].S;
    lo[q] = qs[q].lo;
    hi[q] = qs[q].hi;
    mean[q] = qs[q].mean;
  }
  return kOk;
}

// Density-Weighted Scoring (Eq. 1 / Eq. 4, defined in phi_key) for every
// pending request and parameter vector.  theta is [n_theta][6].  Output
// score[t * n + i] is Phi rounded once to binary32; a request whose Phi is
// NaN gets -inf; an empty slot (len <= 0) gets NaN, which marks it as not
// admissible.
void oracle_score(const int32_t* len, const float* arrival, int64_t n, float now, int32_t k,
                  const int32_t* bounds, const int32_t* lo, const int32_t* hi, int32_t gapped, const double* mean,
                  const float* theta, int32_t n_theta, double c0, double c1, double c2, float* score) {
  for (int32_t t = 0; t < n_theta; ++t) {
    const float* th = theta + 6 * t;
    for (int64_t i = 0; i < n; ++i) {
      const int32_t q = route_table(len[i], bounds, lo, hi, k, gapped);
      if (q < 0) {
        score[(int64_t)t * n + i] = std::numeric_limits<float>::quiet_NaN();
        continue;
      }
      score[(int64_t)t * n + i] = phi_key(len[i], arrival[i], now, q, mean[q], th, c0, c1, c2);
    }
  }
}

// Top-B admission for each parameter vector: the admissible requests
// (score not NaN) in order of (score desc, id asc); the first min(B, count)
// are admitted.  ids/top are [n_theta][B]; unused slots get id -1 / NaN.
void oracle_select(const float* score, int64_t n, int32_t n_theta, int32_t B, int32_t* ids, float* top,
                   int32_t* n_sel) {
  for (int32_t t = 0; t < n_theta; ++t) {
    const float* s = score + (int64_t)t * n;
    std::vector<int64_t> idx;
    for (int64_t i = 0; i < n; ++i)
      if (!std::isnan(s[i])) idx.push_back(i);
    const int64_t take = std::min<int64_t>(B, (int64_t)idx.size());
    auto before = [s](int64_t a, int64_t b) { return s[a] > s[b] || (s[a] == s[b] && a < b); };
    std::partial_sort(idx.begin(), idx.begin() + take, idx.end(), before);
    for (int64_t r = 0; r < B; ++r) {
      ids[(int64_t)t * B + r] = r < take ? (int32_t)idx[r] : -1;
      top[(int64_t)t * B + r] = r < take ? s[idx[r]] : std::numeric_limits<float>::quiet_NaN();
    }
    n_sel[t] = (int32_t)take;
  }
}

// One scheduling step: route, score and select (the scratch score array is
// [n_theta][n] floats supplied by the caller).
void oracle_step(const int32_t* len, const float* arrival, int64_t n, float now, int32_t k,
                 const int32_t* bounds, const int32_t* lo, const int32_t* hi, int32_t gapped, const double* mean,
                 const float* theta, int32_t n_theta, double c0, double c1, double c2, int32_t B,
                 float* score_scratch, int32_t* ids, float* top, int32_t* n_sel) {
  oracle_score(len, arrival, n, now, k, bounds, lo, hi, gapped, mean, theta, n_theta, c0, c1, c2, score_scratch);
  oracle_select(score_scratch, n, n_theta, B, ids, top, n_sel);
}


// One tactical step (Algorithm 1).  The queue table (k, bounds[k-1],
// count, sum, lo, hi, mean) and empty_cnt[k] are read and updated in place
// (queues past the empty threshold are removed after the batch is built).
// Outputs: ids[B] in batch order (-1 after n_sel), head_score[k at entry]
// (NaN for empty queues), q_prim (-1 when every queue is empty), removed[k
// at entry] (1 for the queues removed in this step).
int oracle_tactical_step(const int32_t* len, const float* arrival, int64_t n, float now, int32_t* k_io,
                         int32_t* bounds, int64_t* count, int64_t* sum, int32_t* lo, int32_t* hi, double* mean,
                         int32_t* empty_cnt, int32_t gapped, const float* theta, double c0, double c1, double c2,
                         int32_t B, int32_t empty_threshold, double eps, int32_t* ids, int32_t* n_sel,
                         int32_t* q_prim, float* head_score, int32_t* removed) {
  const int32_t k = *k_io;
  if (k < 1 || B < 0 || n < 0 || empty_threshold < 0) return kErrArg;
  // Dispatcher: every pending request joins the FIFO of its queue.
  std::vector<std::vector<FifoKey>> fifo(k);
  for (int64_t i = 0; i < n; ++i) {
    const int32_t q = route_table(len[i], bounds, lo, hi, k, gapped);
    if (q >= 0) fifo[q].push_back({canonical_arrival(arrival[i]), i});
  }
  for (auto& f : fifo) std::stable_sort(f.begin(), f.end(), older);
  // Score Updater: the head of every non-empty queue; empty queues count up.
  std::vector<bool> marked(k, false);
  for (int32_t q = 0; q < k; ++q) {
    removed[q] = 0;
    if (!fifo[q].empty()) {
      const int64_t h = fifo[q].front().id;
      head_score[q] = phi_key(len[h], arrival[h], now, q, mean[q], theta, c0, c1, c2);
      empty_cnt[q] = 0;
    } else {
      head_score[q] = std::numeric_limits<float>::quiet_NaN();
      empty_cnt[q] += 1;
      if (empty_cnt[q] > empty_threshold) marked[q] = true;
    }
  }
  // Batch Builder: ArgMax, GreedyFill, Backfill.
  int32_t prim = -1;
  for (int32_t q = 0; q < k; ++q)
    if (!fifo[q].empty() && (prim < 0 || head_score[q] > head_score[prim])) prim = q;
  *q_prim = prim;
  int32_t nb = 0;
  auto drain = [&](int32_t q) {
    for (const FifoKey& r : fifo[q]) {
      if (nb >= B) break;
      ids[nb++] = (int32_t)r.id;
    }
  };
  if (prim >= 0) {
    drain(prim);
    if (nb < B) {
      std::vector<int32_t> adj;
      if (prim > 0 && !fifo[prim - 1].empty()) adj.push_back(prim - 1);
      if (prim + 1 < k && !fifo[prim + 1].empty()) adj.push_back(prim + 1);
      if (adj.size() == 2 && head_score[adj[1]] > head_score[adj[0]]) std::swap(adj[0], adj[1]);
      for (int32_t q : adj) drain(q);
    }
  }
  *n_sel = nb;
  for (int32_t r = nb; r < B; ++r) ids[r] = -1;
  // RemoveQueue, after the batch: re-absorb each marked queue into a neighbour.
  std::vector<Leaf> qs(k);
  std::vector<int32_t> cnt(empty_cnt, empty_cnt + k), orig(k), bnd(bounds, bounds + (k - 1));
  for (int32_t q = 0; q < k; ++q) {
    qs[q] = {count[q], sum[q], lo[q], hi[q]};
    orig[q] = q;
  }
  for (;;) {
    int32_t r = -1;
    for (int32_t q = 0; q < (int32_t)qs.size(); ++q)
      if (marked[q]) {
        r = q;
        break;
      }
    if (r < 0 || qs.size() == 1) break;
    int32_t a;  // absorber
    if (r == 0) a = 1;
    else if (r + 1 == (int32_t)qs.size()) a = r - 1;
    else a = utility(qs[r - 1], qs[r], eps) <= utility(qs[r], qs[r + 1], eps) ? r - 1 : r + 1;
    Leaf& A = qs[a];
    A = {A.n + qs[r].n, A.S + qs[r].S, std::min(A.lo, qs[r].lo), std::max(A.hi, qs[r].hi)};
    removed[orig[r]] = 1;
    bnd.erase(bnd.begin() + std::min(r, a));
    qs.erase(qs.begin() + r);
    cnt.erase(cnt.begin() + r);
    orig.erase(orig.begin() + r);
    marked.erase(marked.begin() + r);
  }
  const int32_t k2 = (int32_t)qs.size();
  *k_io = k2;
  for (int32_t q = 0; q < k2; ++q) {
    if (q > 0) bounds[q - 1] = bnd[q - 1];
    count[q] = qs[q].n;
    sum[q] = qs[q].S;
    lo[q] = qs[q].lo;
    hi[q] = qs[q].hi;
    mean[q] = (double)qs[q].S / (double)qs[q].n;
    empty_cnt[q] = cnt[q];
  }
  return kOk;
}

}  // extern "C"
