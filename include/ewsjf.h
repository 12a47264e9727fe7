/*
 * ewsjf.h -- C ABI of the EWSJF scheduler core for AMD Instinct MI355X (gfx950).
 *
 * EWSJF (arXiv 2601.21758) schedules LLM requests above the execution engine.
 * This library implements its data-parallel core:
 *
 *   ewsjf_partition  Refine-and-Prune: an observation window of prompt lengths
 *                    -> contiguous queue intervals (Section 4.2, Stages 1-3,
 *                    Eq. 2 split test, Eq. 3 scheduling utility).
 *   ewsjf_trial_step / ewsjf_trial_finish  trials of batched scoring-parameter
 *                    proposals, each on its own pool with common arrivals, and
 *                    the Eq. 5 reward of each (the meta-optimizer's evaluator).
 *   ewsjf_dispatch   the Dispatcher with on-demand bubble queues (Section 4.3,
 *                    Algorithm 2): arriving requests in a gap between queues
 *                    join a neighbour within tolerance or create a queue.
 *   ewsjf_route      Dynamic Queue Routing: each request -> the one queue whose
 *                    interval holds its prompt length (Section 3.2 Dispatcher;
 *                    Section 5, deterministic routing over contiguous,
 *                    non-overlapping intervals).
 *   ewsjf_score      Density-Weighted Scoring Phi(r, q) of every request
 *                    (Eq. 1 / Eq. 4) with context-aware weights produced by the
 *                    affine meta-policy w_x = a_x * mean_q + b_x (Section 4.1,
 *                    Section 4.4.1).
 *   ewsjf_select     Top-B admission: the B admissible requests with the highest
 *                    score, ties to the lowest request id.
 *   ewsjf_step       route + score + select fused into one pass over the pool.
 *   ewsjf_ring_insert  new requests into a ring pool and the partition window
 *                    (the streaming scheduler's per-step update).
 *   ewsjf_window_histogram / ewsjf_window_advance / ewsjf_partition_hist
 *                    the window's length histogram, moved forward as the
 *                    window slides, and Refine-and-Prune started from it.
 *   ewsjf_ring_step  ewsjf_ring_insert + ewsjf_step (one vector) in the same two
 *                    kernels: the streaming scheduler's per-step update and
 *                    admission.
 *   ewsjf_tactical_step  Algorithm 1's own batch rule: the head-of-line score
 *                    of every queue, the ArgMax queue drained oldest first,
 *                    backfill from its neighbours, removal of queues that stay
 *                    empty (Section 3.2).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  * Array arguments are DEVICE pointers (hipMalloc'd or torch CUDA tensors)
 *    owned by the caller, except where marked "host".  Parameter structs are
 *    host memory, read before the call returns.
 *  * Request id = index into the pool arrays (a ring slot in a streaming pool).
 *    A prompt length <= 0 marks an empty slot: it routes to -1, scores NaN and
 *    is never admitted.
 *  * Pool arrays (len, arrival, qid, score) must be 16-byte aligned; they may
 *    be NULL when n == 0.
 *  * All work is enqueued on `stream`; nothing synchronizes the host.  The
 *    library allocates no memory: scratch space is the caller's workspace,
 *    sized by ewsjf_workspace_bytes().  Calls that share a workspace must not
 *    overlap.  Outputs are valid once the stream reaches the call's end.
 *  * Argument checks run on the host before any launch and return a negative
 *    status without touching the device.  Asynchronous faults surface at the
 *    caller's next synchronization.
 *  * Data-dependent conditions are not errors: fewer than B admissible
 *    requests give n_sel < B; window lengths outside [1, max_len] are clamped.
 */
#ifndef EWSJF_H_
#define EWSJF_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  EWSJF_OK = 0,
  EWSJF_ERR_NULL = -1,      /* a required pointer is NULL */
  EWSJF_ERR_ARG = -2,       /* a size or parameter is out of range */
  EWSJF_ERR_WORKSPACE = -3, /* workspace smaller than ewsjf_workspace_bytes() */
  EWSJF_ERR_LAUNCH = -4,    /* the HIP runtime refused a launch or copy */
  EWSJF_ERR_ALIGN = -5,     /* a pool array is not 16-byte aligned */
  EWSJF_ERR_DEVICE = -6     /* no usable gfx950 device is current */
} ewsjf_status;

enum {
  EWSJF_MAX_QUEUES = 256,    /* queue budget cap (the paper's example is 32) */
  EWSJF_MAX_LEN = 32768,     /* cap on the window clamp L */
  EWSJF_MAX_B = 4096,        /* admissions per step per parameter vector */
  EWSJF_MAX_THETA = 1024,    /* parameter vectors per call */
  EWSJF_MAX_DISPATCH = 4096, /* requests per ewsjf_dispatch call */
  EWSJF_TRIAL_STATS = 8,     /* statistics per trial proposal (ewsjf_trial_step) */
  EWSJF_ROUTE_WORDS = EWSJF_MAX_LEN / 32 + 2, /* 64-bit words of the compact routing map */
  EWSJF_STATIC_SCRATCH_BYTES = 4 << 20        /* scratch of ewsjf_step_static, per device */
};

/* Stage-1 initializers (Section 4.2, Stage 1). */
enum {
  EWSJF_INIT_EQUAL_WIDTH = 0, /* K equal-width bins over the window's [min, max] */
  EWSJF_INIT_KMEANS3 = 1      /* exact one-dimensional 3-means (the paper's k=3) */
};

/* Which gaps form G in the Eq. 2 split test. */
enum {
  EWSJF_GAPS_DISTINCT = 0, /* gaps between distinct window values (default) */
  EWSJF_GAPS_MULTISET = 1  /* gaps between consecutive sorted window entries */
};

/* ewsjf_step flags */
enum {
  EWSJF_STEP_TOMBSTONE = 1 /* after selecting, set len[id] = 0 for every admitted id (n_theta == 1) */
};

/* Operations for ewsjf_workspace_bytes(). */
enum { EWSJF_OP_PARTITION = 0, EWSJF_OP_SELECT = 1, EWSJF_OP_STEP = 2, EWSJF_OP_TACTICAL = 3, EWSJF_OP_TRIAL = 4 };

/* Refine-and-Prune parameters (host struct).  Section 4.2: Stage 1 picks the
 * initializer; Stage 2 splits at gaps larger than alpha * mean gap (alpha > 1,
 * Eq. 2) until no such gap remains or the cluster's value span is below
 * min_width; Stage 3 merges adjacent queues with the lowest utility (Eq. 3,
 * eps in the denominator) until at most max_queues remain. */
typedef struct {
  int32_t init_mode;   /* EWSJF_INIT_* */
  int32_t init_queues; /* K for EWSJF_INIT_EQUAL_WIDTH, 1..EWSJF_MAX_LEN */
  int32_t max_queues;  /* 1..EWSJF_MAX_QUEUES */
  int32_t min_width;   /* >= 0 tokens */
  int32_t max_len;     /* L: window lengths are clamped to [1, L]; 1..EWSJF_MAX_LEN */
  int32_t gap_mode;    /* EWSJF_GAPS_* */
  double alpha;        /* significance ratio, > 1 */
  double eps;          /* > 0 */
} ewsjf_partition_params;

/* One scoring parameter vector (device array of n_theta): the meta-policy maps
 * a queue's mean window length mean_q to the three weights of Eq. 1/Eq. 4:
 *   w_base = a_base*mean_q + b_base, w_urg = a_urg*mean_q + b_urg,
 *   w_fair = a_fair*mean_q + b_fair. */
typedef struct {
  float a_base, b_base, a_urg, b_urg, a_fair, b_fair;
} ewsjf_theta;

/* Estimated prefill cost C_prefill(b) = c0 + c1*b + c2*b^2 seconds (host struct).
 * The kernels evaluate it in binary32: c0 must lie in [FLT_MIN, FLT_MAX], c1
 * and c2 must each be 0 or lie in that range, and (b + 1) C_prefill(b) must
 * not exceed 1 / (2 FLT_MIN) (about 4.25e37) for b = 2^31 - 1 (the longest
 * length), which keeps its binary32 reciprocal a normal number; otherwise
 * EWSJF_ERR_ARG. */
typedef struct {
  double c0, c1, c2;
} ewsjf_cost;

/* Queue table: the queue structure of the active policy (Section 3.1).  A
 * fixed-size device blob of ewsjf_queue_table_bytes() bytes written by
 * ewsjf_partition, ewsjf_table_upload or ewsjf_dispatch.  lo/hi/count/sum/mean
 * describe the window lengths that fell in each queue (a bubble queue: its
 * interval and its creating request, see ewsjf_dispatch); mean is the queue's
 * profile used by the meta-policy.  Two routing readings:
 *   gapped == 0  queue i covers prompt lengths [bounds[i-1], bounds[i]) with
 *                queue 0 open below and queue k-1 open above, so the
 *                intervals cover every length exactly once;
 *   gapped == 1  queue i holds [lo_i, hi_i]; a length between queues i and
 *                i+1 goes to queue i when 10 L <= 11 (hi_i + 1), to queue
 *                i+1 when 10 L >= 9 lo_{i+1}, else to the nearer of the two
 *                (L - hi_i against lo_{i+1} - L, ties to i); below the first
 *                queue 0, above the last k-1 (Section 4.3).
 * lut[b] = queue of length b for b in [1, max_len] under that reading
 * (longer lengths belong to queue k-1).  route[] holds the same map in
 * 8 KiB, the form the per-step kernels stage: under either reading the queue
 * of a length never falls and rises by at most one from one length to the
 * next, so word w covers lengths [32 w, 32 w + 32) as the queue of length
 * 32 w - 1 (high 32 bits; 0 for w = 0) and a mask of the lengths where the
 * queue rises by one (low 32 bits): the queue of b in [1, max_len] is
 * (route[b / 32] >> 32) + popcount of the mask bits 0 .. b % 32.  Lengths
 * past max_len keep the queue of max_len.  Both are written with the table. */
typedef struct {
  int32_t k;
  int32_t max_len;
  int32_t n_distinct; /* diagnostics of the last partition (0 after upload) */
  int32_t n_coarse;
  int32_t n_leaves;
  int32_t gapped;     /* routing reading: 0 contiguous bounds, 1 gapped intervals */
  int64_t n_window;
  int32_t bounds[EWSJF_MAX_QUEUES]; /* bounds[i] = lowest length of queue i+1, i < k-1 */
  int32_t lo[EWSJF_MAX_QUEUES];
  int32_t hi[EWSJF_MAX_QUEUES];
  int64_t count[EWSJF_MAX_QUEUES];
  int64_t sum[EWSJF_MAX_QUEUES];
  double mean[EWSJF_MAX_QUEUES];
  uint8_t lut[EWSJF_MAX_LEN + 16];
  uint64_t route[EWSJF_ROUTE_WORDS];
} ewsjf_queue_table;

/* Size in bytes of the device queue table. */
size_t ewsjf_queue_table_bytes(void);

/* Workspace bytes needed by an operation.  `n` is the pool (or window) size;
 * p is read only for EWSJF_OP_PARTITION (may be NULL otherwise); n_theta is
 * ignored for EWSJF_OP_TACTICAL (one parameter vector). */
size_t ewsjf_workspace_bytes(int op, int64_t n, int32_t n_theta, int32_t B, const ewsjf_partition_params* p);

/* Install a queue structure computed elsewhere (for example a policy loaded
 * from storage).  host_table: host struct with k, max_len, gapped, bounds, lo,
 * hi, count, sum, mean filled in (lut and diagnostics are ignored).  Requires
 * 1 <= k <= EWSJF_MAX_QUEUES, 1 <= max_len <= EWSJF_MAX_LEN and bounds strictly
 * increasing within [1, max_len], finite means; gapped is 0 or 1.  With
 * gapped = 1 the intervals [lo_i, hi_i] lie in [1, max_len] in increasing
 * order without overlap; with gapped = 0, lo_i = bounds[i-1] for i >= 1
 * (queue i starts at its bound, as in the tables ewsjf_partition writes).
 * Otherwise EWSJF_ERR_ARG.  The device copy and its
 * routing lut are written on `stream`; this set-up call then synchronizes
 * `stream` so the host struct may be released on return. */
ewsjf_status ewsjf_table_upload(const ewsjf_queue_table* host_table, void* table, hipStream_t stream);

/* Refine-and-Prune (Section 4.2) over window[0..n_window) (device int32,
 * n_window >= 1).  Writes the queue table.  Needs a workspace of
 * ewsjf_workspace_bytes(EWSJF_OP_PARTITION, n_window, 0, 0, p) bytes. */
ewsjf_status ewsjf_partition(const int32_t* window, int64_t n_window, const ewsjf_partition_params* p,
                             void* table, void* ws, size_t ws_bytes, hipStream_t stream);

/* Trials of scoring-parameter proposals: the simulator side of the
 * meta-optimizer (Section 4.4.2), which runs each candidate Theta for a trial
 * interval, collects statistics and scores them with the reward of Eq. 5.
 * Proposal t has its own pool: slots [t * capacity, (t + 1) * capacity) of
 * len/arrival (device [n_pools][capacity], 16-byte aligned, capacity a
 * multiple of 4), and parameter vector theta[t].  One call is one step of the
 * trial for every proposal: the n_new arrivals go into ring slots (pos + i)
 * mod capacity of every pool (the same requests for all: common arrivals),
 * each pool admits its top B under its own vector (as ewsjf_step; ids/top
 * [n_pools][B], n_sel [n_pools]), then the statistics of the admitted
 * requests are added to stats[t] (device double [n_pools][EWSJF_TRIAL_STATS]:
 * 0 admitted, 1 tokens = sum of their prompt lengths, 2 sum and 3 sum of
 * squares of their waits W = max(0, now - arrival) in seconds (a NaN arrival
 * waits 0), 4 largest such wait, 7 steps; entries 5 and 6 belong to
 * ewsjf_trial_finish) and their queues counted in queue_admits (device int64
 * [n_pools][EWSJF_MAX_QUEUES]), and the admitted slots are emptied.  The
 * caller zeroes stats and queue_admits at the trial's start; sums are
 * reduced in a fixed order, so trials are reproducible.  Workspace
 * ewsjf_workspace_bytes(EWSJF_OP_TRIAL, capacity, n_pools, B, NULL).
 * 1 <= n_pools <= EWSJF_MAX_THETA, 0 <= pos < capacity, 0 <= n_new <=
 * capacity, 1 <= B <= EWSJF_MAX_B. */
ewsjf_status ewsjf_trial_step(int32_t* len, float* arrival, int64_t capacity, int32_t n_pools, int64_t pos,
                              const int32_t* new_len, const float* new_arrival, int64_t n_new, float now,
                              const void* table, const ewsjf_theta* theta, const ewsjf_cost* cost, int32_t B,
                              int32_t* ids, float* top, int32_t* n_sel, double* stats, int64_t* queue_admits,
                              void* ws, size_t ws_bytes, hipStream_t stream);

/* The end of a trial: stats[t][5] = pending requests of pool t and
 * stats[t][6] = their largest wait at `now`, and reward[t] (device double
 * [n_pools]) = Eq. 5, R = lambda[0] C + lambda[1] L - lambda[2] S - lambda[3] U
 * (lambda: host double [4]), with the terms read as: C (compact, homogeneous
 * queues) = minus the mean over queues of (hi - lo) / (hi + lo); L (load
 * imbalance) = minus the coefficient of variation of pool t's admissions per
 * queue (0 without admissions); S (queue proliferation) = k /
 * EWSJF_MAX_QUEUES; U (latency) = the mean wait of pool t's admitted requests
 * (0 without admissions). */
ewsjf_status ewsjf_trial_finish(const int32_t* len, const float* arrival, int64_t capacity, int32_t n_pools, float now,
                                const void* table, const int64_t* queue_admits, const double* lambda, double* stats,
                                double* reward, hipStream_t stream);

/* The Dispatcher with on-demand bubble queues (Section 3.2, Dispatcher;
 * Section 4.3 and the appendix's Algorithm 2): the requests with len > 0 join
 * the table's queues one at a time in arrival order (arrival ascending, equal
 * arrivals by index, a NaN arrival last, -0 as +0), each against the queue set
 * the earlier ones left.  The set is read in its gapped form (queue i holds
 * [lo_i, hi_i]; min_len = lo_i, max_len = hi_i + 1).  A length inside a queue
 * joins it; below the first queue it joins queue 0, above the last queue k-1.
 * A length L between queues i and i+1 joins queue i if 10 L <= 11 max_len_i,
 * else queue i+1 if 10 L >= 9 min_len_{i+1}; otherwise it falls in a true gap
 * and, while the set holds fewer than max_queues queues, creates a bubble
 * queue [L - floor(r/2), L - floor(r/2) + r) clipped to [max_len_i,
 * min_len_{i+1}), r = min(bubble_width, min_len_{i+1} - max_len_i), with
 * count 1, sum L and mean L (its creating request is its profile); once the
 * set is full it joins the nearer neighbour (L - hi_i against lo_{i+1} - L,
 * ties to queue i).  qid[i] = request i's queue in the final set (bubbles
 * shift the queues above them), -1 for len[i] <= 0.  The table is rewritten in
 * place in its gapped reading (gapped = 1, bounds[i-1] = lo_i, lut rebuilt)
 * unless it already was gapped and no bubble was created; a later
 * ewsjf_partition replaces the bubbles with a fresh contiguous table.
 * len, qid: device int32 [n]; arrival: device float32 [n];
 * 0 <= n <= EWSJF_MAX_DISPATCH, bubble_width >= 1, 1 <= max_queues <=
 * EWSJF_MAX_QUEUES (a set already holding max_queues or more queues gets no
 * bubbles).  No alignment requirement; one workgroup, no workspace. */
ewsjf_status ewsjf_dispatch(const int32_t* len, const float* arrival, int64_t n, void* table, int32_t bubble_width,
                            int32_t max_queues, int32_t* qid, hipStream_t stream);

/* Dynamic Queue Routing: qid[i] = queue of len[i], or -1 for len[i] <= 0.
 * len, qid: device int32 [n]. */
ewsjf_status ewsjf_route(const int32_t* len, int64_t n, const void* table, int32_t* qid, hipStream_t stream);

/* Density-Weighted Scoring (Eq. 1 / Eq. 4) of every request for every
 * parameter vector:
 *   Phi = qf * (w_base + w_urg * cs + w_fair * ln(b + 1)),
 *   qf = (q + 1) / (b + 1) with q the 0-based queue (so q_i is 1-based),
 *   cs = max(0, now - arrival) / C_prefill(b).
 * len: device int32 [n]; arrival: device float32 [n] seconds; theta: device
 * ewsjf_theta [n_theta]; score: device float32 [n_theta][n].  Empty slots get
 * NaN; a NaN Phi of an occupied slot is stored as -inf.  Computed in binary32;
 * agrees with the binary64 definition to about 1e-6 relative. */
ewsjf_status ewsjf_score(const int32_t* len, const float* arrival, int64_t n, float now, const void* table,
                         const ewsjf_theta* theta, int32_t n_theta, const ewsjf_cost* cost, float* score,
                         hipStream_t stream);

/* Top-B admission over precomputed scores (device float32 [n_theta][n]; NaN
 * = not admissible).  For each parameter vector t: ids[t][0..n_sel[t]) are the
 * admitted request ids in order of (score desc, id asc), top[t][.] their
 * scores; remaining slots get id -1 and score NaN.  ids/top: device [n_theta][B],
 * n_sel: device int32 [n_theta].  1 <= B <= EWSJF_MAX_B. */
ewsjf_status ewsjf_select(const float* score, int64_t n, int32_t n_theta, int32_t B, int32_t* ids, float* top,
                          int32_t* n_sel, void* ws, size_t ws_bytes, hipStream_t stream);

/* One scheduling step: ewsjf_route + ewsjf_score + ewsjf_select fused, reading
 * each request's length and arrival once and never materializing scores.
 * Outputs as for ewsjf_select.  With EWSJF_STEP_TOMBSTONE (n_theta == 1) the
 * admitted slots are emptied (len[id] = 0) on the device after selection. */
ewsjf_status ewsjf_step(int32_t* len, const float* arrival, int64_t n, float now, const void* table,
                        const ewsjf_theta* theta, int32_t n_theta, const ewsjf_cost* cost, int32_t B,
                        int32_t flags, int32_t* ids, float* top, int32_t* n_sel, void* ws, size_t ws_bytes,
                        hipStream_t stream);

/* ewsjf_step that also times its two kernels with four caller-created events
 * (hipEventCreate, timing enabled): marks[0]/marks[1] take the start/end of
 * the streaming kernel (routing, scoring and per-workgroup candidates),
 * marks[2]/marks[3] the start/end of the merge kernel (exact top-B).  For
 * per-phase timing by a monitor; marks == NULL behaves as ewsjf_step. */
ewsjf_status ewsjf_step_timed(int32_t* len, const float* arrival, int64_t n, float now, const void* table,
                              const ewsjf_theta* theta, int32_t n_theta, const ewsjf_cost* cost, int32_t B,
                              int32_t flags, int32_t* ids, float* top, int32_t* n_sel, void* ws, size_t ws_bytes,
                              hipStream_t stream, hipEvent_t* marks);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, serving loops and harnesses that may not call hipMalloc):
 * ewsjf_step with its workspace in a fixed array of
 * EWSJF_STATIC_SCRATCH_BYTES bytes that the library keeps on each device
 * until the process ends, so the call allocates nothing.  Arguments, outputs
 * and rules as for ewsjf_step, without ws/ws_bytes.  A size whose workspace,
 * ewsjf_workspace_bytes(EWSJF_OP_STEP, n, n_theta, B, NULL), exceeds
 * EWSJF_STATIC_SCRATCH_BYTES returns EWSJF_ERR_WORKSPACE before anything is
 * enqueued (one vector: any pool up to 2^31 - 1 requests and any B; several
 * vectors: up to 13 over 4,194,304 requests with B = 1,024, up to 55 over
 * 1,048,576 requests with B = 256).  Every call on a device
 * uses that device's one array: calls that can run at the same time on one
 * device (other streams, other host threads) race and must be serialized by
 * the caller.  No clearing is needed between calls (each call writes every
 * scratch entry it reads).  The first call on a device looks the array up
 * (hipGetSymbolAddress); EWSJF_ERR_LAUNCH if that fails. */
ewsjf_status ewsjf_step_static(int32_t* len, const float* arrival, int64_t n, float now, const void* table,
                               const ewsjf_theta* theta, int32_t n_theta, const ewsjf_cost* cost, int32_t B,
                               int32_t flags, int32_t* ids, float* top, int32_t* n_sel, hipStream_t stream);

/* Streaming pool update: the tactical loop admits from a pool that new
 * requests keep joining (Section 3.2), and the strategic loop partitions a
 * window of the most recent request lengths (Section 3.1; Section 4.2).  One
 * launch writes n new requests into ring slots (pos + i) mod capacity
 * (ring_len, ring_arrival), overwriting whatever those slots held, and their
 * lengths into window slots (wpos + i) mod window_cap.
 * ring_len, ring_arrival: device [capacity]; window: device int32 [window_cap]
 * (may be NULL with window_cap == 0); new_len, new_arrival: device [n].
 * 0 <= pos < capacity, 0 <= wpos < max(window_cap, 1), n <= capacity and
 * n <= window_cap when a window is given; otherwise EWSJF_ERR_ARG.  The new
 * arrays must not overlap the ring or the window.  No alignment requirement. */
ewsjf_status ewsjf_ring_insert(int32_t* ring_len, float* ring_arrival, int64_t capacity, int64_t pos,
                               int32_t* window, int64_t window_cap, int64_t wpos, const int32_t* new_len,
                               const float* new_arrival, int64_t n, hipStream_t stream);

/* Histogram of a window of prompt lengths: hist[b] = number of window
 * entries whose length clamped to [1, max_len] is b (hist[0] = 0).  The
 * partitioner reads the sorted window only through its distinct values and
 * their multiplicities (Section 4.2), which this histogram holds.  The window
 * is ring[(begin + i) mod ring_cap] for i < n: a plain array is (window,
 * n_window, 0, n_window); a window kept as the last n lengths of a ring of
 * recent lengths (the ring calls' window argument) is a range of it.
 * ring: device int32 [ring_cap] (may be NULL when n == 0); hist: device uint32
 * [max_len + 1], written in full.  0 <= n <= ring_cap, 0 <= begin <
 * max(ring_cap, 1), 1 <= max_len <= EWSJF_MAX_LEN; otherwise EWSJF_ERR_ARG. */
ewsjf_status ewsjf_window_histogram(const int32_t* ring, int64_t ring_cap, int64_t begin, int64_t n, int32_t max_len,
                                    uint32_t* hist, hipStream_t stream);

/* The sliding window of the online strategic loop (Section 3.1: the
 * partitioner's input is a window of recent requests) moved forward by n
 * entries, in the histogram: the counts of the n lengths that leave the window,
 * ring[(sub_pos + i) mod ring_cap], move to the n lengths that join it,
 * ring[(add_pos + i) mod ring_cap], i < n (lengths clamped to [1, max_len]).
 * Exact: the result is the histogram of the moved window whatever the order
 * of the updates.  The caller names the entries; both ranges must still hold
 * those lengths (a ring of at least window + n entries keeps them).  ring:
 * device int32 [ring_cap]; hist: device uint32 [max_len + 1].  1 <= ring_cap,
 * 0 <= add_pos, sub_pos < ring_cap, 0 <= n <= ring_cap, 1 <= max_len <=
 * EWSJF_MAX_LEN; otherwise EWSJF_ERR_ARG.  n == 0 does nothing. */
ewsjf_status ewsjf_window_advance(const int32_t* ring, int64_t ring_cap, int64_t add_pos, int64_t sub_pos, int64_t n,
                                  int32_t max_len, uint32_t* hist, hipStream_t stream);

/* Refine-and-Prune (Section 4.2) from a window histogram (device uint32
 * [p->max_len + 1], bin 0 ignored, as ewsjf_window_histogram and
 * ewsjf_window_advance write it): the same queue table, bit for bit, as
 * ewsjf_partition over any window with that histogram; the table's n_window
 * is the histogram's total.  A histogram with no entries gives one queue
 * covering every length with count 0, sum 0, lo = hi = 0 and mean 0.
 * Workspace: ewsjf_workspace_bytes(EWSJF_OP_PARTITION, 0, 0, 0, p) bytes.  The
 * histogram is only read. */
ewsjf_status ewsjf_partition_hist(const uint32_t* hist, const ewsjf_partition_params* p, void* table, void* ws,
                                  size_t ws_bytes, hipStream_t stream);

/* The streaming scheduler's step (Section 3.2: requests keep joining the pool
 * between admissions): the effect of ewsjf_ring_insert(ring_len, ring_arrival,
 * capacity, pos, window, window_cap, wpos, new_len, new_arrival, n_new) followed
 * by ewsjf_step over the ring (n = capacity) with one parameter vector, in the
 * step's two kernels: the streaming kernel substitutes the new requests for the
 * slots it loads and stores them (and their lengths into the window), so there
 * is no separate insert launch.  Arguments and rules as for those two calls
 * (ring arrays 16-byte aligned; workspace ewsjf_workspace_bytes(EWSJF_OP_STEP,
 * capacity, 1, B, NULL)); the new arrays must not overlap the ring or the
 * window.  EWSJF_STEP_TOMBSTONE empties the admitted slots after selection. */
ewsjf_status ewsjf_ring_step(int32_t* ring_len, float* ring_arrival, int64_t capacity, int64_t pos, int32_t* window,
                             int64_t window_cap, int64_t wpos, const int32_t* new_len, const float* new_arrival,
                             int64_t n_new, float now, const void* table, const ewsjf_theta* theta,
                             const ewsjf_cost* cost, int32_t B, int32_t flags, int32_t* ids, float* top,
                             int32_t* n_sel, void* ws, size_t ws_bytes, hipStream_t stream);

/* One step of the tactical loop as Algorithm 1 states it (Section 3.2),
 * over per-queue FIFOs of the pending pool:
 *  1. Score Updater: every non-empty queue's head-of-line request (its oldest:
 *     arrival ascending, equal arrivals by id, a NaN arrival last) is scored
 *     with Phi (Eq. 1 / Eq. 4, binary64 rounded once to binary32) and the
 *     queue's profile; an empty queue's counter empty_cnt[q] goes up by one
 *     (a non-empty step resets it to 0).
 *  2. Batch Builder: the queue with the highest head score (ties: the lower
 *     queue) gives its requests oldest first until B are taken (GreedyFill);
 *     if the batch is not full, its non-empty neighbours q-1 and q+1 backfill
 *     it oldest first, the one with the higher head score first (ties: the
 *     lower queue).
 *  3. RemoveQueue: after the batch is built, queues with empty_cnt >
 *     empty_threshold are removed, lowest index first; each is re-absorbed
 *     by the neighbour whose pair has the lower Eq. 3 utility (eps as in
 *     ewsjf_partition_params; ties: the lower neighbour): the boundary
 *     between them goes, count/sum add, lo/hi span both, mean = sum/count.
 *     The last queue is never removed.  The table (k, bounds, lo, hi, count,
 *     sum, mean, lut) and empty_cnt are rewritten in place on the device.
 * len, arrival: device [n] pool (16-byte aligned); table: device queue table,
 * read and updated; theta: device, one vector; cost: host; empty_cnt: device
 * int32 [EWSJF_MAX_QUEUES], entries [0, k) in use (zero them when a new table
 * is installed); ids: device int32 [B] in batch order (-1 after n_sel);
 * n_sel, q_prim: device int32 [1] (q_prim = -1 when every queue is empty);
 * head_score: device float32 [EWSJF_MAX_QUEUES] or NULL (NaN for empty
 * queues); removed: device int32 [EWSJF_MAX_QUEUES] or NULL (1 for each queue,
 * indexed as at the start of the step, removed by this step).
 * flags: 0 or EWSJF_STEP_TOMBSTONE (empty the admitted slots).  Workspace:
 * ewsjf_workspace_bytes(EWSJF_OP_TACTICAL, n, 1, B, NULL).  1 <= B <=
 * EWSJF_MAX_B, empty_threshold >= 0, eps > 0, otherwise EWSJF_ERR_ARG. */
ewsjf_status ewsjf_tactical_step(int32_t* len, const float* arrival, int64_t n, float now, void* table,
                                 const ewsjf_theta* theta, const ewsjf_cost* cost, int32_t B, int32_t empty_threshold,
                                 int32_t* empty_cnt, double eps, int32_t flags, int32_t* ids, int32_t* n_sel,
                                 int32_t* q_prim, float* head_score, int32_t* removed, void* ws, size_t ws_bytes,
                                 hipStream_t stream);

/* Human-readable name of a status code (static storage). */
const char* ewsjf_status_string(ewsjf_status s);

/* Library version (major * 10000 + minor * 100 + patch). */
int32_t ewsjf_version(void);

#ifdef __cplusplus
}
#endif

#endif /* EWSJF_H_ */
