"""Pins of the oracle's Dispatcher with on-demand bubble queues (Algorithm 2,
Section 4.3): the hand-derived worked example WE-6, the routing of lengths
that are not dispatched, closed-form special cases, invariants of the queue
set after dispatch, and agreement with an independent formulation of the
same process (rounds in which the earliest request not yet covered creates
the next bubble of its gap)."""
import json
import math
import os

import numpy as np
import pytest

import oracle

HERE = os.path.dirname(os.path.abspath(__file__))
WE6 = json.load(open(os.path.join(HERE, "golden", "we6_bubble.json")))


def table_of(d, gapped=False):
    k = d["k"]
    lo = np.asarray(d["lo"], np.int32)
    count = np.asarray(d["count"], np.int64)
    ssum = np.asarray(d["sum"], np.int64)
    return oracle.Table(k, lo[1:].copy(), count, ssum, lo, np.asarray(d["hi"], np.int32),
                        ssum.astype(np.float64) / count, gapped=gapped)


def arrivals(a):
    return np.array([math.nan if x == "nan" else x for x in a], np.float32)


def check_table(t, d):
    assert t.k == d["k"]
    assert t.bounds.tolist() == d.get("bounds", d["lo"][1:])
    assert t.lo.tolist() == d["lo"] and t.hi.tolist() == d["hi"]
    assert t.count.tolist() == d["count"] and t.sum.tolist() == d["sum"]
    if "mean" in d:
        assert t.mean.tolist() == d["mean"]
    assert t.gapped


@pytest.mark.parametrize("sc", WE6["scenarios"], ids=[s["name"] for s in WE6["scenarios"]])
def test_we6_dispatch(sc):
    qid, t = oracle.dispatch(np.asarray(WE6["len"], np.int32), arrivals(sc["arrival"]), table_of(WE6["table"]),
                             WE6["bubble_width"], sc["max_queues"])
    assert qid.tolist() == sc["expected_qid"]
    check_table(t, sc["expected_table"])


def test_we6_routing_without_dispatch():
    base = WE6["scenarios"][0]
    t = table_of(base["expected_table"], gapped=True)
    r = WE6["routing"]
    assert oracle.route(np.asarray(r["len"], np.int32), t).tolist() == r["expected"]


def test_we6_nearer_neighbour_tie_goes_low():
    tie = WE6["tie"]
    t = table_of(tie["table"], gapped=True)
    assert oracle.route(np.asarray(tie["len"], np.int32), t).tolist() == tie["expected"]


# --- special cases ---------------------------------------------------------------

def gapped_base(rng, k=12, L=32768):
    """k queues with random gaps between them (intervals [lo, hi] in order)."""
    edges = np.sort(rng.choice(np.arange(2, L), 2 * k, replace=False))
    lo, hi = edges[0::2].astype(np.int32), edges[1::2].astype(np.int32)
    count = rng.integers(1, 1000, k).astype(np.int64)
    ssum = np.array([c * ((a + b) // 2) for c, a, b in zip(count, lo, hi)], np.int64)
    return oracle.Table(k, lo[1:].copy(), count, ssum, lo, hi, ssum.astype(np.float64) / count)


def requests(rng, n, L=32768, ties=False):
    length = rng.integers(-5, L + 50, n).astype(np.int32)
    arrival = (rng.integers(0, 40, n) if ties else rng.random(n) * 100).astype(np.float32)
    arrival[rng.random(n) < 0.02] = np.nan
    return length, arrival


def test_full_set_means_routing_without_dispatch():
    rng = np.random.default_rng(1)
    t = gapped_base(rng)
    length, arrival = requests(rng, 3000)
    qid, t2 = oracle.dispatch(length, arrival, t, 64, t.k)
    assert t2.k == t.k
    t.gapped = True
    assert np.array_equal(qid, oracle.route(length, t))


def test_width_one_bubbles_hold_their_creator_only():
    rng = np.random.default_rng(2)
    t = gapped_base(rng, k=5)
    length, arrival = requests(rng, 400)
    qid, t2 = oracle.dispatch(length, arrival, t, 1, 256)
    orig = set(zip(t.lo.tolist(), t.hi.tolist()))
    bubbles = [q for q in range(t2.k) if (t2.lo[q], t2.hi[q]) not in orig]
    assert bubbles
    for q in bubbles:
        assert t2.lo[q] == t2.hi[q] == t2.sum[q] and t2.count[q] == 1
        # the first request of that length created it and every later one lands inside
        assert np.all(qid[length == t2.lo[q]] == q)


def test_wide_bubbles_reach_a_neighbour():
    # a bubble as wide as its gap, centred on its creator and clipped to the
    # gap, reaches the queue on at least one side; a creator at the gap's
    # middle gets the whole gap
    rng = np.random.default_rng(3)
    t = gapped_base(rng, k=8)
    length, arrival = requests(rng, 2000)
    qid, t2 = oracle.dispatch(length, arrival, t, 1 << 20, 256)
    orig = list(zip(t.lo.tolist(), t.hi.tolist()))
    n_bubbles = 0
    for q in range(t2.k):
        if (t2.lo[q], t2.hi[q]) in orig:
            continue
        n_bubbles += 1
        assert t2.lo[q] == t2.hi[q - 1] + 1 or t2.hi[q] == t2.lo[q + 1] - 1
    assert n_bubbles > 0
    mid = oracle.Table(2, np.array([300], np.int32), np.array([1, 1], np.int64), np.array([100, 300], np.int64),
                       np.array([100, 300], np.int32), np.array([100, 300], np.int32), np.array([100.0, 300.0]))
    _, t3 = oracle.dispatch(np.array([200], np.int32), np.zeros(1, np.float32), mid, 1 << 20, 8)
    # available = 300 - 101 = 199, [200 - 99, 200 + 100) = [101, 300): the whole gap
    assert t3.lo.tolist() == [100, 101, 300] and t3.hi.tolist() == [100, 299, 300]
    # off-centre (a true gap: 2600 > 11 * 101 and 2600 < 9 * 300):
    # [260 - 99, 260 + 100) = [161, 360) clipped to [161, 300)
    _, t4 = oracle.dispatch(np.array([260], np.int32), np.zeros(1, np.float32), mid, 1 << 20, 8)
    assert t4.lo.tolist() == [100, 161, 300] and t4.hi.tolist() == [100, 299, 300]
    # width 50: [260 - 25, 260 + 25) = [235, 285)
    _, t5 = oracle.dispatch(np.array([260], np.int32), np.zeros(1, np.float32), mid, 50, 8)
    assert t5.lo.tolist() == [100, 235, 300] and t5.hi.tolist() == [100, 284, 300]
    # 280 is within the upper tolerance (2800 >= 2700): no bubble
    q6, t6 = oracle.dispatch(np.array([280], np.int32), np.zeros(1, np.float32), mid, 50, 8)
    assert t6.k == 2 and q6.tolist() == [1]


def test_no_true_gap_requests_leave_the_set_alone():
    rng = np.random.default_rng(4)
    t = gapped_base(rng, k=6)
    t.gapped = True
    inside = np.concatenate([rng.integers(a, b + 1, 50) for a, b in zip(t.lo, t.hi)]).astype(np.int32)
    qid, t2 = oracle.dispatch(inside, rng.random(inside.size).astype(np.float32), t, 64, 256)
    assert t2.k == t.k and np.array_equal(t2.lo, t.lo) and np.array_equal(t2.hi, t.hi)
    assert np.array_equal(qid, oracle.route(inside, t))


def test_only_arrival_order_matters():
    # relabelling requests (same arrivals) permutes the result; equal arrivals
    # are taken in id order
    rng = np.random.default_rng(5)
    t = gapped_base(rng, k=6)
    length, arrival = requests(rng, 600)
    qid, t2 = oracle.dispatch(length, arrival, t, 48, 40)
    order = np.lexsort((np.arange(length.size), np.where(np.isnan(arrival), np.inf, arrival)))
    perm = np.empty_like(order)
    perm[order] = np.arange(order.size)
    # new id of request i = its place in arrival order, with arrivals made strictly increasing
    l2 = np.empty_like(length)
    l2[perm] = length
    a2 = np.arange(length.size, dtype=np.float32)
    q2, t3 = oracle.dispatch(l2, a2, t, 48, 40)
    assert np.array_equal(q2[perm], qid)
    assert np.array_equal(t3.lo, t2.lo) and np.array_equal(t3.hi, t2.hi)


# --- invariants ---------------------------------------------------------------------

@pytest.mark.parametrize("seed", range(6))
def test_dispatch_invariants(seed):
    rng = np.random.default_rng(10 + seed)
    t = gapped_base(rng, k=int(rng.integers(1, 20)))
    length, arrival = requests(rng, int(rng.integers(1, 3000)), ties=seed % 2 == 0)
    width = int(rng.choice([1, 7, 64, 500]))
    mq = int(rng.integers(t.k, 257))
    qid, t2 = oracle.dispatch(length, arrival, t, width, mq)
    # the set stays in length order, disjoint, within the cap
    assert t.k <= t2.k <= mq
    assert np.all(t2.lo <= t2.hi) and np.all(t2.hi[:-1] < t2.lo[1:])
    assert np.array_equal(t2.bounds, t2.lo[1:])
    # the original queues are untouched and in order
    orig = {(a, b): (c, s) for a, b, c, s in zip(t.lo, t.hi, t.count, t.sum)}
    kept = [q for q in range(t2.k) if (t2.lo[q], t2.hi[q]) in orig]
    assert len(kept) == t.k
    for q in kept:
        assert (t2.count[q], t2.sum[q]) == orig[(t2.lo[q], t2.hi[q])]
    # every bubble sits in a gap of the original set, holds its creator, is at
    # most `width` wide and has the creator's profile
    for q in range(t2.k):
        if (t2.lo[q], t2.hi[q]) in orig:
            continue
        j = np.searchsorted(t.lo, t2.lo[q]) - 1
        assert 0 <= j < t.k - 1 and t.hi[j] < t2.lo[q] and t2.hi[q] < t.lo[j + 1]
        assert t2.count[q] == 1 and t2.lo[q] <= t2.sum[q] <= t2.hi[q] and t2.mean[q] == t2.sum[q]
        assert t2.hi[q] - t2.lo[q] + 1 <= width
        assert np.any(qid[length == t2.sum[q]] == q)
    # empty slots are not dispatched; everything else has a queue
    assert np.all((qid == -1) == (length <= 0))


# --- an independent formulation -------------------------------------------------------

def rounds_dispatch(length, arrival, t, width, max_queues):
    """The same process computed another way.  A request is covered by a
    queue set when it lies in a queue, below the first or above the last, or
    within Algorithm 2's tolerance of the queues around it; coverage only
    grows as bubbles are added, so the sequential process creates its
    bubbles in the order 'earliest request not covered by the bubbles so
    far'.  With a cap, only the first max_queues - k of them exist; each
    request is then routed against the bubbles whose creator came before
    it."""
    n = length.size
    key = np.where(np.isnan(arrival), np.inf, arrival.astype(np.float64))
    order = [i for i in np.lexsort((np.arange(n), key)) if length[i] > 0]
    base = [(int(a), int(b)) for a, b in zip(t.lo, t.hi)]

    def where(L, ivs):
        """('in', q) | ('tol', q) | ('gap', i) for L against the sorted intervals."""
        i = -1
        for q, (a, b) in enumerate(ivs):
            if a <= L:
                i = q
        if i < 0:
            return "in", 0
        if L <= ivs[i][1] or i == len(ivs) - 1:
            return "in", i
        if 10 * L <= 11 * (ivs[i][1] + 1):
            return "tol", i
        if 10 * L >= 9 * ivs[i + 1][0]:
            return "tol", i + 1
        return "gap", i

    creators = []  # (request, interval) in creation order
    ivs = list(base)
    while True:
        first = next((r for r in order if where(int(length[r]), ivs)[0] == "gap"), None)
        if first is None:
            break
        L = int(length[first])
        _, i = where(L, ivs)
        mx, mn = ivs[i][1] + 1, ivs[i + 1][0]
        rng_ = min(width, mn - mx)
        a, b = max(L - rng_ // 2, mx), min(L - rng_ // 2 + rng_, mn)
        creators.append((first, (a, b - 1)))
        ivs = sorted(ivs + [(a, b - 1)])
    creators = creators[:max_queues - t.k]
    made = {r: iv for r, iv in creators}
    final = sorted(base + [iv for _, iv in creators])
    place = {iv: q for q, iv in enumerate(final)}
    rank = {r: p for p, r in enumerate(order)}
    qid = np.full(n, -1, np.int32)
    for r in order:
        L = int(length[r])
        if r in made:
            qid[r] = place[made[r]]
            continue
        ivs = sorted(base + [iv for c, iv in creators if rank[c] < rank[r]])
        kind, q = where(L, ivs)
        if kind == "gap":  # the cap bound before this request: the nearer neighbour
            q = q if L - ivs[q][1] <= ivs[q + 1][0] - L else q + 1
        qid[r] = place[ivs[q]]
    return qid, final


@pytest.mark.parametrize("seed", range(8))
def test_dispatch_equals_the_rounds_formulation(seed):
    rng = np.random.default_rng(100 + seed)
    t = gapped_base(rng, k=int(rng.integers(2, 9)), L=3000)
    length, arrival = requests(rng, int(rng.integers(50, 400)), L=3000, ties=seed % 3 == 0)
    width = int(rng.choice([1, 5, 40, 300]))
    mq = int(rng.integers(t.k, t.k + 30))
    qid, t2 = oracle.dispatch(length, arrival, t, width, mq)
    rq, final = rounds_dispatch(length, arrival, t, width, mq)
    assert [(int(a), int(b)) for a, b in zip(t2.lo, t2.hi)] == final
    assert np.array_equal(qid, rq)
