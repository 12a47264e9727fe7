"""Pins for the oracle's tactical step (Algorithm 1, Section 3.2): a hand
derivation, the FCFS limit, brute-force re-derivations of the batch from the
pinned routing and scoring functions, the empty-threshold rule and the Eq. 3
re-absorption, each independent of the oracle's own loop."""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
from paper_2601_21758_amd import workloads as W

GOLD = os.path.join(os.path.dirname(__file__), "golden")
COST = (0.01, 1e-4, 0.0)
MID = W.THETA_MID


def gold(name):
    with open(os.path.join(GOLD, name)) as f:
        return json.load(f)


def table_of(d):
    cnt = np.asarray(d["count"], np.int64)
    s = np.asarray(d["sum"], np.int64)
    return oracle.Table(int(d["k"]), np.asarray(d["bounds"], np.int32), cnt, s, np.asarray(d["lo"], np.int32),
                        np.asarray(d["hi"], np.int32), s.astype(np.float64) / cnt.astype(np.float64))


def assert_table(t, d):
    assert t.k == d["k"]
    assert t.bounds.tolist() == d["bounds"]
    assert t.count.tolist() == d["count"] and t.sum.tolist() == d["sum"]
    assert t.lo.tolist() == d["lo"] and t.hi.tolist() == d["hi"]
    assert t.mean.tolist() == [s / c for s, c in zip(d["sum"], d["count"])]


def within_one_f32_ulp(got, exact):
    e = np.float32(exact)
    return abs(float(got) - exact) <= float(np.spacing(np.abs(e)))


def test_we5_three_hand_derived_steps():
    g = gold("we5_tactical.json")
    t, ec = None, None
    for st in g["steps"]:
        if t is None or st.get("fresh_table"):
            t, ec = table_of(g["table"]), np.zeros(g["table"]["k"], np.int32)
        r = oracle.tactical_step(st["len"], st["arrival"], g["now"], t, ec, g["theta"], st["B"], g["empty_threshold"],
                                 g["cost"])
        assert r.ids.tolist() == st["expected_ids"], st["name"]
        assert r.q_prim == st["expected_q_prim"]
        for got, want in zip(r.head_score, st["expected_head_score"]):
            if want is None:
                assert np.isnan(got)
            else:
                assert within_one_f32_ulp(got, want), (got, want)
        assert r.removed.tolist() == st["expected_removed"]
        assert_table(r.table, st["expected_table"])
        assert r.empty_cnt.tolist() == st["expected_empty_cnt"]
        t, ec = r.table, r.empty_cnt


def fifo_order(ids, arrival):
    """Ids in queue order: arrival ascending (NaN as +inf, -0 as +0), then id."""
    a = np.asarray(arrival, np.float64)[ids]
    a = np.where(np.isnan(a), np.inf, a) + 0.0
    return ids[np.lexsort((ids, a))]


def test_fcfs_limit_single_queue_takes_the_oldest():
    rng = np.random.default_rng(5)
    n = 3000
    length = rng.integers(-3, 500, n).astype(np.int32)
    arrival = rng.integers(0, 400, n).astype(np.float32)  # many equal arrivals
    arrival[::97] = np.nan
    t = oracle.partition(np.maximum(length, 1), init_queues=1, max_queues=1)
    assert t.k == 1
    valid = np.flatnonzero(length > 0)
    for B in (1, 17, 256, valid.size, valid.size + 5):
        r = oracle.tactical_step(length, arrival, 500.0, t, np.zeros(1, np.int32), MID, B, 3, COST)
        assert r.q_prim == 0
        assert r.ids.tolist() == fifo_order(valid, arrival)[:B].tolist()


def rederive(length, arrival, now, t, theta, B):
    """The batch of Algorithm 1 from the pinned routing and scoring functions."""
    q = oracle.route(length, t)
    sc = oracle.score(length, arrival, now, t, theta, COST)[0]
    fifos = [fifo_order(np.flatnonzero(q == j), arrival) for j in range(t.k)]
    heads = np.array([sc[f[0]] if f.size else np.nan for f in fifos], np.float32)
    nonempty = [j for j in range(t.k) if fifos[j].size]
    if not nonempty:
        return [], -1, heads
    prim = max(nonempty, key=lambda j: (heads[j], -j))
    batch = fifos[prim][:B].tolist()
    adj = [j for j in (prim - 1, prim + 1) if 0 <= j < t.k and fifos[j].size]
    adj.sort(key=lambda j: (-heads[j], j))
    for j in adj:
        batch += fifos[j][:B - len(batch)].tolist()
    return batch, prim, heads


@pytest.mark.parametrize("cfg", [0, 1])
def test_batch_matches_rederivation_on_workloads(cfg):
    p = W.config(cfg)
    t = oracle.partition(p.window, init_queues=p.init_queues, max_queues=p.max_queues)
    rng = np.random.default_rng(cfg)
    n = min(p.length.size, 20000)
    length, arrival = p.length[:n].copy(), p.arrival[:n].copy()
    for B in (1, 64, 4096):
        # thin the pool so that some queues run short and backfill is needed
        keep = rng.random(n) < (0.02 if B == 4096 else 1.0)
        L = np.where(keep, length, 0).astype(np.int32)
        r = oracle.tactical_step(L, arrival, p.now, t, np.zeros(t.k, np.int32), MID, B, 5, COST)
        batch, prim, heads = rederive(L, arrival, p.now, t, MID, B)
        assert r.ids.tolist() == batch
        assert r.q_prim == prim
        np.testing.assert_array_equal(r.head_score, heads)


def test_backfill_order_and_partial_batch():
    # Three queues; only the primary and its upper neighbour hold requests.
    t = table_of({"k": 3, "bounds": [100, 1000], "count": [10, 10, 2], "sum": [55, 1045, 2001], "lo": [1, 100, 1000],
                  "hi": [10, 109, 1001]})
    L = np.array([150, 120, 2000, 0], np.int32)
    A = np.array([0.0, 10.0, 5.0, 0.0], np.float32)
    r = oracle.tactical_step(L, A, 60.0, t, np.zeros(3, np.int32), (0, 1, 0, 1, 0, 1), 10, 9, COST)
    assert r.q_prim == 1
    assert r.ids.tolist() == [0, 1, 2]  # q1 oldest first, then q2; q0 is empty; the batch stays partial
    assert np.isnan(r.head_score[0]) and r.empty_cnt.tolist() == [1, 0, 0]


def test_backfill_takes_the_higher_scoring_neighbour_first():
    t = table_of({"k": 3, "bounds": [100, 1000], "count": [10, 10, 2], "sum": [55, 1045, 2001], "lo": [1, 100, 1000],
                  "hi": [10, 109, 1001]})
    # heads (all weights 1, now = 60): q1 id0 b=100 W=60 -> 59.5; q2 id2 b=1000 W=60 -> 1.66;
    # q0 id1 b=9 W=0 -> (1/10)(1 + ln 10) = 0.33.  The upper neighbour drains first.
    L = np.array([100, 9, 1000, 5, 2000], np.int32)
    A = np.array([0.0, 60.0, 0.0, 60.0, 1.0], np.float32)
    r = oracle.tactical_step(L, A, 60.0, t, np.zeros(3, np.int32), (0, 1, 0, 1, 0, 1), 4, 9, COST)
    assert r.q_prim == 1
    assert r.head_score[2] > r.head_score[0]
    assert r.ids.tolist() == [0, 2, 4, 1]


def test_argmax_ties_go_to_the_lower_queue():
    t = table_of({"k": 3, "bounds": [100, 1000], "count": [10, 10, 2], "sum": [55, 1045, 2001], "lo": [1, 100, 1000],
                  "hi": [10, 109, 1001]})
    # all weights zero: every head scores exactly 0
    L = np.array([2000, 150], np.int32)
    A = np.array([0.0, 5.0], np.float32)
    r = oracle.tactical_step(L, A, 60.0, t, np.zeros(3, np.int32), (0, 0, 0, 0, 0, 0), 1, 9, COST)
    assert r.head_score[1] == r.head_score[2] == 0.0
    assert r.q_prim == 1 and r.ids.tolist() == [1]


def test_empty_threshold_counts_consecutive_steps_and_resets():
    t = table_of({"k": 3, "bounds": [100, 1000], "count": [10, 10, 2], "sum": [55, 1045, 2001], "lo": [1, 100, 1000],
                  "hi": [10, 109, 1001]})
    ec = np.zeros(3, np.int32)
    only_q1 = (np.array([150], np.int32), np.array([0.0], np.float32))
    all_q = (np.array([5, 150, 2000], np.int32), np.array([0.0, 0.0, 0.0], np.float32))
    T = 2
    # q0 and q2 are empty for T steps: counted, not removed
    for s in range(T):
        r = oracle.tactical_step(*only_q1, 60.0, t, ec, MID, 4, T, COST)
        assert not r.removed.any() and r.empty_cnt.tolist() == [s + 1, 0, s + 1]
        t, ec = r.table, r.empty_cnt
    # one non-empty step resets both counters
    r = oracle.tactical_step(*all_q, 60.0, t, ec, MID, 4, T, COST)
    assert r.empty_cnt.tolist() == [0, 0, 0]
    t, ec = r.table, r.empty_cnt
    for s in range(T):
        r = oracle.tactical_step(*only_q1, 60.0, t, ec, MID, 4, T, COST)
        t, ec = r.table, r.empty_cnt
        assert t.k == 3
    # the (T+1)-th consecutive empty step removes both; q1 absorbs q0, then the merged queue absorbs q2
    r = oracle.tactical_step(*only_q1, 60.0, t, ec, MID, 4, T, COST)
    assert r.removed.tolist() == [True, False, True]
    assert r.table.k == 1 and r.table.bounds.size == 0
    assert r.table.count.tolist() == [22] and r.table.sum.tolist() == [3101]
    assert r.table.lo.tolist() == [1] and r.table.hi.tolist() == [1001]
    assert r.empty_cnt.tolist() == [0]
    # the last queue is never removed
    r2 = oracle.tactical_step(np.zeros(4, np.int32), np.zeros(4, np.float32), 60.0, r.table, np.array([9], np.int32),
                              MID, 4, 0, COST)
    assert r2.table.k == 1 and r2.q_prim == -1 and r2.ids.size == 0 and r2.empty_cnt.tolist() == [10]


def utility_exact(a, b, eps=Fraction(1, 10**6)):
    # Eq. 3 in exact rationals; eps = 1e-6 is not exactly representable but
    # only orders utilities that differ by far more than its rounding.
    ra = Fraction(int(a[0]), int(a[3]) - int(a[2]) + 1)
    rb = Fraction(int(b[0]), int(b[3]) - int(b[2]) + 1)
    ma, mb = Fraction(int(a[1]), int(a[0])), Fraction(int(b[1]), int(b[0]))
    return (ra + rb) / (abs(mb - ma) + eps)


@pytest.mark.parametrize("seed", range(6))
def test_removed_queue_goes_to_lower_utility_neighbour(seed):
    p = W.config(1)
    t = oracle.partition(p.window, init_queues=p.init_queues, max_queues=p.max_queues)
    rng = np.random.default_rng(seed)
    r_q = int(rng.integers(1, t.k - 1))  # a middle queue
    # pool: one request in every queue but r_q (its own lo length routes to it)
    L = np.array([t.lo[j] for j in range(t.k) if j != r_q], np.int32)
    A = np.zeros(L.size, np.float32)
    r = oracle.tactical_step(L, A, 10.0, t, np.zeros(t.k, np.int32), MID, 1, 0, COST)
    assert r.removed.tolist() == [j == r_q for j in range(t.k)]
    Q = [(t.count[j], t.sum[j], t.lo[j], t.hi[j]) for j in range(t.k)]
    to_lower = utility_exact(Q[r_q - 1], Q[r_q]) <= utility_exact(Q[r_q], Q[r_q + 1])
    a = r_q - 1 if to_lower else r_q + 1
    n2 = r.table
    j = r_q - 1 if to_lower else r_q  # index of the merged queue after the removal
    assert n2.k == t.k - 1
    assert n2.count[j] == t.count[a] + t.count[r_q] and n2.sum[j] == t.sum[a] + t.sum[r_q]
    assert n2.lo[j] == min(t.lo[a], t.lo[r_q]) and n2.hi[j] == max(t.hi[a], t.hi[r_q])
    # invariants of the queue table
    assert n2.count.sum() == t.count.sum() and n2.sum.sum() == t.sum.sum()
    assert np.all(np.diff(n2.bounds) > 0) and n2.bounds.tolist() == n2.lo[1:].tolist()
    assert n2.mean.tolist() == (n2.sum / n2.count).tolist()


@pytest.mark.parametrize("s3,to_lower", [(3200, True), (3900, False)])
def test_removal_deletes_the_shared_boundary(s3, to_lower):
    # Reading T6: the removed queue's boundary with its absorber goes; the
    # other bounds stay where they were.  The window extremes lo/hi sit
    # inside the routing intervals here (lo != the bounds), so a rule that
    # rebuilt the bounds from lo would give other bounds.
    t = table_of({"k": 4, "bounds": [100, 200, 300], "count": [10, 10, 10, 10], "sum": [500, 1500, 2600, s3],
                  "lo": [1, 120, 230, 310], "hi": [90, 180, 290, 400]})
    Q = [(t.count[j], t.sum[j], t.lo[j], t.hi[j]) for j in range(4)]
    assert (utility_exact(Q[1], Q[2]) <= utility_exact(Q[2], Q[3])) == to_lower
    # one request in queues 0, 1 and 3 (routed by the bounds); queue 2 is empty
    L = np.array([50, 150, 350], np.int32)
    r = oracle.tactical_step(L, np.zeros(3, np.float32), 60.0, t, np.zeros(4, np.int32), MID, 3, 0, COST)
    assert r.removed.tolist() == [False, False, True, False]
    n2 = r.table
    assert n2.bounds.tolist() == ([100, 300] if to_lower else [100, 200])
    j = 1 if to_lower else 2  # the merged queue
    a = 1 if to_lower else 3
    assert n2.count[j] == 20 and n2.sum[j] == t.sum[a] + t.sum[2]
    assert n2.lo[j] == min(t.lo[a], t.lo[2]) and n2.hi[j] == max(t.hi[a], t.hi[2])
    # routing of the merged set by the remaining bounds: 250 joins the absorber
    assert oracle.route(np.array([250], np.int32), n2)[0] == j


def test_batch_invariant_under_pool_permutation():
    p = W.config(0)
    t = oracle.partition(p.window, init_queues=p.init_queues, max_queues=p.max_queues)
    rng = np.random.default_rng(3)
    arrival = rng.permutation(p.length.size).astype(np.float32)  # distinct arrivals
    perm = rng.permutation(p.length.size)
    r1 = oracle.tactical_step(p.length, arrival, 1e4, t, np.zeros(t.k, np.int32), MID, 100, 1, COST)
    r2 = oracle.tactical_step(p.length[perm], arrival[perm], 1e4, t, np.zeros(t.k, np.int32), MID, 100, 1, COST)
    assert r1.q_prim == r2.q_prim
    assert list(zip(p.length[r1.ids], arrival[r1.ids])) == list(zip(p.length[perm][r2.ids], arrival[perm][r2.ids]))


def test_tactical_arguments_rejected():
    t = table_of({"k": 1, "bounds": [], "count": [1], "sum": [1], "lo": [1], "hi": [1]})
    with pytest.raises(ValueError):
        oracle.tactical_step([1], [0.0], 1.0, t, np.zeros(1, np.int32), MID, -1, 0)
    with pytest.raises(ValueError):
        oracle.tactical_step([1], [0.0], 1.0, t, np.zeros(1, np.int32), MID, 1, -1)
    with pytest.raises(ValueError):
        oracle.tactical_step([1], [0.0], 1.0, t, np.zeros(2, np.int32), MID, 1, 0)
