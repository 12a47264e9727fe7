"""Pins of the trial oracle (the simulator side of the meta-optimizer,
Section 4.4.2) and of the Eq. 5 reward under its readings: the FCFS limit
recomputed by sorting, a draining trial in closed form, a hand-computed
reward, and the symmetries of common arrivals."""
import math

import numpy as np

import oracle
from oracle import trial as T

COST = (0.01, 1e-4, 0.0)
FCFS_THETA = (0.0, 0.0, 0.0, 1.0, 0.0, 0.0)  # w_base = w_fair = 0, w_urg = 1


def one_queue(L=32768):
    return oracle.Table(1, np.zeros(0, np.int32), np.array([1], np.int64), np.array([100], np.int64),
                        np.array([100], np.int32), np.array([100], np.int32), np.array([100.0]))


def test_fcfs_limit_by_sorting():
    # all lengths equal and one queue: Phi grows with the wait alone, so every
    # step admits the B oldest pending requests (equal arrivals by slot)
    rng = np.random.default_rng(1)
    cap, B, steps, per = 2000, 37, 12, 50
    length = np.where(rng.random(cap) < 0.7, 100, 0).astype(np.int32)
    arrival = rng.integers(0, 300, cap).astype(np.float32)
    batches = []
    for s in range(steps):
        batches.append((np.full(per, 100, np.int32), (300 + 10 * s + rng.integers(0, 10, per)).astype(np.float32),
                        float(310 + 10 * s)))
    stats, qad, hist = T.trial(length, arrival, one_queue(), [FCFS_THETA], batches, B, COST)
    # the same trial by sorting
    L, A = length.copy(), arrival.copy()
    adm_all, pos = [], 0
    for s, (nl, na, now) in enumerate(batches):
        slots = (pos + np.arange(per)) % cap
        L[slots], A[slots] = nl, na
        pos = (pos + per) % cap
        live = np.flatnonzero(L > 0)
        order = live[np.lexsort((live, A[live]))][:B]
        assert np.array_equal(np.sort(hist[s][0]), np.sort(order)), f"step {s}"
        adm_all.append((order.copy(), A[order].astype(np.float64), now))
        L[order] = 0
    waits = np.concatenate([np.maximum(0.0, np.float64(np.float32(now)) - a) for _, a, now in adm_all])
    n = sum(len(o) for o, _, _ in adm_all)
    assert stats[0, 0] == n and stats[0, 1] == 100 * n
    assert math.isclose(stats[0, 2], waits.sum(), rel_tol=1e-12)
    assert math.isclose(stats[0, 3], (waits ** 2).sum(), rel_tol=1e-12)
    assert stats[0, 4] == waits.max()
    assert stats[0, 5] == int((L > 0).sum()) and stats[0, 7] == steps
    last_now = np.float64(np.float32(batches[-1][2]))
    assert stats[0, 6] == np.max(np.maximum(0.0, last_now - A[L > 0].astype(np.float64)))
    assert qad[0, 0] == n


def test_draining_trial_in_closed_form():
    # B above the pool and no arrivals: the first step admits every pending
    # request, the rest admit nothing
    rng = np.random.default_rng(2)
    cap = 500
    length = np.where(rng.random(cap) < 0.5, rng.integers(1, 5000, cap), 0).astype(np.int32)
    arrival = (rng.random(cap) * 20).astype(np.float32)
    arrival[::37] = np.nan
    t = oracle.partition(length[length > 0], init_queues=4, max_queues=4)
    empty = (np.zeros(0, np.int32), np.zeros(0, np.float32))
    stats, qad, _ = T.trial(length, arrival, t, [FCFS_THETA, (1, 2, 3, 4, 5, 6)],
                            [(*empty, 30.0), (*empty, 31.0), (*empty, 32.0)], 1000, COST)
    live = length > 0
    w = np.maximum(0.0, np.float64(np.float32(30.0)) - arrival[live].astype(np.float64))
    w[np.isnan(w)] = 0.0
    for p in range(2):
        assert stats[p, 0] == live.sum() and stats[p, 1] == length[live].astype(np.int64).sum()
        assert math.isclose(stats[p, 2], math.fsum(w), rel_tol=1e-15) and stats[p, 4] == w.max()
        assert stats[p, 5] == 0 and stats[p, 6] == 0 and stats[p, 7] == 3
        assert np.array_equal(qad[p], np.bincount(oracle.route(length[live], t), minlength=t.k))


def test_reward_by_hand():
    # two queues [10, 20] and [100, 300]; proposal 0 admitted 3 + 1 requests
    # with waits summing to 8 s; proposal 1 admitted nothing
    t = oracle.Table(2, np.array([100], np.int32), np.array([5, 5], np.int64), np.array([75, 1000], np.int64),
                     np.array([10, 100], np.int32), np.array([20, 300], np.int32), np.array([15.0, 200.0]))
    stats = np.zeros((2, 8))
    stats[0, 0], stats[0, 2] = 4, 8.0
    qad = np.array([[3, 1], [0, 0]])
    lam = (1.0, 2.0, 3.0, 0.5)
    C = -((10 / 30) + (200 / 400)) / 2        # -0.41666...
    Lb = -1.0 / 2.0                            # counts 3, 1: mean 2, population std 1
    S = 2 / 256
    U = 8.0 / 4
    R = T.reward(stats, qad, t, lam)
    assert math.isclose(R[0], 1.0 * C + 2.0 * Lb - 3.0 * S - 0.5 * U, rel_tol=1e-15)
    assert math.isclose(R[1], 1.0 * C - 3.0 * S, rel_tol=1e-15)


def test_common_arrivals_make_proposals_comparable():
    # identical proposals give identical trials; reordering the proposals
    # reorders the results
    rng = np.random.default_rng(3)
    cap = 3000
    length = rng.integers(1, 4000, cap).astype(np.int32)
    arrival = (rng.random(cap) * 10).astype(np.float32)
    t = oracle.partition(length, init_queues=8, max_queues=8)
    batches = [(rng.integers(1, 4000, 200).astype(np.int32), (10 + s + rng.random(200)).astype(np.float32),
                11.0 + s) for s in range(6)]
    th = np.array([[0, 1, 0, 1, 0, 1], [0, 1, 0, 1, 0, 1], [0.001, 0.5, 0.0, 2.0, 0.01, 0.2]], np.float32)
    s1, q1, _ = T.trial(length, arrival, t, th, batches, 64, COST)
    assert np.array_equal(s1[0], s1[1]) and np.array_equal(q1[0], q1[1])
    s2, q2, _ = T.trial(length, arrival, t, th[[2, 0, 1]], batches, 64, COST)
    assert np.array_equal(s2, s1[[2, 0, 1]]) and np.array_equal(q2, q1[[2, 0, 1]])
    # admissions plus what is left pending account for every request
    total = int((length > 0).sum()) + sum(len(b[0]) for b in batches)
    assert np.all(s1[:, 0] + s1[:, 5] <= total)
