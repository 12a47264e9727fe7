"""Trials of scoring-parameter proposals -- TEST INFRASTRUCTURE ONLY.

The simulator side of the meta-optimizer (Section 4.4.2): each proposal
Theta is run for a trial of T steps of the tactical step (per-request scoring
and top-B admission) on its own copy of the pool, every copy receiving the
same arrivals, and the trial's statistics feed the reward of Eq. 5.  Plain
and slow: one oracle.step per proposal and step.  Only the tests use it.

Readings (the paper describes the trial and the reward terms in words only):
  M0 A trial runs under the queue structure in force at its start (the
     optimizer tunes the scoring parameters of that structure).  Step s first
     writes the step's arrivals into ring slots (pos + i) mod capacity of
     every copy, then admits and tombstones.
  M1 Statistics of the admitted requests: count, tokens (sum of prompt
     lengths), sum, sum of squares and maximum of the wait W = max(0, now -
     arrival) in seconds (a NaN arrival waits 0), admissions per queue; at the
     trial's end, the pending requests and their maximum wait.
  M2 Eq. 5: C (compact, homogeneous queues) = minus the mean over queues of
     (hi - lo) / (hi + lo); L (load imbalance) = minus the coefficient of
     variation (population) of the admissions per queue, 0 without
     admissions; S (queue proliferation) = k / 256; U (user experience,
     latency) = the mean wait of the admitted requests, 0 without admissions.
     R = lambda1 C + lambda2 L - lambda3 S - lambda4 U.
"""
from __future__ import annotations

import math

import numpy as np

from . import Table, route, step

STATS = ("admitted", "tokens", "wait_sum", "wait_sq_sum", "wait_max", "pending", "pending_wait_max", "steps")
MAX_QUEUES = 256


def wait(arrival, now) -> np.ndarray:
    """W = max(0, now - arrival) in binary64 (NaN -> 0)."""
    w = np.float64(np.float32(now)) - np.asarray(arrival, np.float32).astype(np.float64)
    return np.where(w > 0.0, w, 0.0)


def trial(length, arrival, table: Table, thetas, batches, B: int, cost=(0.01, 1e-4, 0.0)):
    """length, arrival: the pool at the trial's start (capacity slots);
    thetas: [P][6]; batches: [(new_len, new_arrival, now)] per step.
    Returns (stats [P][8] float64, queue_admits [P][k] int64, admitted ids
    per step [T][P] arrays)."""
    th = np.asarray(thetas, np.float32).reshape(-1, 6)
    P, cap, k = th.shape[0], len(length), table.k
    pools = [(np.asarray(length, np.int32).copy(), np.asarray(arrival, np.float32).copy()) for _ in range(P)]
    stats = np.zeros((P, len(STATS)), np.float64)
    qad = np.zeros((P, k), np.int64)
    history = []
    pos = 0
    now = 0.0
    for new_len, new_arr, now in batches:
        n = len(new_len)
        slots = (pos + np.arange(n)) % cap
        admitted = []
        for p in range(P):
            L, A = pools[p]
            L[slots] = new_len
            A[slots] = new_arr
            ids, _, nsel, _ = step(L, A, now, table, th[p], B, cost)
            adm = ids[0][:int(nsel[0])]
            w = wait(A[adm], now)
            stats[p, 0] += adm.size
            stats[p, 1] += float(np.sum(L[adm].astype(np.int64)))
            stats[p, 2] += math.fsum(w)
            stats[p, 3] += math.fsum(w * w)
            stats[p, 4] = max(stats[p, 4], float(w.max()) if w.size else 0.0)
            qad[p] += np.bincount(route(L[adm], table), minlength=k)[:k]
            L[adm] = 0
            admitted.append(adm.copy())
        history.append(admitted)
        pos = (pos + n) % cap
        stats[:, 7] += 1
    for p in range(P):
        L, A = pools[p]
        pend = L > 0
        stats[p, 5] = int(pend.sum())
        w = wait(A[pend], now)
        stats[p, 6] = float(w.max()) if w.size else 0.0
    return stats, qad, history


def reward(stats, queue_admits, table: Table, lam) -> np.ndarray:
    """Eq. 5 with reading M2, one value per proposal."""
    lo = np.asarray(table.lo, np.float64)
    hi = np.asarray(table.hi, np.float64)
    C = -float(np.mean((hi - lo) / (hi + lo)))
    S = table.k / MAX_QUEUES
    out = np.zeros(len(stats))
    for p, (s, c) in enumerate(zip(stats, np.asarray(queue_admits, np.float64))):
        m = c.mean()
        Lb = -float(np.sqrt(np.mean((c - m) ** 2)) / m) if m > 0 else 0.0
        U = s[2] / s[0] if s[0] > 0 else 0.0
        out[p] = lam[0] * C + lam[1] * Lb - lam[2] * S - lam[3] * U
    return out
