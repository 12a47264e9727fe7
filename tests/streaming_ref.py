"""Host-side lockstep reference of the streaming scheduler, built on the
oracle: the same ring, window and hand-over rules as
paper_2601_21758_amd.streaming, with the oracle's partition and step."""
from __future__ import annotations

import numpy as np

import oracle


class OracleStream:
    def __init__(self, capacity: int, window: int, B: int, init_queues: int, max_queues: int, theta, cost,
                 bubbles=None):
        self.capacity, self.window, self.B = capacity, window, B
        self.kw = dict(init_queues=init_queues, max_queues=max_queues)
        self.theta = np.asarray(theta, np.float32).reshape(1, 6)
        self.cost = cost
        self.len = np.zeros(capacity, np.int32)
        self.arr = np.zeros(capacity, np.float32)
        self.win = np.zeros(window, np.int32)
        self.ring_pos = 0
        self.win_pos = 0
        self.table = None
        self.next_table = None
        self.bubbles = bubbles  # (width, max_queues): arrivals dispatched before each step (Algorithm 2)
        self.undispatched = []
        self.created = 0  # bubble queues created so far

    def fill(self, length, arrival):
        self.len[:] = length
        self.arr[:] = arrival
        self.win[:] = length[self.capacity - self.window:]
        self.ring_pos = self.win_pos = 0
        self.table = oracle.partition(self.win, **self.kw)
        self.next_table = None

    def insert(self, length, arrival):
        n = len(length)
        slots = (self.ring_pos + np.arange(n)) % self.capacity
        self.len[slots] = length
        self.arr[slots] = arrival
        wslots = (self.win_pos + np.arange(n)) % self.window
        self.win[wslots] = length
        self.ring_pos = (self.ring_pos + n) % self.capacity
        self.win_pos = (self.win_pos + n) % self.window
        if self.bubbles is not None:
            self.undispatched.append((np.asarray(length, np.int32), np.asarray(arrival, np.float32)))

    def repartition(self):
        self.next_table = oracle.partition(self.win, **self.kw)
        return self.next_table

    def step(self, now, take_new=None):
        """Route, score and select over the ring with the current table; the
        partition of the last repartition() takes effect here first (at the
        step after it, or, with take_new given, when take_new is true)."""
        if self.next_table is not None and (take_new is None or take_new):
            self.table, self.next_table = self.next_table, None
        for length, arrival in self.undispatched:
            k0 = self.table.k
            _, self.table = oracle.dispatch(length, arrival, self.table, *self.bubbles)
            self.created += self.table.k - k0
        self.undispatched = []
        ids, top, nsel, sc = oracle.step(self.len, self.arr, now, self.table, self.theta, self.B, self.cost)
        return ids[0], top[0], int(nsel[0]), sc[0]

    def tombstone(self, ids):
        self.len[np.asarray(ids, np.int64)] = 0
