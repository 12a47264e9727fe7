"""Streaming scheduler state on one GPU: a ring of request slots, a sliding
window of recent arrival lengths, and double-buffered queue tables.

Each step inserts the step's arrivals into the ring (request id = ring slot;
an overwritten, still-pending request is evicted) and runs the fused step
(route + score + top-B admission), tombstoning the admitted slots; with
step(now, length=..., arrival=...) the insert happens inside the step's own
kernels (ewsjf_ring_step).  After step s, launch_repartition() starts
Refine-and-Prune over the window (which holds step s's arrivals) on a side
stream; the new table takes effect at step s + 1.  The paper runs the
partitioner off the critical path, in the strategic loop (Section 3.1;
Section 5), over a window of recent requests (Section 4.2).

With incremental=True (the default) the inserts also keep the window's
length histogram current (each overwritten length's count moves to the new
length), and the repartition starts from a copy of that histogram
(ewsjf_partition_hist) instead of re-reading the window: the same table, bit
for bit, since Refine-and-Prune sees the window only through its distinct
lengths and their multiplicities.

Every step runs in libewsjf.so's kernels: ewsjf_ring_step (or
ewsjf_ring_insert and ewsjf_step), and ewsjf_partition_hist (or
ewsjf_partition).
"""
from __future__ import annotations

import numpy as np
import torch

from . import ewsjf
from . import _lib as L


def _dev(a, dtype, device):
    if isinstance(a, torch.Tensor):
        return a.to(device=device, dtype=dtype).contiguous()
    return torch.from_numpy(np.ascontiguousarray(a)).to(device=device, dtype=dtype)


class StreamingScheduler:
    """Device state of the streaming scheduler.

    capacity: ring slots (request ids); window: partitioner window length;
    B: admissions per step; params: ewsjf.params(...); theta: one parameter
    vector (6 floats); cost: (c0, c1, c2); incremental: keep the window's
    histogram and partition from it.
    """

    def __init__(self, capacity: int, window: int, B: int, params: L.PartitionParams, theta, cost=ewsjf.DEFAULT_COST,
                 device="cuda", incremental: bool = True):
        if capacity <= 0 or window <= 0 or window > capacity:
            raise ValueError("need 0 < window <= capacity")
        self.device = torch.device(device)
        self.capacity, self.window, self.B = int(capacity), int(window), int(B)
        self.params, self.cost = params, cost
        self.theta = _dev(np.asarray(theta, np.float32).reshape(1, 6), torch.float32, self.device)
        self.len = torch.zeros(self.capacity, dtype=torch.int32, device=self.device)
        self.arr = torch.zeros(self.capacity, dtype=torch.float32, device=self.device)
        self.win = torch.zeros(self.window, dtype=torch.int32, device=self.device)
        self.incremental = bool(incremental)
        if self.incremental:  # the window's histogram and the copy a partition reads
            self.hist = torch.zeros(params.max_len + 1, dtype=torch.int32, device=self.device)
            self.snap = torch.zeros(params.max_len + 1, dtype=torch.int32, device=self.device)
        else:  # the copy of the window a partition reads
            self.hist = None
            self.snap = torch.zeros(self.window, dtype=torch.int32, device=self.device)
        self.tables = [ewsjf.new_table(self.device), ewsjf.new_table(self.device)]
        self.cur = 0
        self.ws_step = ewsjf.Workspace(self.device)
        self.ws_part = ewsjf.Workspace(self.device)
        self.out = (torch.empty((1, self.B), dtype=torch.int32, device=self.device),
                    torch.empty((1, self.B), dtype=torch.float32, device=self.device),
                    torch.empty((1,), dtype=torch.int32, device=self.device))
        self.side = torch.cuda.Stream(device=self.device)  # default priority
        self.pending = None  # event of a partition that takes effect at the next step
        self.ring_pos = 0    # next ring slot to write
        self.win_pos = 0     # next window slot to write (the oldest entry)

    # -- state ----------------------------------------------------------------
    def table(self) -> torch.Tensor:
        """The queue table the next step uses (once any pending partition lands)."""
        return self.tables[self.cur if self.pending is None else 1 - self.cur]

    def fill(self, length, arrival) -> None:
        """Fill every ring slot (ids 0..capacity-1), take the window from the
        last `window` of them and partition it synchronously on the current
        stream."""
        length = _dev(length, torch.int32, self.device)
        arrival = _dev(arrival, torch.float32, self.device)
        if length.numel() != self.capacity or arrival.numel() != self.capacity:
            raise ValueError("the initial fill covers every ring slot")
        self.len.copy_(length)
        self.arr.copy_(arrival)
        # window slot i holds the i-th oldest of the last `window` arrivals
        self.win.copy_(length[self.capacity - self.window:])
        self.win_pos = 0
        self.ring_pos = 0
        if self.incremental:
            ewsjf.window_histogram(self.win, self.params.max_len, hist=self.hist)
            ewsjf.partition_hist(self.hist, self.params, table=self.tables[self.cur], ws=self.ws_part)
        else:
            ewsjf.partition(self.win, self.params, table=self.tables[self.cur], ws=self.ws_part)
        self.pending = None

    def insert(self, length: torch.Tensor, arrival: torch.Tensor) -> None:
        """Write one step's arrivals into the next ring slots (evicting what
        was there) and into the window (replacing its oldest entries)."""
        n = length.numel()
        if arrival.numel() != n or n > self.capacity or n > self.window:
            raise ValueError("one step inserts at most min(capacity, window) arrivals")
        ewsjf.ring_insert(self.len, self.arr, self.ring_pos, length, arrival, window=self.win, wpos=self.win_pos,
                          hist=self.hist)
        self.ring_pos = (self.ring_pos + n) % self.capacity
        self.win_pos = (self.win_pos + n) % self.window

    def launch_repartition(self) -> None:
        """Partition the current window on the side stream; the new table
        takes effect at the next step()."""
        if self.pending is not None:
            raise RuntimeError("a partition is already pending")
        main = torch.cuda.current_stream(self.device)
        # the next insert may change the window and its histogram
        self.snap.copy_(self.hist if self.incremental else self.win)
        ready = torch.cuda.Event()
        ready.record(main)
        nxt = 1 - self.cur
        with torch.cuda.stream(self.side):
            self.side.wait_event(ready)
            if self.incremental:
                ewsjf.partition_hist(self.snap, self.params, table=self.tables[nxt], ws=self.ws_part,
                                     stream=self.side)
            else:
                ewsjf.partition(self.snap, self.params, table=self.tables[nxt], ws=self.ws_part, stream=self.side)
            done = torch.cuda.Event()
            done.record(self.side)
        self.pending = done

    def step(self, now: float, tombstone: bool = True, length: torch.Tensor | None = None,
             arrival: torch.Tensor | None = None):
        """One scheduling step over the ring: (ids[1,B], top[1,B], n_sel[1]).
        With length/arrival, the step's arrivals are inserted first, inside
        the step's kernels (same effect as insert() then step())."""
        main = torch.cuda.current_stream(self.device)
        if self.pending is not None:
            main.wait_event(self.pending)
            self.cur = 1 - self.cur
            self.pending = None
        if length is None:
            return ewsjf.step(self.len, self.arr, now, self.tables[self.cur], self.theta, self.B, self.cost,
                              tombstone=tombstone, out=self.out, ws=self.ws_step)
        n = length.numel()
        if arrival is None or arrival.numel() != n or n > self.capacity or n > self.window:
            raise ValueError("one step inserts at most min(capacity, window) arrivals")
        out = ewsjf.ring_step(self.len, self.arr, self.ring_pos, length, arrival, now, self.tables[self.cur],
                              self.theta, self.B, self.cost, window=self.win, wpos=self.win_pos, tombstone=tombstone,
                              out=self.out, ws=self.ws_step, hist=self.hist)
        self.ring_pos = (self.ring_pos + n) % self.capacity
        self.win_pos = (self.win_pos + n) % self.window
        return out

    def apply_tombstones(self, ids) -> None:
        """Mark the given slots empty (len = 0)."""
        idx = _dev(np.asarray(ids, np.int64).reshape(-1), torch.int64, self.device)
        if idx.numel():
            self.len.index_fill_(0, idx, 0)
