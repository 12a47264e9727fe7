"""Streaming scheduler state on one GPU: a ring of request slots, a log of
recent arrival lengths holding the partitioner's sliding window, and
double-buffered queue tables.

Each step inserts the step's arrivals into the ring (request id = ring slot;
an overwritten, still-pending request is evicted) and runs the fused step
(route + score + top-B admission), tombstoning the admitted slots; with
step(now, length=..., arrival=...) the insert happens inside the step's own
kernels (ewsjf_ring_step).  The step also stores the arrivals' lengths into
the log (a ring of `log_capacity` >= `window` entries); the window is always
its last `window` entries.

The paper runs the partitioner off the critical path, in the strategic loop
(Section 3.1; Section 5), over a window of recent requests (Section 4.2).
launch_repartition() after step s does its work on a side stream: it brings
the window's length histogram up to date (ewsjf_window_advance moves the
counts of the lengths that left the window to the ones that joined it, when
the log still holds both; otherwise ewsjf_window_histogram recounts the
window from the log) and runs Refine-and-Prune from the histogram
(ewsjf_partition_hist: the same table, bit for bit, as partitioning the
window, since Refine-and-Prune sees it only through its distinct lengths and
their multiplicities).  The new table takes effect at step s + 1 (handover
"next_step", which makes that step wait for the partition), or at the first
step issued after the partition has finished on the device (handover
"when_ready": the paper's non-blocking background optimizer, where no step
waits).  A step whose log writes would overwrite entries a queued
side-stream read still needs waits for that read first.

With bubbles=(width, max_queues), the Dispatcher's on-demand bubble queues
(Section 4.3, Algorithm 2) place each step's arrivals in the table the step
is about to use (the new one, at a hand-over) before the step, so an arrival
in a gap between queues can open a queue of its own until the next
repartition replaces the set.

Every step runs in libewsjf.so's kernels: ewsjf_ring_step (or
ewsjf_ring_insert and ewsjf_step), and ewsjf_dispatch with bubbles, on the
caller's stream; ewsjf_window_advance or ewsjf_window_histogram, then
ewsjf_partition_hist, on the side stream.
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
    vector (6 floats); cost: (c0, c1, c2); incremental: move the window's
    histogram forward when the log allows it (False: recount the window at
    every repartition); log_capacity: length-log entries (default 2 *
    window); bubbles: (bubble_width, max_queues) to dispatch each step's
    arrivals with on-demand bubble queues (ewsjf_dispatch) into the table the
    step uses, before the step (None: the table's contiguous routing);
    handover: "next_step" (a partition launched after step s takes effect at
    step s + 1, which waits for it) or "when_ready" (it takes effect at the
    first step issued after it has finished on the device; no step waits,
    and a repartition requested while one is still running is skipped).
    """

    def __init__(self, capacity: int, window: int, B: int, params: L.PartitionParams, theta, cost=ewsjf.DEFAULT_COST,
                 device="cuda", incremental: bool = True, log_capacity: int | None = None,
                 bubbles: tuple[int, int] | None = None, handover: str = "next_step"):
        if handover not in ("next_step", "when_ready"):
            raise ValueError("handover is 'next_step' or 'when_ready'")
        if capacity <= 0 or window <= 0 or window > capacity:
            raise ValueError("need 0 < window <= capacity")
        log_capacity = 2 * int(window) if log_capacity is None else int(log_capacity)
        if log_capacity < window:
            raise ValueError("the length log must hold the window")
        self.device = torch.device(device)
        self.capacity, self.window, self.B = int(capacity), int(window), int(B)
        self.log_cap = log_capacity
        self.params, self.cost = params, cost
        self.incremental = bool(incremental)
        self.theta = _dev(np.asarray(theta, np.float32).reshape(1, 6), torch.float32, self.device)
        self.len = torch.zeros(self.capacity, dtype=torch.int32, device=self.device)
        self.arr = torch.zeros(self.capacity, dtype=torch.float32, device=self.device)
        self.log = torch.zeros(self.log_cap, dtype=torch.int32, device=self.device)
        self.hist = torch.zeros(params.max_len + 1, dtype=torch.int32, device=self.device)
        self.tables = [ewsjf.new_table(self.device), ewsjf.new_table(self.device)]
        self.cur = 0
        self.ws_step = ewsjf.Workspace(self.device)
        self.ws_part = ewsjf.Workspace(self.device)
        self.out = (torch.empty((1, self.B), dtype=torch.int32, device=self.device),
                    torch.empty((1, self.B), dtype=torch.float32, device=self.device),
                    torch.empty((1,), dtype=torch.int32, device=self.device))
        self.side = torch.cuda.Stream(device=self.device)  # default priority
        self.pending = None    # event of a partition that takes effect at the next step
        self.ring_pos = 0      # next ring slot to write
        self.head = 0          # lengths written to the log so far; the window is [head - window, head)
        self.hist_head = 0     # self.hist counts the window [hist_head - window, hist_head)
        self.read_lo = None    # oldest log entry a queued side-stream read still needs
        self.read_done = None  # event after that read
        self.advanced = 0      # repartitions that moved the histogram (the rest recounted the window)
        self.bubbles = None if bubbles is None else (int(bubbles[0]), int(bubbles[1]))
        self.undispatched = []  # (length, arrival) inserted since the last step, in order
        self.qid = torch.empty(L.MAX_DISPATCH, dtype=torch.int32, device=self.device)
        self.handover = handover
        self.skipped = 0     # repartitions skipped while one was still running (when_ready)
        self.swaps = []      # step numbers at which a new table took effect
        self.steps_done = 0

    # -- state ----------------------------------------------------------------
    def table(self) -> torch.Tensor:
        """The queue table the next step uses (once any pending partition lands)."""
        return self.tables[self.cur if self.pending is None else 1 - self.cur]

    def window_lengths(self) -> torch.Tensor:
        """The current window (a copy, oldest first), after the side stream's
        queued reads; for checks."""
        main = torch.cuda.current_stream(self.device)
        main.wait_stream(self.side)
        idx = (torch.arange(self.head - self.window, self.head, device=self.device) % self.log_cap)
        return self.log[idx]

    def fill(self, length, arrival) -> None:
        """Fill every ring slot (ids 0..capacity-1), take the window from the
        last `window` of them and partition it synchronously on the current
        stream."""
        length = _dev(length, torch.int32, self.device)
        arrival = _dev(arrival, torch.float32, self.device)
        if length.numel() != self.capacity or arrival.numel() != self.capacity:
            raise ValueError("the initial fill covers every ring slot")
        main = torch.cuda.current_stream(self.device)
        main.wait_stream(self.side)  # earlier side-stream work is done
        self.len.copy_(length)
        self.arr.copy_(arrival)
        self.log[:self.window].copy_(length[self.capacity - self.window:])
        self.ring_pos = 0
        self.head = self.hist_head = self.window
        self.read_lo = self.read_done = None
        ewsjf.window_histogram(self.log, self.params.max_len, hist=self.hist, begin=0, n=self.window)
        ewsjf.partition_hist(self.hist, self.params, table=self.tables[self.cur], ws=self.ws_part)
        self.pending = None
        self.side.wait_stream(main)  # the side stream's next reads follow the fill

    def _log_slot(self, n: int) -> int:
        """The log slot of the next n lengths; first makes the current stream
        wait for a queued side-stream read those writes would overwrite."""
        if n > self.log_cap:
            raise ValueError("one step inserts at most log_capacity arrivals")
        if self.read_lo is not None and self.head + n - self.log_cap > self.read_lo:
            torch.cuda.current_stream(self.device).wait_event(self.read_done)
            self.read_lo = self.read_done = None
        return self.head % self.log_cap

    def insert(self, length: torch.Tensor, arrival: torch.Tensor) -> None:
        """Write one step's arrivals into the next ring slots (evicting what
        was there) and their lengths into the log."""
        n = length.numel()
        if arrival.numel() != n or n > self.capacity:
            raise ValueError("one step inserts at most capacity arrivals")
        wpos = self._log_slot(n)
        ewsjf.ring_insert(self.len, self.arr, self.ring_pos, length, arrival, window=self.log, wpos=wpos)
        self.ring_pos = (self.ring_pos + n) % self.capacity
        self.head += n
        if self.bubbles is not None:
            self.undispatched.append((length, arrival))

    def _dispatch(self, batches) -> None:
        """Arrivals through the Dispatcher with bubble queues into the current
        table, batch by batch in arrival order."""
        width, mq = self.bubbles
        for length, arrival in batches:
            for a in range(0, length.numel(), L.MAX_DISPATCH):
                b = min(length.numel(), a + L.MAX_DISPATCH)
                ewsjf.dispatch(length[a:b], arrival[a:b], self.tables[self.cur], width, mq, qid=self.qid[:b - a])

    def launch_repartition(self) -> None:
        """Partition the window as of the last step on the side stream; the
        new table takes effect at the next step()."""
        if self.pending is not None:
            if self.handover == "when_ready":
                self.skipped += 1  # the strategic loop is still busy with the previous one
                return
            raise RuntimeError("a partition is already pending")
        main = torch.cuda.current_stream(self.device)
        self.side.wait_stream(main)  # the log holds every step so far
        H, W, R, new = self.head, self.window, self.log_cap, self.head - self.hist_head
        if self.incremental and new < W and new <= R - W:
            # the entries that left ([hist_head - W, H - W)) and joined ([hist_head, H)) are both in the log
            ewsjf.window_advance(self.log, self.hist_head % R, (self.hist_head - W) % R, new, self.hist,
                                 stream=self.side)
            lo = self.hist_head - W
            self.advanced += 1
        else:
            ewsjf.window_histogram(self.log, self.params.max_len, hist=self.hist, begin=(H - W) % R, n=W,
                                   stream=self.side)
            lo = H - W
        self.hist_head = H
        read = torch.cuda.Event()
        read.record(self.side)
        self.read_lo = lo if self.read_lo is None else min(self.read_lo, lo)
        self.read_done = read
        ewsjf.partition_hist(self.hist, self.params, table=self.tables[1 - self.cur], ws=self.ws_part,
                             stream=self.side)
        done = torch.cuda.Event()
        done.record(self.side)
        self.pending = done

    def step(self, now: float, tombstone: bool = True, length: torch.Tensor | None = None,
             arrival: torch.Tensor | None = None):
        """One scheduling step over the ring: (ids[1,B], top[1,B], n_sel[1]).
        With length/arrival, the step's arrivals are inserted first, inside
        the step's kernels (same effect as insert() then step())."""
        main = torch.cuda.current_stream(self.device)
        if self.pending is not None and (self.handover == "next_step" or self.pending.query()):
            main.wait_event(self.pending)  # free once the partition has finished (when_ready)
            self.cur = 1 - self.cur
            self.pending = None
            self.swaps.append(self.steps_done)
        self.steps_done += 1
        if self.bubbles is not None:
            batches, self.undispatched = self.undispatched, []
            if length is not None:
                batches.append((length, arrival))
            self._dispatch(batches)
        if length is None:
            return ewsjf.step(self.len, self.arr, now, self.tables[self.cur], self.theta, self.B, self.cost,
                              tombstone=tombstone, out=self.out, ws=self.ws_step)
        n = length.numel()
        if arrival is None or arrival.numel() != n or n > self.capacity:
            raise ValueError("one step inserts at most capacity arrivals")
        wpos = self._log_slot(n)
        out = ewsjf.ring_step(self.len, self.arr, self.ring_pos, length, arrival, now, self.tables[self.cur],
                              self.theta, self.B, self.cost, window=self.log, wpos=wpos, tombstone=tombstone,
                              out=self.out, ws=self.ws_step)
        self.ring_pos = (self.ring_pos + n) % self.capacity
        self.head += n
        return out

    def apply_tombstones(self, ids) -> None:
        """Mark the given slots empty (len = 0)."""
        idx = _dev(np.asarray(ids, np.int64).reshape(-1), torch.int64, self.device)
        if idx.numel():
            self.len.index_fill_(0, idx, 0)
