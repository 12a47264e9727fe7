"""Trials of batched scoring-parameter proposals on one GPU: the simulator
side of the meta-optimizer (Section 4.4.2).

The optimizer executes each candidate Theta for a trial interval, collects
statistics and updates its posterior with the reward of Eq. 5.  Here P
proposals run side by side: proposal t owns pool t (a copy of the starting
pool), every pool receives the same arrivals, and each step admits each
pool's top B under its own parameter vector (ewsjf_trial_step, which also
accumulates the statistics of the admitted requests).  finish() adds the
pending-side statistics and returns Eq. 5 per proposal (ewsjf_trial_finish).
The queue structure stays the one in force when the trial starts.  The
optimizer that proposes the next batch is not part of this module.
"""
from __future__ import annotations

import numpy as np
import torch

from . import _lib as L
from . import ewsjf

STATS = ("admitted", "tokens", "wait_sum", "wait_sq_sum", "wait_max", "pending", "pending_wait_max", "steps")


def _dev(a, dtype, device):
    if isinstance(a, torch.Tensor):
        return a.to(device=device, dtype=dtype).contiguous()
    return torch.from_numpy(np.ascontiguousarray(a)).to(device=device, dtype=dtype)


class Trial:
    """P proposals (thetas [P][6]) over pools of `capacity` slots (a multiple
    of 4), B admissions per step, one queue table for the whole trial."""

    def __init__(self, capacity: int, thetas, B: int, table: torch.Tensor, cost=ewsjf.DEFAULT_COST, device="cuda"):
        if capacity <= 0 or capacity % 4:
            raise ValueError("capacity must be a positive multiple of 4")
        self.device = torch.device(device)
        self.theta = _dev(np.asarray(thetas, np.float32).reshape(-1, 6), torch.float32, self.device)
        self.P, self.capacity, self.B = self.theta.shape[0], int(capacity), int(B)
        self.table, self.cost = table, cost
        self.len = torch.zeros((self.P, self.capacity), dtype=torch.int32, device=self.device)
        self.arr = torch.zeros((self.P, self.capacity), dtype=torch.float32, device=self.device)
        self.stats = torch.zeros((self.P, L.TRIAL_STATS), dtype=torch.float64, device=self.device)
        self.queue_admits = torch.zeros((self.P, L.MAX_QUEUES), dtype=torch.int64, device=self.device)
        self.out = ewsjf._outs(self.P, self.B, self.device, None)
        self.ws = ewsjf.Workspace(self.device)
        self.pos = 0
        self.now = 0.0

    def start(self, length, arrival) -> None:
        """Every proposal starts from the same pool (capacity slots)."""
        length = _dev(length, torch.int32, self.device)
        arrival = _dev(arrival, torch.float32, self.device)
        if length.numel() != self.capacity or arrival.numel() != self.capacity:
            raise ValueError("the starting pool covers every slot")
        self.len.copy_(length.expand(self.P, -1))
        self.arr.copy_(arrival.expand(self.P, -1))
        self.stats.zero_()
        self.queue_admits.zero_()
        self.pos = 0

    def step(self, length: torch.Tensor, arrival: torch.Tensor, now: float):
        """The step's arrivals into every pool, then each pool's admission:
        (ids[P,B], top[P,B], n_sel[P])."""
        n = length.numel()
        if arrival.numel() != n or n > self.capacity:
            raise ValueError("one step inserts at most capacity arrivals")
        out = ewsjf.trial_step(self.len, self.arr, self.pos, length, arrival, now, self.table, self.theta, self.B,
                               self.stats, self.queue_admits, self.cost, out=self.out, ws=self.ws)
        self.pos = (self.pos + n) % self.capacity
        self.now = float(now)
        return out

    def finish(self, lam=(1.0, 1.0, 1.0, 1.0)) -> torch.Tensor:
        """Eq. 5 per proposal (float64 [P]); self.stats holds the statistics."""
        return ewsjf.trial_finish(self.len, self.arr, self.now, self.table, self.stats, self.queue_admits, lam)
