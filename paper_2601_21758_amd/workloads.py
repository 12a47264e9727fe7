"""Seeded synthetic request pools, windows and scoring-parameter vectors.

This module only draws inputs: prompt lengths, arrival times, observation
windows, scoring parameter vectors and the streaming arrival process.  It
holds none of the scheduler's arithmetic (no partitioning, routing, scoring
or selection), so both the HIP path and the CPU oracle can be fed from it.

The workloads stand in for the paper's unnamed datasets (Section 6,
"Datasets and workloads": a bimodal mix of short interactive and long
batch prompts under Poisson arrivals, 80% short / 20% long).  Nothing from
any real dataset is used.

Every generator is ``numpy.random.Generator(PCG64(seed))`` with a fixed
draw order per chunk of requests:
  1. one uniform per request picks the mixture component,
  2. one standard normal per request gives the lognormal length
     ``clip(rint(exp(mu + sigma * z)), lo, hi)`` (round half to even),
  3. the arrival times,
  4. scoring parameter vectors (batched-parameter workload only).
"""
from __future__ import annotations

import hashlib
from dataclasses import dataclass, field

import numpy as np

MAX_LEN = 32768

# Mixture components: (weight, median tokens, sigma, clip lo, clip hi).
# "two": 80% short / 20% long, the clip point 2048 separates the modes.
MIX_TWO = ((0.8, 128.0, 0.6, 1, 2048), (0.2, 6000.0, 0.4, 2048, MAX_LEN))
# "three": short / medium / long modes, all clipped to [1, 32768].
MIX_THREE = ((0.6, 64.0, 0.5, 1, MAX_LEN), (0.3, 1024.0, 0.5, 1, MAX_LEN),
             (0.1, 12000.0, 0.4, 1, MAX_LEN))

# Scoring parameter vector layout: (a_base, b_base, a_urg, b_urg, a_fair, b_fair);
# every weight is affine in the queue's mean prompt length.
THETA_LO = np.array([-1.5e-5, 0.5, -3.0e-5, 1.0, 0.0, 0.5])
THETA_HI = np.array([1.5e-5, 1.5, 0.0, 2.0, 3.0e-5, 1.5])
THETA_MID = ((THETA_LO + THETA_HI) / 2.0).astype(np.float32)

# Prefill-cost model C(b) = c0 + c1*b + c2*b*b seconds.
DEFAULT_COST = (0.01, 1e-4, 0.0)


def _lengths(rng: np.random.Generator, n: int, mix) -> np.ndarray:
    w = np.array([m[0] for m in mix], dtype=np.float64)
    cum = np.cumsum(w)[:-1]
    u = rng.random(n)
    comp = np.searchsorted(cum, u, side="right")
    z = rng.standard_normal(n)
    mu = np.log(np.array([m[1] for m in mix]))[comp]
    sg = np.array([m[2] for m in mix])[comp]
    lo = np.array([m[3] for m in mix])[comp]
    hi = np.array([m[4] for m in mix])[comp]
    x = np.rint(np.exp(mu + sg * z))
    return np.clip(x, lo, hi).astype(np.int32)


def _two_mix_with_short_weight(p_short: float):
    (_, m0, s0, l0, h0), (_, m1, s1, l1, h1) = MIX_TWO
    return ((p_short, m0, s0, l0, h0), (1.0 - p_short, m1, s1, l1, h1))


@dataclass
class Pool:
    """One scheduling step's input: request id = index into the arrays."""
    name: str
    seed: int
    length: np.ndarray          # int32 [n]; <= 0 marks an empty slot
    arrival: np.ndarray         # float32 [n], seconds
    now: float                  # float32-representable clock, seconds
    window: np.ndarray          # int32 [W], lengths the partitioner sees
    init_queues: int            # K: equal-width coarse bins
    max_queues: int
    B: int
    theta: np.ndarray           # float32 [n_theta, 6]
    cost: tuple = DEFAULT_COST
    extra: dict = field(default_factory=dict)

    @property
    def n(self) -> int:
        return int(self.length.shape[0])

    def digest(self) -> str:
        h = hashlib.sha256()
        for a in (self.length, self.arrival, self.window, self.theta):
            h.update(np.ascontiguousarray(a).tobytes())
        h.update(np.float32(self.now).tobytes())
        return h.hexdigest()


def make_pool(mix: str, n: int, seed: int, *, arrivals: str, horizon: float = 60.0,
              rate: float = 1e4, window: int | None = None, K: int = 16, B: int = 64,
              n_theta: int = 1, name: str = "custom") -> Pool:
    """Draw a pool with the given recipe.

    arrivals: "uniform" -> fp32 U[0, horizon), now = horizon;
              "poisson" -> cumulative Exp(1/rate) gaps summed in fp64, stored
              fp32, now = the largest fp32 arrival.
    window:   None -> the same lengths as the pool; else the last `window`
              pool entries by id.
    """
    rng = np.random.Generator(np.random.PCG64(seed))
    mixdef = MIX_TWO if mix == "two" else MIX_THREE
    length = _lengths(rng, n, mixdef)
    if arrivals == "uniform":
        arrival = (rng.random(n) * horizon).astype(np.float32)
        now = float(np.float32(horizon))
    elif arrivals == "poisson":
        arrival = np.cumsum(rng.exponential(1.0 / rate, n)).astype(np.float32)
        now = float(arrival.max()) if n else 0.0
    else:
        raise ValueError(arrivals)
    if n_theta == 1:
        theta = THETA_MID.reshape(1, 6).copy()
    else:
        theta = rng.uniform(THETA_LO, THETA_HI, size=(n_theta, 6)).astype(np.float32)
    win = length.copy() if window is None else length[n - window:].copy()
    return Pool(name=name, seed=seed, length=length, arrival=arrival, now=now, window=win,
                init_queues=K, max_queues=K, B=B, theta=theta)


def config(idx: int, scale: float = 1.0, draw: int = 0) -> Pool:
    """The five evaluation workloads (0..3 here; 4 is `Streaming`).

    `scale` < 1 shrinks pool and window (keeping K and B) for quick tests.
    `draw` > 0 gives another independent pool of the same recipe (seed
    shifted by 7919 * draw); draw 0 is the workload itself.
    """
    def sz(x):
        return max(1, int(round(x * scale)))
    sd = 7919 * draw
    if idx == 0:
        return make_pool("two", sz(4096), 0 + sd, arrivals="uniform", horizon=60.0, window=None,
                         K=16, B=64, name="tiny_mixed_4k")
    if idx == 1:
        return make_pool("three", sz(262144), 1 + sd, arrivals="uniform", horizon=300.0,
                         window=sz(65536), K=64, B=256, name="mid_3mode_256k")
    if idx == 2:
        return make_pool("two", sz(4194304), 2 + sd, arrivals="poisson", rate=1e4,
                         window=sz(1048576), K=256, B=1024, name="large_mixed_4m")
    if idx == 3:
        return make_pool("three", sz(1048576), 3 + sd, arrivals="uniform", horizon=300.0,
                         window=sz(65536), K=64, B=256, n_theta=256,
                         name="batched_theta_1m")
    raise ValueError(idx)


class Streaming:
    """Streaming workload with drift: a ring of `capacity` request slots.

    Request id = ring slot.  The ring starts full (`capacity` arrivals at the
    initial short-request weight).  Step s then inserts `per_step` arrivals
    into slots (capacity + s*per_step + j) mod capacity, overwriting (evicting)
    whatever was there.  The short-request weight drifts linearly from
    `p_start` at step 0 to `p_end` at the last step.  Arrivals continue one
    Poisson process at `rate` per second (gaps summed in fp64, stored fp32).
    The partitioner window is the last `window` arrivals.

    `start_step` > 0 starts a run part-way through the drift: the fill is
    then the last `capacity` arrivals the run drew before that step (the
    step-0 fill and every earlier step's arrivals, drawn in the same order),
    oldest in slot 0, and steps start_step, start_step + 1, ... follow.
    """

    def __init__(self, seed: int = 4, capacity: int = 1 << 20, per_step: int = 4096,
                 steps: int = 10000, window: int = 65536, rp_every: int = 100, B: int = 512,
                 K: int = 64, p_start: float = 0.9, p_end: float = 0.3, rate: float = 1e4,
                 start_step: int = 0):
        self.rng = np.random.Generator(np.random.PCG64(seed))
        self.capacity, self.per_step, self.steps = capacity, per_step, steps
        self.window_size, self.rp_every, self.B, self.K = window, rp_every, B, K
        self.p_start, self.p_end, self.rate = p_start, p_end, rate
        self.clock = 0.0
        self.theta = THETA_MID.reshape(1, 6).copy()
        self.cost = DEFAULT_COST
        self.start_step = start_step
        self.next_step = start_step

    def p_short(self, s: int) -> float:
        if self.steps <= 1:
            return self.p_start
        return self.p_start + (self.p_end - self.p_start) * s / (self.steps - 1)

    def _chunk(self, n: int, p: float):
        length = _lengths(self.rng, n, _two_mix_with_short_weight(p))
        gaps = self.rng.exponential(1.0 / self.rate, n)
        t = self.clock + np.cumsum(gaps)
        self.clock = float(t[-1])
        return length, t.astype(np.float32)

    def initial_fill(self):
        """(length, arrival) for all `capacity` slots: at the step-0 weight,
        or from a later start step the last `capacity` arrivals before it."""
        length, arrival = self._chunk(self.capacity, self.p_start)
        if self.start_step == 0:
            return length, arrival
        pos = 0  # the ring slot the next arrival overwrites (the oldest)
        for s in range(self.start_step):
            ln, ar = self._chunk(self.per_step, self.p_short(s))
            idx = (pos + np.arange(self.per_step)) % self.capacity
            length[idx] = ln
            arrival[idx] = ar
            pos = (pos + self.per_step) % self.capacity
        return np.roll(length, -pos), np.roll(arrival, -pos)

    def arrivals(self, s: int):
        """Step s's arrivals; steps must be drawn in order start_step, start_step + 1, ..."""
        if s != self.next_step:
            raise ValueError("streaming arrivals must be drawn in step order")
        self.next_step += 1
        return self._chunk(self.per_step, self.p_short(s))

    def slots(self, s: int) -> np.ndarray:
        start = ((s - self.start_step) * self.per_step) % self.capacity
        return (start + np.arange(self.per_step)) % self.capacity


def adversarial(kind: str, n: int, seed: int = 0) -> tuple[np.ndarray, np.ndarray, float]:
    """Edge-case pools: (length int32[n], arrival float32[n], now)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    if kind == "equal_len":
        return np.full(n, 300, np.int32), (rng.random(n) * 60).astype(np.float32), 60.0
    if kind == "equal_arrival":
        return _lengths(rng, n, MIX_TWO), np.full(n, 10.0, np.float32), 60.0
    if kind == "all_equal":
        return np.full(n, 777, np.int32), np.full(n, 5.0, np.float32), 60.0
    if kind == "clip_spikes":
        l = np.where(rng.random(n) < 0.5, 2048, 32768).astype(np.int32)
        return l, (rng.random(n) * 60).astype(np.float32), 60.0
    if kind == "tombstones":
        l = _lengths(rng, n, MIX_TWO)
        l[rng.random(n) < 0.7] = 0
        l[rng.random(n) < 0.05] = -5
        return l, (rng.random(n) * 60).astype(np.float32), 60.0
    if kind == "over_max":
        l = rng.integers(1, 70000, n).astype(np.int32)
        return l, (rng.random(n) * 60).astype(np.float32), 60.0
    if kind == "future_arrivals":
        return _lengths(rng, n, MIX_TWO), (rng.random(n) * 120).astype(np.float32), 60.0
    if kind == "oldest_first":
        # equal lengths and arrivals rising with the id: the scores fall with
        # the id, so every top request sits in the first few slots
        return np.full(n, 100, np.int32), np.linspace(0.0, 60.0, n).astype(np.float32), 60.0
    if kind == "hot_blocks":
        # a few runs of 300 consecutive slots waited much longer than the rest
        l = _lengths(rng, n, MIX_TWO)
        a = (rng.random(n) * 10 + 50).astype(np.float32)
        for start in rng.integers(0, max(1, n - 300), 6):
            a[start:start + 300] = (rng.random(min(300, n - start)) * 5).astype(np.float32)
        return l, a, 60.0
    raise ValueError(kind)


ADVERSARIAL_KINDS = ("equal_len", "equal_arrival", "all_equal", "clip_spikes", "tombstones", "oldest_first",
                     "hot_blocks",
                     "over_max", "future_arrivals")


def digest(*arrays) -> str:
    h = hashlib.sha256()
    for a in arrays:
        h.update(np.ascontiguousarray(a).tobytes())
    return h.hexdigest()


__all__ = ["MAX_LEN", "THETA_LO", "THETA_HI", "THETA_MID", "DEFAULT_COST", "Pool", "make_pool",
           "config", "Streaming", "adversarial", "ADVERSARIAL_KINDS", "digest"]
