"""Thin PyTorch binding of the EWSJF C ABI (include/ewsjf.h).

Each function checks tensor dtypes and devices, passes raw device pointers
and the current HIP stream to libewsjf.so and returns output tensors.  All
computation happens in the library's HIP kernels.
"""
from __future__ import annotations

import ctypes as C

import numpy as np
import torch

from . import _lib as L

DEFAULT_COST = (0.01, 1e-4, 0.0)


def _vp(t: torch.Tensor) -> C.c_void_p:
    return C.c_void_p(t.data_ptr())


def _stream(stream=None) -> C.c_void_p:
    s = stream if stream is not None else torch.cuda.current_stream()
    return C.c_void_p(s.cuda_stream)


def _need(t: torch.Tensor, dtype: torch.dtype, name: str) -> torch.Tensor:
    if not isinstance(t, torch.Tensor) or t.dtype != dtype or not t.is_cuda or not t.is_contiguous():
        raise TypeError(f"{name} must be a contiguous CUDA tensor of {dtype}")
    return t


def params(init_mode: int = L.INIT_EQUAL_WIDTH, init_queues: int = 16, max_queues: int = 16,
           min_width: int = 16, max_len: int = L.MAX_LEN, gap_mode: int = L.GAPS_DISTINCT,
           alpha: float = 2.0, eps: float = 1e-6) -> L.PartitionParams:
    return L.PartitionParams(init_mode, init_queues, max_queues, min_width, max_len, gap_mode, alpha, eps)


def cost(c0: float = DEFAULT_COST[0], c1: float = DEFAULT_COST[1], c2: float = DEFAULT_COST[2]) -> L.Cost:
    return L.Cost(c0, c1, c2)


def _cost(c) -> L.Cost:
    if isinstance(c, L.Cost):
        return c
    return L.Cost(*[float(x) for x in c])


def table_bytes() -> int:
    return int(L.lib().ewsjf_queue_table_bytes())


def workspace_bytes(op: int, n: int, n_theta: int = 1, B: int = 1, p: L.PartitionParams | None = None) -> int:
    pp = C.byref(p) if p is not None else None
    return int(L.lib().ewsjf_workspace_bytes(op, int(n), int(n_theta), int(B), pp))


class Workspace:
    """A growable device scratch buffer for the calls that need one."""

    def __init__(self, device=None):
        self.device = torch.device(device or "cuda")
        self.buf = None

    def get(self, nbytes: int) -> torch.Tensor:
        nbytes = max(256, int(nbytes))
        if self.buf is None or self.buf.numel() < nbytes:
            self.buf = torch.empty(nbytes, dtype=torch.uint8, device=self.device)
        return self.buf


def new_table(device=None) -> torch.Tensor:
    return torch.zeros(table_bytes(), dtype=torch.uint8, device=device or "cuda")


def partition(window: torch.Tensor, p: L.PartitionParams, table: torch.Tensor | None = None,
              ws: Workspace | None = None, stream=None) -> torch.Tensor:
    """Refine-and-Prune over `window` (int32 lengths) -> device queue table."""
    _need(window, torch.int32, "window")
    table = table if table is not None else new_table(window.device)
    ws = ws or Workspace(window.device)
    need = workspace_bytes(L.OP_PARTITION, window.numel(), p=p)
    buf = ws.get(need)
    L.check(L.lib().ewsjf_partition(_vp(window), window.numel(), C.byref(p), _vp(table), _vp(buf), buf.numel(),
                                    _stream(stream)), "ewsjf_partition")
    return table


def window_histogram(ring: torch.Tensor, max_len: int, hist: torch.Tensor | None = None, begin: int = 0,
                     n: int | None = None, stream=None) -> torch.Tensor:
    """Histogram of the window ring[(begin + i) mod len(ring)], i < n (the
    whole array by default), lengths clamped to [1, max_len]: int32
    [max_len + 1] (the library's uint32 counts, bit for bit), hist[0] = 0."""
    _need(ring, torch.int32, "ring")
    n = ring.numel() if n is None else int(n)
    if hist is None:
        hist = torch.empty(int(max_len) + 1, dtype=torch.int32, device=ring.device)
    _need(hist, torch.int32, "hist")
    if hist.numel() != int(max_len) + 1:
        raise ValueError("hist needs max_len + 1 entries")
    L.check(L.lib().ewsjf_window_histogram(_vp(ring), ring.numel(), int(begin), n, int(max_len), _vp(hist),
                                           _stream(stream)), "ewsjf_window_histogram")
    return hist


def window_advance(ring: torch.Tensor, add_pos: int, sub_pos: int, n: int, hist: torch.Tensor, stream=None) -> None:
    """Move the window's histogram (int32 [max_len + 1]) forward by n entries:
    the counts of ring[(sub_pos + i) mod len(ring)] go to ring[(add_pos + i)
    mod len(ring)], i < n."""
    _need(ring, torch.int32, "ring")
    _need(hist, torch.int32, "hist")
    L.check(L.lib().ewsjf_window_advance(_vp(ring), ring.numel(), int(add_pos), int(sub_pos), int(n),
                                         hist.numel() - 1, _vp(hist), _stream(stream)), "ewsjf_window_advance")


def partition_hist(hist: torch.Tensor, p: L.PartitionParams, table: torch.Tensor | None = None,
                   ws: Workspace | None = None, stream=None) -> torch.Tensor:
    """Refine-and-Prune from a window histogram (int32 [p.max_len + 1]) ->
    device queue table, identical to partition() over the window."""
    _need(hist, torch.int32, "hist")
    if hist.numel() != p.max_len + 1:
        raise ValueError("hist needs p.max_len + 1 entries")
    table = table if table is not None else new_table(hist.device)
    ws = ws or Workspace(hist.device)
    buf = ws.get(workspace_bytes(L.OP_PARTITION, 0, p=p))
    L.check(L.lib().ewsjf_partition_hist(_vp(hist), C.byref(p), _vp(table), _vp(buf), buf.numel(), _stream(stream)),
            "ewsjf_partition_hist")
    return table


def trial_step(len_pools: torch.Tensor, arr_pools: torch.Tensor, pos: int, new_len: torch.Tensor,
               new_arrival: torch.Tensor, now: float, table: torch.Tensor, theta: torch.Tensor, B: int,
               stats: torch.Tensor, queue_admits: torch.Tensor, cost_=DEFAULT_COST, out=None,
               ws: Workspace | None = None, stream=None):
    """One step of a trial for every proposal (ewsjf_trial_step): pools are
    [P][capacity]; stats float64 [P][8] and queue_admits int64 [P][256]
    accumulate.  Returns (ids[P,B], top[P,B], n_sel[P])."""
    _need(len_pools, torch.int32, "len_pools")
    _need(arr_pools, torch.float32, "arr_pools")
    _need(new_len, torch.int32, "new_len")
    _need(new_arrival, torch.float32, "new_arrival")
    _need(stats, torch.float64, "stats")
    _need(queue_admits, torch.int64, "queue_admits")
    P, cap = len_pools.shape
    theta = _theta(theta)
    if theta.shape[0] != P or stats.shape != (P, L.TRIAL_STATS) or queue_admits.shape != (P, L.MAX_QUEUES):
        raise ValueError("one parameter vector, one statistics row and one queue row per pool")
    ids, top, nsel = _outs(P, B, len_pools.device, out)
    ws = ws or Workspace(len_pools.device)
    buf = ws.get(workspace_bytes(L.OP_TRIAL, cap, P, B))
    c = _cost(cost_)
    L.check(L.lib().ewsjf_trial_step(_vp(len_pools), _vp(arr_pools), cap, P, int(pos), _vp(new_len),
                                     _vp(new_arrival), new_len.numel(), float(now), _vp(table), _vp(theta),
                                     C.byref(c), int(B), _vp(ids), _vp(top), _vp(nsel), _vp(stats),
                                     _vp(queue_admits), _vp(buf), buf.numel(), _stream(stream)), "ewsjf_trial_step")
    return ids, top, nsel


def trial_finish(len_pools: torch.Tensor, arr_pools: torch.Tensor, now: float, table: torch.Tensor,
                 stats: torch.Tensor, queue_admits: torch.Tensor, lam=(1.0, 1.0, 1.0, 1.0), reward=None,
                 stream=None) -> torch.Tensor:
    """The trial's end (ewsjf_trial_finish): pending statistics into stats,
    Eq. 5 per pool (float64 [P])."""
    _need(len_pools, torch.int32, "len_pools")
    _need(arr_pools, torch.float32, "arr_pools")
    P, cap = len_pools.shape
    reward = reward if reward is not None else torch.empty(P, dtype=torch.float64, device=len_pools.device)
    lam_h = (C.c_double * 4)(*[float(x) for x in lam])
    L.check(L.lib().ewsjf_trial_finish(_vp(len_pools), _vp(arr_pools), cap, P, float(now), _vp(table),
                                       _vp(queue_admits), lam_h, _vp(stats), _vp(reward), _stream(stream)),
            "ewsjf_trial_finish")
    return reward


def dispatch(length: torch.Tensor, arrival: torch.Tensor, table: torch.Tensor, bubble_width: int, max_queues: int,
             qid: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """The Dispatcher with on-demand bubble queues (ewsjf_dispatch): int32
    queue of each request in the updated (gapped) table, -1 for empty slots."""
    _need(length, torch.int32, "length")
    _need(arrival, torch.float32, "arrival")
    if arrival.numel() != length.numel():
        raise ValueError("length and arrival differ in size")
    qid = qid if qid is not None else torch.empty_like(length)
    L.check(L.lib().ewsjf_dispatch(_vp(length), _vp(arrival), length.numel(), _vp(table), int(bubble_width),
                                   int(max_queues), _vp(qid), _stream(stream)), "ewsjf_dispatch")
    return qid


def upload_table(bounds, mean, max_len: int = L.MAX_LEN, lo=None, hi=None, count=None, sum=None,
                 device=None, stream=None, gapped: bool = False) -> torch.Tensor:
    """Install a queue structure given on the host (bounds: k-1 ints, mean: k
    floats; gapped: route by the lo/hi intervals).  Without lo/hi, each
    queue's lo/hi are its routing interval (queue 0 from length 1, the last
    queue up to max_len)."""
    bounds = np.asarray(bounds, np.int64).reshape(-1)
    mean = np.asarray(mean, np.float64).reshape(-1)
    k = mean.size
    if bounds.size != k - 1:
        raise ValueError("need k-1 bounds for k means")
    if lo is None:
        lo = np.concatenate([[1], bounds])
    if hi is None:
        hi = np.concatenate([bounds - 1, [max_len]])
    h = L.QueueTable()
    h.k, h.max_len, h.gapped = k, int(max_len), int(bool(gapped))
    for i, b in enumerate(bounds):
        h.bounds[i] = int(b)
    for i in range(k):
        h.mean[i] = float(mean[i])
        h.lo[i] = int(lo[i]) if lo is not None else 0
        h.hi[i] = int(hi[i]) if hi is not None else 0
        h.count[i] = int(count[i]) if count is not None else 0
        h.sum[i] = int(sum[i]) if sum is not None else 0
    table = new_table(device)
    L.check(L.lib().ewsjf_table_upload(C.byref(h), _vp(table), _stream(stream)), "ewsjf_table_upload")
    return table


def read_table(table: torch.Tensor) -> dict:
    """Copy a device queue table to the host and decode it."""
    raw = table.detach().to("cpu").numpy().tobytes()
    h = L.QueueTable.from_buffer_copy(raw[:C.sizeof(L.QueueTable)])
    k = h.k
    return {
        "k": k, "max_len": h.max_len, "n_distinct": h.n_distinct, "n_coarse": h.n_coarse,
        "n_leaves": h.n_leaves, "n_window": h.n_window, "gapped": bool(h.gapped),
        "bounds": np.array(h.bounds[:max(k - 1, 0)], np.int32),
        "lo": np.array(h.lo[:k], np.int32), "hi": np.array(h.hi[:k], np.int32),
        "count": np.array(h.count[:k], np.int64), "sum": np.array(h.sum[:k], np.int64),
        "mean": np.array(h.mean[:k], np.float64),
        "lut": np.frombuffer(bytes(h.lut), np.uint8)[:h.max_len + 1].copy(),
        "route": np.frombuffer(bytes(h.route), np.uint64).copy(),
    }


def route_map_queues(route: np.ndarray, max_len: int) -> np.ndarray:
    """Decode a table's compact routing map: the queue of every length
    0..max_len (length 0 decodes to 0), as the per-step kernels read it."""
    b = np.arange(max_len + 1, dtype=np.int64)
    w = route[b >> 5]
    base = (w >> np.uint64(32)).astype(np.int64)
    mask = (w & np.uint64(0xFFFFFFFF)).astype(np.uint64)
    keep = (mask << (np.uint64(31) - (b & 31).astype(np.uint64))) & np.uint64(0xFFFFFFFF)
    bits = np.unpackbits(keep.astype(">u4").view(np.uint8).reshape(-1, 4), axis=1).sum(axis=1)
    return (base + bits).astype(np.int64)


def route(length: torch.Tensor, table: torch.Tensor, out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    _need(length, torch.int32, "length")
    out = out if out is not None else torch.empty_like(length)
    L.check(L.lib().ewsjf_route(_vp(length), length.numel(), _vp(table), _vp(out), _stream(stream)), "ewsjf_route")
    return out


def _theta(theta: torch.Tensor) -> torch.Tensor:
    _need(theta, torch.float32, "theta")
    if theta.dim() == 1:
        theta = theta.reshape(1, -1)
    if theta.shape[-1] != 6:
        raise ValueError("theta rows are (a_base, b_base, a_urg, b_urg, a_fair, b_fair)")
    return theta


def score(length: torch.Tensor, arrival: torch.Tensor, now: float, table: torch.Tensor, theta: torch.Tensor,
          cost_=DEFAULT_COST, out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    _need(length, torch.int32, "length")
    _need(arrival, torch.float32, "arrival")
    theta = _theta(theta)
    n, nt = length.numel(), theta.shape[0]
    out = out if out is not None else torch.empty((nt, n), dtype=torch.float32, device=length.device)
    c = _cost(cost_)
    L.check(L.lib().ewsjf_score(_vp(length), _vp(arrival), n, float(now), _vp(table), _vp(theta), nt, C.byref(c),
                                _vp(out), _stream(stream)), "ewsjf_score")
    return out


def _outs(nt: int, B: int, device, out):
    if out is not None:
        return out
    ids = torch.empty((nt, B), dtype=torch.int32, device=device)
    top = torch.empty((nt, B), dtype=torch.float32, device=device)
    nsel = torch.empty((nt,), dtype=torch.int32, device=device)
    return ids, top, nsel


def select(scores: torch.Tensor, B: int, out=None, ws: Workspace | None = None, stream=None):
    _need(scores, torch.float32, "scores")
    if scores.dim() == 1:
        scores = scores.reshape(1, -1)
    nt, n = scores.shape
    ids, top, nsel = _outs(nt, B, scores.device, out)
    ws = ws or Workspace(scores.device)
    buf = ws.get(workspace_bytes(L.OP_SELECT, n, nt, B))
    L.check(L.lib().ewsjf_select(_vp(scores), n, nt, int(B), _vp(ids), _vp(top), _vp(nsel), _vp(buf), buf.numel(),
                                 _stream(stream)), "ewsjf_select")
    return ids, top, nsel


def step(length: torch.Tensor, arrival: torch.Tensor, now: float, table: torch.Tensor, theta: torch.Tensor, B: int,
         cost_=DEFAULT_COST, tombstone: bool = False, out=None, ws: Workspace | None = None, stream=None):
    """One fused scheduling step: route + score + top-B admission."""
    _need(length, torch.int32, "length")
    _need(arrival, torch.float32, "arrival")
    theta = _theta(theta)
    n, nt = length.numel(), theta.shape[0]
    ids, top, nsel = _outs(nt, B, length.device, out)
    ws = ws or Workspace(length.device)
    buf = ws.get(workspace_bytes(L.OP_STEP, n, nt, B))
    c = _cost(cost_)
    flags = L.STEP_TOMBSTONE if tombstone else 0
    L.check(L.lib().ewsjf_step(_vp(length), _vp(arrival), n, float(now), _vp(table), _vp(theta), nt, C.byref(c),
                               int(B), flags, _vp(ids), _vp(top), _vp(nsel), _vp(buf), buf.numel(), _stream(stream)),
            "ewsjf_step")
    return ids, top, nsel


def step_static(length: torch.Tensor, arrival: torch.Tensor, now: float, table: torch.Tensor, theta: torch.Tensor,
                B: int, cost_=DEFAULT_COST, tombstone: bool = False, out=None, stream=None):
    """ewsjf_step with the library's fixed per-device scratch (no workspace,
    no allocation in the call; the outputs are allocated here unless given)."""
    _need(length, torch.int32, "length")
    _need(arrival, torch.float32, "arrival")
    th = _theta(theta)
    nt, n = th.shape[0], length.numel()
    ids, top, nsel = _outs(nt, B, length.device, out)
    c = _cost(cost_)
    L.check(L.lib().ewsjf_step_static(_vp(length), _vp(arrival), n, float(now), _vp(table), _vp(th), nt, C.byref(c),
                                      int(B), L.STEP_TOMBSTONE if tombstone else 0, _vp(ids), _vp(top), _vp(nsel),
                                      _stream(stream)), "ewsjf_step_static")
    return ids, top, nsel


def ring_step(ring_len: torch.Tensor, ring_arrival: torch.Tensor, pos: int, new_len: torch.Tensor,
              new_arrival: torch.Tensor, now: float, table: torch.Tensor, theta: torch.Tensor, B: int,
              cost_=DEFAULT_COST, window: torch.Tensor | None = None, wpos: int = 0, tombstone: bool = False, out=None,
              ws: Workspace | None = None, stream=None):
    """ring_insert + step (one vector) fused (ewsjf_ring_step)."""
    _need(ring_len, torch.int32, "ring_len")
    _need(ring_arrival, torch.float32, "ring_arrival")
    _need(new_len, torch.int32, "new_len")
    _need(new_arrival, torch.float32, "new_arrival")
    if window is not None:
        _need(window, torch.int32, "window")
    theta = _theta(theta)
    if theta.shape[0] != 1:
        raise ValueError("ring_step takes one parameter vector")
    cap = ring_len.numel()
    ids, top, nsel = _outs(1, B, ring_len.device, out)
    ws = ws or Workspace(ring_len.device)
    buf = ws.get(workspace_bytes(L.OP_STEP, cap, 1, B))
    c = _cost(cost_)
    wp, wc = (_vp(window), window.numel()) if window is not None else (None, 0)
    flags = L.STEP_TOMBSTONE if tombstone else 0
    L.check(L.lib().ewsjf_ring_step(_vp(ring_len), _vp(ring_arrival), cap, int(pos), wp, wc, int(wpos),
                                    _vp(new_len), _vp(new_arrival), new_len.numel(), float(now), _vp(table),
                                    _vp(theta), C.byref(c), int(B), flags, _vp(ids), _vp(top), _vp(nsel), _vp(buf),
                                    buf.numel(), _stream(stream)),
            "ewsjf_ring_step")
    return ids, top, nsel


def new_empty_counters(device=None) -> torch.Tensor:
    """Per-queue empty-step counters for tactical_step (zero for a new table)."""
    return torch.zeros(L.MAX_QUEUES, dtype=torch.int32, device=device)


def tactical_step(length: torch.Tensor, arrival: torch.Tensor, now: float, table: torch.Tensor, theta: torch.Tensor,
                  B: int, empty_threshold: int, empty_cnt: torch.Tensor, eps: float = 1e-6, cost_=DEFAULT_COST,
                  tombstone: bool = False, ws: Workspace | None = None, stream=None):
    """One step of Algorithm 1 (ewsjf_tactical_step): returns ids[B] (batch
    order), n_sel[1], q_prim[1], head_score[MAX_QUEUES], removed[MAX_QUEUES].
    The table and empty_cnt are updated in place."""
    _need(length, torch.int32, "length")
    _need(arrival, torch.float32, "arrival")
    _need(empty_cnt, torch.int32, "empty_cnt")
    theta = _theta(theta)
    if theta.shape[0] != 1:
        raise ValueError("tactical_step takes one parameter vector")
    n, dev = length.numel(), length.device
    ids = torch.empty(B, dtype=torch.int32, device=dev)
    nsel = torch.empty(1, dtype=torch.int32, device=dev)
    qp = torch.empty(1, dtype=torch.int32, device=dev)
    hs = torch.empty(L.MAX_QUEUES, dtype=torch.float32, device=dev)
    rm = torch.empty(L.MAX_QUEUES, dtype=torch.int32, device=dev)
    ws = ws or Workspace(dev)
    buf = ws.get(workspace_bytes(L.OP_TACTICAL, n, 1, B))
    c = _cost(cost_)
    flags = L.STEP_TOMBSTONE if tombstone else 0
    L.check(L.lib().ewsjf_tactical_step(_vp(length), _vp(arrival), n, float(now), _vp(table), _vp(theta), C.byref(c),
                                        int(B), int(empty_threshold), _vp(empty_cnt), float(eps), flags, _vp(ids),
                                        _vp(nsel), _vp(qp), _vp(hs), _vp(rm), _vp(buf), buf.numel(),
                                        _stream(stream)),
            "ewsjf_tactical_step")
    return ids, nsel, qp, hs, rm


def ring_insert(ring_len: torch.Tensor, ring_arrival: torch.Tensor, pos: int, new_len: torch.Tensor,
                new_arrival: torch.Tensor, window: torch.Tensor | None = None, wpos: int = 0, stream=None) -> None:
    """Write new requests into ring slots (pos + i) mod capacity and their
    lengths into window slots (wpos + i) mod len(window), in one launch."""
    _need(ring_len, torch.int32, "ring_len")
    _need(ring_arrival, torch.float32, "ring_arrival")
    _need(new_len, torch.int32, "new_len")
    _need(new_arrival, torch.float32, "new_arrival")
    if window is not None:
        _need(window, torch.int32, "window")
    wv = _vp(window) if window is not None else C.c_void_p(None)
    wc = window.numel() if window is not None else 0
    L.check(L.lib().ewsjf_ring_insert(_vp(ring_len), _vp(ring_arrival), ring_len.numel(), int(pos), wv, wc,
                                      int(wpos), _vp(new_len), _vp(new_arrival), new_len.numel(), _stream(stream)),
            "ewsjf_ring_insert")
