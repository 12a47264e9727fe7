"""CPU oracle for the EWSJF scheduler core -- TEST INFRASTRUCTURE ONLY.

Thin numpy/ctypes wrapper around ``libewsjf_oracle.so`` (built from
``ewsjf_oracle.cpp`` by ``oracle/build.py``).  Only the tests, the smoke
check and the benchmark's CPU-baseline leg use it; the product path never
does.  It shares no code with the HIP library.
"""
from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.environ.get("EWSJF_ORACLE_LIB") or os.path.join(HERE, "libewsjf_oracle.so")

EQUAL_WIDTH = 0
KMEANS3 = 1

_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            from . import build as _b  # noqa: PLC0415
            _b.build()
        _lib = C.CDLL(LIB_PATH)
        _declare(_lib)
    return _lib


def _p(t):
    return C.POINTER(t)


def _declare(L):
    i32, i64, f32, f64 = C.c_int32, C.c_int64, C.c_float, C.c_double
    L.oracle_distinct.argtypes = [_p(i32), i64, i32, _p(i32), _p(i64)]
    L.oracle_distinct.restype = i64
    L.oracle_stage1.argtypes = [_p(i32), _p(i64), i32, i32, i32, _p(i32)]
    L.oracle_stage1.restype = i32
    L.oracle_stage2.argtypes = [_p(i32), _p(i64), i32, _p(i32), i32, f64, i32, i32, _p(i32)]
    L.oracle_stage2.restype = i32
    L.oracle_stage3.argtypes = [_p(i64), _p(i64), _p(i32), _p(i32), i32, i32, f64,
                                _p(i64), _p(i64), _p(i32), _p(i32)]
    L.oracle_stage3.restype = i32
    L.oracle_partition.argtypes = [_p(i32), i64, i32, i32, i32, i32, i32, f64, f64, i32,
                                   _p(i32), _p(i32), _p(i64), _p(i64), _p(i32), _p(i32), _p(f64),
                                   _p(i32)]
    L.oracle_partition.restype = C.c_int
    L.oracle_route.argtypes = [_p(i32), i64, _p(i32), i32, _p(i32)]
    L.oracle_route.restype = None
    L.oracle_route_gapped.argtypes = [_p(i32), i64, _p(i32), _p(i32), i32, _p(i32)]
    L.oracle_route_gapped.restype = None
    L.oracle_score.argtypes = [_p(i32), _p(f32), i64, f32, i32, _p(i32), _p(i32), _p(i32), i32, _p(f64), _p(f32),
                               i32, f64, f64, f64, _p(f32)]
    L.oracle_score.restype = None
    L.oracle_select.argtypes = [_p(f32), i64, i32, i32, _p(i32), _p(f32), _p(i32)]
    L.oracle_select.restype = None
    L.oracle_tactical_step.argtypes = [_p(i32), _p(f32), i64, f32, _p(i32), _p(i32), _p(i64), _p(i64), _p(i32),
                                       _p(i32), _p(f64), _p(i32), i32, _p(f32), f64, f64, f64, i32, i32, f64,
                                       _p(i32), _p(i32), _p(i32), _p(f32), _p(i32)]
    L.oracle_tactical_step.restype = C.c_int
    L.oracle_dispatch.argtypes = [_p(i32), _p(f32), i64, _p(i32), _p(i32), _p(i64), _p(i64), _p(i32), _p(i32),
                                  _p(f64), i32, i32, _p(i32)]
    L.oracle_dispatch.restype = C.c_int


def _ptr(a, t):
    return a.ctypes.data_as(C.POINTER(t))


def _arr(a, dtype):
    return np.ascontiguousarray(np.asarray(a, dtype=dtype))


@dataclass
class Table:
    """Queue table: k intervals in length order; bounds[i] = lo of queue i+1.
    Routing reads them as a contiguous cover of bounds, or (gapped, after a
    dispatch with bubble queues) as the lengths [lo_i, hi_i] of each queue
    with Algorithm 2's rule in the gaps."""
    k: int
    bounds: np.ndarray   # int32 [k-1]
    count: np.ndarray    # int64 [k]
    sum: np.ndarray      # int64 [k]
    lo: np.ndarray       # int32 [k]
    hi: np.ndarray       # int32 [k]
    mean: np.ndarray     # float64 [k]
    n_distinct: int = 0
    n_coarse: int = 0
    n_leaves: int = 0
    gapped: bool = False


@dataclass
class PartitionParams:
    init_mode: int = EQUAL_WIDTH
    init_queues: int = 16
    max_queues: int = 16
    min_width: int = 16
    max_len: int = 32768
    alpha: float = 2.0
    eps: float = 1e-6
    gap_mode: int = 0


def distinct(window, max_len=32768):
    w = _arr(window, np.int32)
    v = np.zeros(max(1, w.size), np.int32)
    c = np.zeros(max(1, w.size), np.int64)
    V = lib().oracle_distinct(_ptr(w, C.c_int32), w.size, max_len, _ptr(v, C.c_int32), _ptr(c, C.c_int64))
    if V < 0:
        raise ValueError("bad arguments")
    return v[:V].copy(), c[:V].copy()


def stage1(v, c, init_mode=EQUAL_WIDTH, init_queues=16):
    v, c = _arr(v, np.int32), _arr(c, np.int64)
    out = np.zeros(max(3, v.size), np.int32)
    r = lib().oracle_stage1(_ptr(v, C.c_int32), _ptr(c, C.c_int64), v.size, init_mode, init_queues,
                            _ptr(out, C.c_int32))
    if r < 0:
        raise ValueError("bad arguments")
    return out[:r].copy()


def stage2(v, c, coarse_starts, alpha=2.0, min_width=16, gap_mode=0):
    v, c = _arr(v, np.int32), _arr(c, np.int64)
    cs = _arr(coarse_starts, np.int32)
    out = np.zeros(max(1, v.size), np.int32)
    r = lib().oracle_stage2(_ptr(v, C.c_int32), _ptr(c, C.c_int64), v.size, _ptr(cs, C.c_int32), cs.size,
                            alpha, min_width, gap_mode, _ptr(out, C.c_int32))
    if r < 0:
        raise ValueError("bad arguments")
    return out[:r].copy()


def stage3(n, S, lo, hi, max_queues, eps=1e-6):
    n, S = _arr(n, np.int64), _arr(S, np.int64)
    lo, hi = _arr(lo, np.int32), _arr(hi, np.int32)
    m = n.size
    no, So = np.zeros(m, np.int64), np.zeros(m, np.int64)
    loo, hio = np.zeros(m, np.int32), np.zeros(m, np.int32)
    k = lib().oracle_stage3(_ptr(n, C.c_int64), _ptr(S, C.c_int64), _ptr(lo, C.c_int32), _ptr(hi, C.c_int32),
                            m, max_queues, eps, _ptr(no, C.c_int64), _ptr(So, C.c_int64),
                            _ptr(loo, C.c_int32), _ptr(hio, C.c_int32))
    if k < 0:
        raise ValueError("bad arguments")
    return no[:k].copy(), So[:k].copy(), loo[:k].copy(), hio[:k].copy()


def partition(window, p: PartitionParams | None = None, **kw) -> Table:
    p = p or PartitionParams()
    for key, val in kw.items():
        setattr(p, key, val)
    w = _arr(window, np.int32)
    cap = max(1, p.max_queues)
    k = np.zeros(1, np.int32)
    bounds = np.zeros(cap, np.int32)
    count, ssum = np.zeros(cap, np.int64), np.zeros(cap, np.int64)
    lo, hi = np.zeros(cap, np.int32), np.zeros(cap, np.int32)
    mean = np.zeros(cap, np.float64)
    diag = np.zeros(3, np.int32)
    r = lib().oracle_partition(_ptr(w, C.c_int32), w.size, p.init_mode, p.init_queues, p.max_queues,
                               p.min_width, p.max_len, p.alpha, p.eps, p.gap_mode, _ptr(k, C.c_int32),
                               _ptr(bounds, C.c_int32), _ptr(count, C.c_int64), _ptr(ssum, C.c_int64),
                               _ptr(lo, C.c_int32), _ptr(hi, C.c_int32), _ptr(mean, C.c_double),
                               _ptr(diag, C.c_int32))
    if r != 0:
        raise ValueError("bad partition arguments")
    kk = int(k[0])
    return Table(kk, bounds[:kk - 1].copy(), count[:kk].copy(), ssum[:kk].copy(), lo[:kk].copy(),
                 hi[:kk].copy(), mean[:kk].copy(), int(diag[0]), int(diag[1]), int(diag[2]))


def route(length, table_or_bounds):
    L = _arr(length, np.int32)
    q = np.zeros(L.size, np.int32)
    if isinstance(table_or_bounds, Table) and table_or_bounds.gapped:
        t = table_or_bounds
        lo, hi = _arr(t.lo, np.int32), _arr(t.hi, np.int32)
        lib().oracle_route_gapped(_ptr(L, C.c_int32), L.size, _ptr(lo, C.c_int32), _ptr(hi, C.c_int32), t.k,
                                  _ptr(q, C.c_int32))
        return q
    bounds = table_or_bounds.bounds if isinstance(table_or_bounds, Table) else table_or_bounds
    b = _arr(bounds, np.int32)
    lib().oracle_route(_ptr(L, C.c_int32), L.size, _ptr(b, C.c_int32), b.size + 1, _ptr(q, C.c_int32))
    return q


def dispatch(length, arrival, table: Table, bubble_width: int, max_queues: int):
    """The Dispatcher with on-demand bubble queues (Algorithm 2) over the
    requests with length > 0 in arrival order: (qid per request in the final
    queue set, the gapped table after the bubbles)."""
    L = _arr(length, np.int32)
    A = _arr(arrival, np.float32)
    cap = max(int(max_queues), table.k)
    k = np.array([table.k], np.int32)
    bounds = np.zeros(cap, np.int32)
    count, ssum = np.zeros(cap, np.int64), np.zeros(cap, np.int64)
    lo, hi = np.zeros(cap, np.int32), np.zeros(cap, np.int32)
    mean = np.zeros(cap, np.float64)
    count[:table.k], ssum[:table.k] = table.count, table.sum
    lo[:table.k], hi[:table.k], mean[:table.k] = table.lo, table.hi, table.mean
    qid = np.zeros(L.size, np.int32)
    r = lib().oracle_dispatch(_ptr(L, C.c_int32), _ptr(A, C.c_float), L.size, _ptr(k, C.c_int32),
                              _ptr(bounds, C.c_int32), _ptr(count, C.c_int64), _ptr(ssum, C.c_int64),
                              _ptr(lo, C.c_int32), _ptr(hi, C.c_int32), _ptr(mean, C.c_double), int(bubble_width),
                              int(max_queues), _ptr(qid, C.c_int32))
    if r != 0:
        raise ValueError("bad dispatch arguments")
    kk = int(k[0])
    t2 = Table(kk, bounds[:kk - 1].copy(), count[:kk].copy(), ssum[:kk].copy(), lo[:kk].copy(), hi[:kk].copy(),
               mean[:kk].copy(), table.n_distinct, table.n_coarse, table.n_leaves, True)
    return qid, t2


def score(length, arrival, now, table: Table, theta, cost=(0.01, 1e-4, 0.0)):
    L = _arr(length, np.int32)
    A = _arr(arrival, np.float32)
    th = _arr(theta, np.float32).reshape(-1, 6)
    b = np.zeros(max(1, table.k - 1), np.int32)
    b[:table.k - 1] = table.bounds
    lo, hi = _arr(table.lo, np.int32), _arr(table.hi, np.int32)
    m = _arr(table.mean, np.float64)
    out = np.zeros((th.shape[0], L.size), np.float32)
    lib().oracle_score(_ptr(L, C.c_int32), _ptr(A, C.c_float), L.size, float(np.float32(now)), table.k,
                       _ptr(b, C.c_int32), _ptr(lo, C.c_int32), _ptr(hi, C.c_int32), int(table.gapped),
                       _ptr(m, C.c_double), _ptr(th, C.c_float), th.shape[0], float(cost[0]), float(cost[1]),
                       float(cost[2]), _ptr(out, C.c_float))
    return out


def select(scores, B):
    s = _arr(scores, np.float32)
    if s.ndim == 1:
        s = s.reshape(1, -1)
    nt, n = s.shape
    ids = np.zeros((nt, B), np.int32)
    top = np.zeros((nt, B), np.float32)
    nsel = np.zeros(nt, np.int32)
    lib().oracle_select(_ptr(s, C.c_float), n, nt, B, _ptr(ids, C.c_int32), _ptr(top, C.c_float),
                        _ptr(nsel, C.c_int32))
    return ids, top, nsel


def step(length, arrival, now, table: Table, theta, B, cost=(0.01, 1e-4, 0.0)):
    """Route, score and select: returns (ids, top, n_sel, scores)."""
    sc = score(length, arrival, now, table, theta, cost)
    ids, top, nsel = select(sc, B)
    return ids, top, nsel, sc


@dataclass
class TacticalResult:
    ids: np.ndarray         # int32 [n_sel], batch order
    q_prim: int             # -1 when every queue is empty
    head_score: np.ndarray  # float32 [k at entry], NaN for empty queues
    removed: np.ndarray     # bool [k at entry]
    table: Table            # after this step's removals
    empty_cnt: np.ndarray   # int32 [k after removals]


def tactical_step(length, arrival, now, table: Table, empty_cnt, theta, B, empty_threshold,
                  cost=(0.01, 1e-4, 0.0), eps=1e-6) -> TacticalResult:
    """One step of Algorithm 1 (Section 3.2): ArgMax queue, GreedyFill,
    Backfill from adjacent queues, EmptyThreshold removal."""
    L = _arr(length, np.int32)
    A = _arr(arrival, np.float32)
    k0 = int(table.k)
    k = np.array([k0], np.int32)
    bounds = np.zeros(max(1, k0), np.int32)
    bounds[:k0 - 1] = table.bounds
    count, ssum = _arr(table.count, np.int64).copy(), _arr(table.sum, np.int64).copy()
    lo, hi = _arr(table.lo, np.int32).copy(), _arr(table.hi, np.int32).copy()
    mean = _arr(table.mean, np.float64).copy()
    ec = _arr(empty_cnt, np.int32).copy()
    if ec.size != k0:
        raise ValueError("empty_cnt needs one entry per queue")
    th = _arr(theta, np.float32).reshape(6)
    ids = np.zeros(max(1, B), np.int32)
    nsel = np.zeros(1, np.int32)
    qp = np.zeros(1, np.int32)
    hs = np.zeros(k0, np.float32)
    rm = np.zeros(k0, np.int32)
    r = lib().oracle_tactical_step(_ptr(L, C.c_int32), _ptr(A, C.c_float), L.size, float(np.float32(now)),
                                   _ptr(k, C.c_int32), _ptr(bounds, C.c_int32), _ptr(count, C.c_int64),
                                   _ptr(ssum, C.c_int64), _ptr(lo, C.c_int32), _ptr(hi, C.c_int32),
                                   _ptr(mean, C.c_double), _ptr(ec, C.c_int32), int(table.gapped),
                                   _ptr(th, C.c_float),
                                   float(cost[0]), float(cost[1]), float(cost[2]), int(B), int(empty_threshold),
                                   float(eps), _ptr(ids, C.c_int32), _ptr(nsel, C.c_int32), _ptr(qp, C.c_int32),
                                   _ptr(hs, C.c_float), _ptr(rm, C.c_int32))
    if r != 0:
        raise ValueError("bad tactical-step arguments")
    k1 = int(k[0])
    t2 = Table(k1, bounds[:k1 - 1].copy(), count[:k1].copy(), ssum[:k1].copy(), lo[:k1].copy(), hi[:k1].copy(),
               mean[:k1].copy(), table.n_distinct, table.n_coarse, table.n_leaves, table.gapped)
    return TacticalResult(ids[:int(nsel[0])].copy(), int(qp[0]), hs, rm.astype(bool), t2, ec[:k1].copy())
