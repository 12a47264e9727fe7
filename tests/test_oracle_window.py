"""Pins of the oracle's Refine-and-Prune as a function of the window's
multiset of clamped lengths, the property the sliding-window partitioner
rests on: Section 4.2 sorts the window and then reads only the sorted
sequence, so any order of the same lengths, and the window rebuilt from its
histogram, give the same queue table."""
import numpy as np
import pytest

import oracle
from paper_2601_21758_amd import workloads as W

CASES = [
    ("cfg0", lambda: W.config(0).window, dict(init_queues=16, max_queues=16)),
    ("cfg1_multiset", lambda: W.config(1).window[:40000], dict(init_queues=64, max_queues=64, gap_mode=1)),
    ("kmeans3", lambda: W.make_pool("three", 3000, 61, arrivals="uniform").window,
     dict(init_mode=oracle.KMEANS3, max_queues=32)),
    ("many_leaves", lambda: np.cumsum(np.random.default_rng(3).integers(1, 40, 3000)).astype(np.int32) % 32768 + 1,
     dict(init_queues=1, max_queues=50, min_width=0, alpha=1.05)),
    ("clamped", lambda: np.array([-5, 0, 1, 40000, 32768, 7, 7, 100000, 2000, 2001], np.int32),
     dict(init_queues=4, max_queues=4, min_width=0)),
    ("max_len_1000", lambda: W.config(0).window[:20000], dict(init_queues=16, max_queues=16, max_len=1000)),
]


def same(a: oracle.Table, b: oracle.Table):
    assert a.k == b.k
    for f in ("bounds", "count", "sum", "lo", "hi"):
        assert np.array_equal(getattr(a, f), getattr(b, f)), f
    assert np.array_equal(a.mean.view(np.uint64), b.mean.view(np.uint64))
    assert (a.n_distinct, a.n_coarse, a.n_leaves) == (b.n_distinct, b.n_coarse, b.n_leaves)


@pytest.mark.parametrize("name,win,kw", CASES, ids=[c[0] for c in CASES])
def test_partition_ignores_the_window_order(name, win, kw):
    w = win()
    ref = oracle.partition(w, **kw)
    rng = np.random.default_rng(1)
    same(oracle.partition(rng.permutation(w), **kw), ref)
    same(oracle.partition(np.sort(w)[::-1].copy(), **kw), ref)


@pytest.mark.parametrize("name,win,kw", CASES, ids=[c[0] for c in CASES])
def test_partition_of_the_window_rebuilt_from_its_histogram(name, win, kw):
    w = win()
    L = kw.get("max_len", 32768)
    h = np.bincount(np.clip(w.astype(np.int64), 1, L), minlength=L + 1)
    rebuilt = np.repeat(np.arange(L + 1, dtype=np.int32), h)
    assert rebuilt.size == w.size
    same(oracle.partition(rebuilt, **kw), oracle.partition(w, **kw))


def test_partition_depends_on_multiplicities():
    # the same distinct lengths with other multiplicities change the queue
    # statistics (and, in the multiset gap mode, the split test), so a
    # histogram that dropped counts would be caught
    w = np.array([10, 10, 10, 11, 500, 900, 901, 902], np.int32)
    a = oracle.partition(w, init_queues=2, max_queues=2, min_width=0, gap_mode=1)
    b = oracle.partition(np.unique(w), init_queues=2, max_queues=2, min_width=0, gap_mode=1)
    assert not np.array_equal(a.count, b.count)
    assert a.count.sum() == w.size and b.count.sum() == np.unique(w).size
