"""The sliding-window partitioner input on the GPU: the window's length
histogram (built once, then kept current by the ring inserts) and
Refine-and-Prune started from it.  The histogram must equal a count of the
window's clamped lengths bit for bit, and the table partitioned from it must
equal, bit for bit, both the table partitioned from the window and the
oracle's."""
import sys

import numpy as np
import pytest

import oracle
from paper_2601_21758_amd import workloads as W
from parity_util import check_table
from test_gpu_parity import PART_CASES

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def E():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2601_21758_amd import ewsjf
    ewsjf.table_bytes()  # loads libewsjf.so or raises
    return ewsjf


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t):
    return t.detach().cpu().numpy()


def count(window, L):
    """The histogram by definition: entries per clamped length, bin 0 empty."""
    h = np.bincount(np.clip(np.asarray(window, np.int64), 1, L), minlength=L + 1).astype(np.int32)
    assert h[0] == 0
    return h


@pytest.mark.parametrize("n,L,seed", [(1, 32768, 0), (1000, 32768, 1), (16385, 32768, 2), (65536, 32768, 3),
                                      (1 << 20, 32768, 4), (50001, 100, 5), (7, 1, 6), (300000, 4096, 7)])
def test_window_histogram_counts_every_length(E, n, L, seed):
    rng = np.random.default_rng(seed)
    w = rng.integers(-50, L + 200, n).astype(np.int32)  # below 1 and above max_len clamp
    w[: min(n, 5)] = [L, 1, 0, -(1 << 31), (1 << 31) - 1][: min(n, 5)]
    say(f"window histogram n={n} L={L}")
    h = torch.full((L + 1,), 12345, dtype=torch.int32, device="cuda")  # written in full
    E.window_histogram(dev(w), L, hist=h)
    assert np.array_equal(host(h), count(w, L))


def test_window_histogram_of_an_empty_window(E):
    h = torch.full((101,), 7, dtype=torch.int32, device="cuda")
    E.window_histogram(torch.zeros(0, dtype=torch.int32, device="cuda"), 100, hist=h)
    assert not host(h).any()


@pytest.mark.parametrize("name", list(PART_CASES))
def test_partition_hist_equals_partition_and_oracle(E, name):
    win, kw = PART_CASES[name]()
    prm = E.params(**kw)
    say(f"partition_hist {name} W={len(win)}")
    w = dev(np.asarray(win, np.int32))
    t_win = E.partition(w, prm)
    h = E.window_histogram(w, prm.max_len)
    t_hist = E.partition_hist(h, prm)
    assert torch.equal(t_win, t_hist), "tables differ"  # every byte, lut and diagnostics included
    g = E.read_table(t_hist)
    assert g["n_window"] == len(win)
    check_table(g, oracle.partition(win, **kw))


@pytest.mark.parametrize("seed", range(3))
def test_partition_hist_kmeans3(E, seed):
    win = W.make_pool("three", 3000, 60 + seed, arrivals="uniform").window
    kw = dict(init_mode=oracle.KMEANS3, max_queues=32)
    prm = E.params(**kw)
    say(f"partition_hist kmeans3 seed={seed}")
    t = E.partition_hist(E.window_histogram(dev(win), prm.max_len), prm)
    check_table(E.read_table(t), oracle.partition(win, **kw))


@pytest.mark.parametrize("mode", [0, 1])
def test_partition_hist_of_an_empty_histogram(E, mode):
    prm = E.params(init_mode=mode, init_queues=8, max_queues=8)
    say(f"partition_hist empty mode={mode}")
    t = E.partition_hist(torch.zeros(prm.max_len + 1, dtype=torch.int32, device="cuda"), prm)
    g = E.read_table(t)
    assert g["k"] == 1 and g["n_window"] == 0 and g["n_distinct"] == 0 and g["n_leaves"] == 0
    assert g["count"][0] == 0 and g["sum"][0] == 0 and g["lo"][0] == 0 and g["hi"][0] == 0 and g["mean"][0] == 0.0
    assert not g["lut"].any()
    # the table routes every length to its one queue
    q = E.route(dev(np.array([1, 5, 32768, 40000, 0], np.int32)), t)
    assert host(q).tolist() == [0, 0, 0, 0, -1]


def _steps(rng, cap, wcap, L, steps):
    """(pos, wpos, new lengths, new arrivals) of a run of inserts that wraps
    both rings several times; lengths include clamped values and repeats."""
    pos = wpos = 0
    out = []
    for s in range(steps):
        n = int(rng.choice([0, 1, 17, wcap // 3, wcap]))
        nl = rng.integers(-3, L + 40, n).astype(np.int32)
        if n > 4:
            nl[:4] = [1, L, nl[4], nl[4]]
        na = (s + rng.random(n)).astype(np.float32)
        out.append((pos, wpos, nl, na))
        pos = (pos + n) % cap
        wpos = (wpos + n) % wcap
    return out


@pytest.mark.parametrize("L", [32768, 600])
def test_ring_insert_keeps_the_histogram(E, L):
    rng = np.random.default_rng(11)
    cap, wcap = 5000, 1201
    win = rng.integers(1, L + 1, wcap).astype(np.int32)
    g_rl = torch.zeros(cap, dtype=torch.int32, device="cuda")
    g_ra = torch.zeros(cap, dtype=torch.float32, device="cuda")
    g_w = dev(win.copy())
    g_h = E.window_histogram(g_w, L)
    say(f"ring_insert histogram L={L}")
    for pos, wpos, nl, na in _steps(rng, cap, wcap, L, 60):
        E.ring_insert(g_rl, g_ra, pos, dev(nl), dev(na), window=g_w, wpos=wpos, hist=g_h)
        win[(wpos + np.arange(nl.size)) % wcap] = nl
        assert np.array_equal(host(g_w), win)
        assert np.array_equal(host(g_h), count(win, L)), "histogram drifted from the window"


def test_ring_step_keeps_the_histogram_and_admits_the_same(E):
    """ewsjf_ring_step with and without the histogram: same ring, window and
    admissions; the kept histogram is the window's."""
    rng = np.random.default_rng(12)
    cap, wcap, B, L = 70001, 20000, 300, 32768
    p = W.config(0)
    t = oracle.partition(p.window, init_queues=16, max_queues=16)
    tab = E.upload_table(t.bounds, t.mean, L, t.lo, t.hi, t.count, t.sum)
    th = dev(W.THETA_MID.reshape(1, 6))
    L0 = rng.integers(1, 9000, cap).astype(np.int32)
    A0 = rng.random(cap).astype(np.float32)
    a_rl, a_ra, b_rl, b_ra = dev(L0), dev(A0), dev(L0), dev(A0)
    win = L0[:wcap].copy()
    a_w, b_w = dev(win), dev(win)
    h = E.window_histogram(a_w, L)
    say("ring_step histogram")
    for s, (pos, wpos, nl, na) in enumerate(_steps(rng, cap, wcap, L, 25)):
        now = float(s + 1)
        ga = E.ring_step(a_rl, a_ra, pos, dev(nl), dev(na), now, tab, th, B, window=a_w, wpos=wpos, tombstone=True,
                         hist=h)
        gb = E.ring_step(b_rl, b_ra, pos, dev(nl), dev(na), now, tab, th, B, window=b_w, wpos=wpos, tombstone=True)
        for x, y in zip(ga, gb):
            assert np.array_equal(host(x), host(y), equal_nan=True)
        assert torch.equal(a_rl, b_rl) and torch.equal(a_w, b_w)
        win[(wpos + np.arange(nl.size)) % wcap] = nl
        assert np.array_equal(host(a_w), win)
        assert np.array_equal(host(h), count(win, L)), f"histogram drifted at step {s}"


def test_streaming_scheduler_incremental_equals_window_mode(E):
    """The streaming scheduler with the kept histogram and with the window
    re-read at every repartition: the same tables after every repartition
    and the same admissions at every step; the tables are the oracle's."""
    from paper_2601_21758_amd.streaming import StreamingScheduler
    s = W.Streaming(seed=5, capacity=1 << 15, per_step=1024, steps=120, window=8192, rp_every=20, B=128, K=32)
    prm = E.params(init_queues=32, max_queues=32)
    a = StreamingScheduler(s.capacity, s.window_size, s.B, prm, s.theta[0], s.cost, incremental=True)
    b = StreamingScheduler(s.capacity, s.window_size, s.B, prm, s.theta[0], s.cost, incremental=False)
    L0, A0 = s.initial_fill()
    a.fill(L0, A0)
    b.fill(L0, A0)
    hist_win = [L0[-s.window_size:]]
    say("streaming incremental vs window re-read")
    for i in range(120):
        Ln, An = s.arrivals(i)
        now = float(An[-1])
        ra = a.step(now, length=dev(Ln), arrival=dev(An))
        rb = b.step(now, length=dev(Ln), arrival=dev(An))
        for x, y in zip(ra, rb):
            assert np.array_equal(host(x), host(y), equal_nan=True), f"admissions differ at step {i}"
        hist_win.append(Ln)
        if i % 20 == 0:
            a.launch_repartition()
            b.launch_repartition()
            torch.cuda.synchronize()
            ta, tb = a.table(), b.table()
            assert torch.equal(ta, tb), f"tables differ after step {i}"
            window = np.concatenate(hist_win)[-s.window_size:]
            assert np.array_equal(host(a.hist), count(window, prm.max_len))
            check_table(E.read_table(ta), oracle.partition(window, init_queues=32, max_queues=32))
