"""The sliding-window partitioner input on the GPU: the window's length
histogram (counted from a range of a ring of recent lengths, or moved
forward as the window slides) and Refine-and-Prune started from it.  The
histogram must equal a count of the window's clamped lengths bit for bit,
and the table partitioned from it must equal, bit for bit, both the table
partitioned from the window and the oracle's."""
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


@pytest.mark.parametrize("cap,begin,n", [(1000, 0, 1000), (1000, 999, 1000), (1000, 600, 700), (1000, 300, 1),
                                         (70001, 50000, 65536), (1 << 20, (1 << 20) - 5, 300000), (5, 4, 0)])
def test_window_histogram_of_a_ring_range(E, cap, begin, n):
    rng = np.random.default_rng(cap + begin + n)
    L = 32768
    ring = rng.integers(-2, L + 9, cap).astype(np.int32)
    say(f"window histogram of ring[{begin}..+{n}) mod {cap}")
    h = E.window_histogram(dev(ring), L, begin=begin, n=n)
    assert np.array_equal(host(h), count(ring[(begin + np.arange(n)) % cap], L))


@pytest.mark.parametrize("L,W,R", [(32768, 4096, 8192), (32768, 1000, 1001), (700, 3001, 9000), (32768, 65536, 131072)])
def test_window_advance_follows_the_window(E, L, W, R):
    """A log ring of R recent lengths with the window its last W entries:
    every few writes the histogram moves forward by the entries written since
    (ewsjf_window_advance) and must equal a recount of the window."""
    rng = np.random.default_rng(L + W + R)
    log = np.zeros(R, np.int32)
    log[:W] = rng.integers(1, L + 1, W)
    g_log = dev(log)
    h = E.window_histogram(g_log, L, begin=0, n=W)
    head = hist_head = W
    say(f"window advance L={L} W={W} R={R}")
    for it in range(40):
        # write a burst of lengths (clamped values and repeats included)
        for _ in range(int(rng.integers(1, 4))):
            n = int(rng.choice([1, 17, max(1, (R - W) // 5), R - W]))
            n = min(n, R - W - (head - hist_head))  # the leaving entries must still be in the log
            if n <= 0:
                break
            x = rng.integers(-3, L + 40, n).astype(np.int32)
            if n > 4:
                x[:2] = x[2]
            slots = (head + np.arange(n)) % R
            log[slots] = x
            g_log[torch.from_numpy(slots).cuda()] = dev(x)
            head += n
        new = head - hist_head
        E.window_advance(g_log, hist_head % R, (hist_head - W) % R, new, h)
        hist_head = head
        window = log[(head - W + np.arange(W)) % R]
        assert np.array_equal(host(h), count(window, L)), f"histogram drifted at burst {it}"


def test_window_advance_of_nothing_and_of_a_whole_window(E):
    L, W = 32768, 5000
    rng = np.random.default_rng(3)
    log = rng.integers(1, 9000, 2 * W).astype(np.int32)
    g = dev(log)
    h = E.window_histogram(g, L, begin=0, n=W)
    E.window_advance(g, W, 0, 0, h)  # nothing moves
    assert np.array_equal(host(h), count(log[:W], L))
    E.window_advance(g, W, 0, W, h)  # the window becomes the second half
    assert np.array_equal(host(h), count(log[W:], L))


@pytest.mark.parametrize("per_step,rp_every", [(1024, 20), (200, 7)])
def test_streaming_scheduler_incremental_equals_recount(E, per_step, rp_every):
    """The streaming scheduler moving the window's histogram forward and
    recounting the window at every repartition: the same tables after every
    repartition and the same admissions at every step; the tables are the
    oracle's partition of the window.  (1024, 20) turns the window over
    between partitions, (200, 7) does not."""
    from paper_2601_21758_amd.streaming import StreamingScheduler
    steps = 120
    s = W.Streaming(seed=5, capacity=1 << 15, per_step=per_step, steps=steps, window=8192, rp_every=rp_every, B=128,
                    K=32)
    prm = E.params(init_queues=32, max_queues=32)
    a = StreamingScheduler(s.capacity, s.window_size, s.B, prm, s.theta[0], s.cost, incremental=True)
    b = StreamingScheduler(s.capacity, s.window_size, s.B, prm, s.theta[0], s.cost, incremental=False)
    L0, A0 = s.initial_fill()
    a.fill(L0, A0)
    b.fill(L0, A0)
    seen = [L0[-s.window_size:]]
    say(f"streaming incremental vs recount per_step={per_step} rp_every={rp_every}")
    for i in range(steps):
        Ln, An = s.arrivals(i)
        now = float(An[-1])
        ra = a.step(now, length=dev(Ln), arrival=dev(An))
        rb = b.step(now, length=dev(Ln), arrival=dev(An))
        for x, y in zip(ra, rb):
            assert np.array_equal(host(x), host(y), equal_nan=True), f"admissions differ at step {i}"
        seen.append(Ln)
        if i % rp_every == 0:
            a.launch_repartition()
            b.launch_repartition()
            torch.cuda.synchronize()
            ta, tb = a.table(), b.table()
            assert torch.equal(ta, tb), f"tables differ after step {i}"
            window = np.concatenate(seen)[-s.window_size:]
            assert np.array_equal(host(a.hist), count(window, prm.max_len))
            assert np.array_equal(np.sort(host(a.window_lengths())), np.sort(window))
            check_table(E.read_table(ta), oracle.partition(window, init_queues=32, max_queues=32))
    assert b.advanced == 0
    # the histogram moves forward when fewer than `window` entries joined since
    # the last count (the first partition follows one step; later ones follow
    # rp_every steps); otherwise the window is recounted
    joined = [per_step] + [per_step * rp_every] * ((steps - 1) // rp_every)
    assert a.advanced == sum(j < s.window_size for j in joined)
