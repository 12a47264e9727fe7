"""Streaming harness: ring insertion, eviction, tombstones, Refine-and-Prune
every rp_every steps on the sliding window with a one-step hand-over, checked
in lockstep against the oracle (both sides apply the oracle's admitted set so
an allowed near-tie difference cannot make the states diverge)."""
import os
import sys

import numpy as np
import pytest
import torch

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

from paper_2601_21758_amd import workloads as W  # noqa: E402
from paper_2601_21758_amd.streaming import StreamingScheduler  # noqa: E402
from parity_util import check_admission, check_table  # noqa: E402
from streaming_ref import OracleStream  # noqa: E402
import oracle  # noqa: E402


# ---- host-side logic (CPU) ------------------------------------------------------
@pytest.mark.gpu
def test_ring_insert_matches_numpy():
    from paper_2601_21758_amd import ewsjf
    rng = np.random.default_rng(7)
    cap, wcap = 1000, 300
    rl = rng.integers(1, 5000, cap).astype(np.int32)
    ra = rng.random(cap).astype(np.float32)
    win = rng.integers(1, 5000, wcap).astype(np.int32)
    g_rl, g_ra, g_w = (torch.from_numpy(a.copy()).cuda() for a in (rl, ra, win))
    for pos, wpos, n in [(0, 0, 10), (995, 290, 7), (500, 0, 300), (999, 299, 1), (3, 5, 0)]:
        nl = rng.integers(1, 5000, n).astype(np.int32)
        na = rng.random(n).astype(np.float32)
        ewsjf.ring_insert(g_rl, g_ra, pos, torch.from_numpy(nl).cuda(), torch.from_numpy(na).cuda(), window=g_w,
                          wpos=wpos)
        slots = (pos + np.arange(n)) % cap
        rl[slots] = nl
        ra[slots] = na
        win[(wpos + np.arange(n)) % wcap] = nl
        torch.cuda.synchronize()
        assert np.array_equal(g_rl.cpu().numpy(), rl)
        assert np.array_equal(g_ra.cpu().numpy(), ra)
        assert np.array_equal(g_w.cpu().numpy(), win)


def test_reference_ring_and_window_follow_the_generator():
    s = W.Streaming(seed=4, capacity=1 << 12, per_step=256, steps=40, window=1024, rp_every=10, B=32)
    ref = OracleStream(s.capacity, s.window_size, s.B, 16, 16, s.theta, s.cost)
    L0, A0 = s.initial_fill()
    ref.fill(L0, A0)
    assert np.array_equal(np.sort(ref.win), np.sort(L0[-1024:]))
    history = [L0]
    for step in range(40):
        L, A = s.arrivals(step)
        ref.insert(L, A)
        history.append(L)
        # the request with id = slot holds the latest arrival written there
        assert np.array_equal(ref.len[s.slots(step)], L)
        # the window is the multiset of the last `window` arrival lengths
        last = np.concatenate(history)[-1024:]
        assert np.array_equal(np.sort(ref.win), np.sort(last))


def test_late_start_fill_is_the_runs_last_arrivals():
    # a run started at step 7 begins from the ring the run from step 0 would
    # hold before step 7 (no admissions), oldest first, and draws the same
    # step-7 arrivals into the same relative slots
    cap, per = 1000, 300
    full = W.Streaming(seed=4, capacity=cap, per_step=per, steps=20, window=256)
    L0, A0 = full.initial_fill()
    hist_l, hist_a = [L0], [A0]
    for s in range(7):
        l, a = full.arrivals(s)
        hist_l.append(l)
        hist_a.append(a)
    late = W.Streaming(seed=4, capacity=cap, per_step=per, steps=20, window=256, start_step=7)
    Lf, Af = late.initial_fill()
    assert np.array_equal(Lf, np.concatenate(hist_l)[-cap:])
    assert np.array_equal(Af, np.concatenate(hist_a)[-cap:])
    l7, a7 = full.arrivals(7)
    m7, b7 = late.arrivals(7)
    assert np.array_equal(l7, m7) and np.array_equal(a7, b7)
    assert late.p_short(7) == full.p_short(7)
    assert np.array_equal(late.slots(7), np.arange(per))
    with pytest.raises(ValueError):
        late.arrivals(9)


def test_constructor_rejects_window_larger_than_ring():
    from paper_2601_21758_amd import ewsjf
    with pytest.raises(ValueError):
        StreamingScheduler(100, 200, 8, ewsjf.params(), W.THETA_MID, device="cpu")


# ---- lockstep parity on the GPU ---------------------------------------------------
def _lockstep(capacity, per_step, steps, window, rp_every, B, K, label, tombstone_check_every=0, fused=False,
              incremental=True, bubbles=None, novel=0.0, start=0, total=None, report_every=50):
    """`steps` steps from step `start` of a drift schedule of `total` steps
    (default: `steps`)."""
    from paper_2601_21758_amd import ewsjf
    s = W.Streaming(seed=4, capacity=capacity, per_step=per_step, steps=total or steps, window=window,
                    rp_every=rp_every, B=B, K=K, start_step=start)
    prm = ewsjf.params(init_queues=K, max_queues=K)
    gpu = StreamingScheduler(capacity, window, B, prm, s.theta[0], s.cost, incremental=incremental, bubbles=bubbles)
    ref = OracleStream(capacity, window, B, K, K, s.theta, s.cost, bubbles=bubbles)
    L0, A0 = s.initial_fill()
    gpu.fill(L0, A0)
    ref.fill(L0, A0)
    check_table(ewsjf.read_table(gpu.table()), ref.table)
    near = 0
    grown = 0
    novel_rng = np.random.default_rng(99)
    for step in range(start, start + steps):
        L, A = s.arrivals(step)
        if novel:  # a fraction of the arrivals are of lengths the window has not seen
            pick = novel_rng.random(L.size) < novel
            L = np.where(pick, novel_rng.integers(1, 32769, L.size), L).astype(np.int32)
        Lg, Ag = torch.from_numpy(L).cuda(), torch.from_numpy(A).cuda()
        ref.insert(L, A)
        now = float(A[-1])
        tomb = tombstone_check_every and step % tombstone_check_every == 0
        if fused:  # the insert inside the step's kernels
            ids, top, nsel = gpu.step(now, tombstone=bool(tomb), length=Lg, arrival=Ag)
        else:
            gpu.insert(Lg, Ag)
            ids, top, nsel = gpu.step(now, tombstone=bool(tomb))
        rids, rtop, rnsel, rsc = ref.step(now)
        # the partition over the window after this step's arrivals takes effect at the next step
        if step % rp_every == 0:
            gpu.launch_repartition()
            rt = ref.repartition()
        torch.cuda.synchronize()
        gi = ids.cpu().numpy()[0]
        near += check_admission(gi, top.cpu().numpy()[0], nsel.cpu().numpy()[0], rids, rtop, rnsel, rsc)
        if step % rp_every == 0:
            check_table(ewsjf.read_table(gpu.table()), rt)
        if bubbles is not None:
            g = ewsjf.read_table(gpu.tables[gpu.cur])
            assert g["k"] == ref.table.k and np.array_equal(g["lo"], ref.table.lo), f"{label}: bubbles differ"
            assert np.array_equal(g["hi"], ref.table.hi) and g["gapped"]
        if tomb:
            # the step tombstoned its own admitted set; restore the slots the
            # oracle did not admit (near-ties only) before applying the oracle's
            glen = gpu.len.cpu().numpy()
            assert np.all(glen[gi[:int(nsel[0])]] == 0)
            extra = np.setdiff1d(gi[:int(nsel[0])], rids[:rnsel])
            if extra.size:
                gpu.len[torch.from_numpy(extra.astype(np.int64)).cuda()] = torch.from_numpy(ref.len[extra]).cuda()
        gpu.apply_tombstones(rids[:rnsel])
        ref.tombstone(rids[:rnsel])
        if step % report_every == 0 or step == start + steps - 1:
            assert np.array_equal(gpu.len.cpu().numpy(), ref.len), f"{label}: ring lengths diverged at step {step}"
            print(f"{label}: step {step} ok (short weight {s.p_short(step):.3f}, near-tie differences so far "
                  f"{near})", flush=True)
    assert np.array_equal(gpu.arr.cpu().numpy(), ref.arr)
    assert np.array_equal(np.sort(gpu.window_lengths().cpu().numpy()), np.sort(ref.win)), f"{label}: window differs"
    if bubbles is not None:
        print(f"{label}: bubble queues created {ref.created}", flush=True)
        assert ref.created > 0, f"{label}: no bubble queue was created"
    return near, gpu


@pytest.mark.gpu
@pytest.mark.parametrize("incremental", [True, False])
def test_streaming_lockstep_small(incremental):
    # the window turns over between partitions: every partition but the first
    # (one step after the fill) recounts it
    _, gpu = _lockstep(capacity=1 << 14, per_step=512, steps=120, window=4096, rp_every=10, B=64, K=16,
                       label="small", tombstone_check_every=7, incremental=incremental)
    assert gpu.advanced == (1 if incremental else 0)


@pytest.mark.gpu
@pytest.mark.parametrize("incremental", [True, False])
def test_streaming_lockstep_slow_window(incremental):
    # 100 arrivals per step and a partition every 7 steps over a 4,096-length
    # window: the histogram moves forward by 700 entries per partition (or
    # the window is recounted, without incremental)
    _, gpu = _lockstep(capacity=1 << 13, per_step=100, steps=150, window=4096, rp_every=7, B=32, K=16,
                       label="slow", tombstone_check_every=5, fused=incremental, incremental=incremental)
    assert (gpu.advanced > 0) == incremental


@pytest.mark.gpu
def test_streaming_lockstep_ring_wraps_many_times():
    # 24 steps of 1024 into a 4096-slot ring: every slot is overwritten six
    # times, evicting pending requests
    _lockstep(capacity=4096, per_step=1024, steps=24, window=2048, rp_every=5, B=128, K=8, label="wrap",
              tombstone_check_every=3)


@pytest.mark.gpu
def test_streaming_lockstep_fused_insert():
    # arrivals inserted inside the step's kernels (ewsjf_ring_step): a ring
    # that wraps, with tombstone and partition hand-overs
    _lockstep(capacity=6144, per_step=1000, steps=30, window=3000, rp_every=4, B=100, K=8, label="fused-wrap",
              tombstone_check_every=2, fused=True)
    _lockstep(capacity=1 << 16, per_step=700, steps=60, window=8192, rp_every=10, B=64, K=16, label="fused",
              tombstone_check_every=5, fused=True)


@pytest.mark.gpu
@pytest.mark.parametrize("fused", [True, False])
def test_streaming_lockstep_with_bubble_queues(fused):
    # every step's arrivals go through the Dispatcher (Algorithm 2) before the
    # step; long arrivals in the gaps of the sparse tail open bubble queues
    # that the next partition replaces
    _lockstep(capacity=1 << 14, per_step=300, steps=60, window=512, rp_every=15, B=64, K=64, label="bubbles",
              tombstone_check_every=4, fused=fused, bubbles=(64, 128), novel=0.05)


@pytest.mark.gpu
def test_streaming_nonblocking_handover():
    """handover="when_ready": a partition takes effect at the first step
    issued after it finished, and a repartition requested while one runs is
    skipped.  The reference takes each new table at the step the scheduler
    recorded; tables and admissions agree throughout."""
    from paper_2601_21758_amd import ewsjf
    s = W.Streaming(seed=8, capacity=1 << 15, per_step=1024, steps=80, window=8192, rp_every=3, B=64, K=16)
    prm = ewsjf.params(init_queues=16, max_queues=16)
    gpu = StreamingScheduler(s.capacity, s.window_size, s.B, prm, s.theta[0], s.cost, handover="when_ready")
    ref = OracleStream(s.capacity, s.window_size, s.B, 16, 16, s.theta, s.cost)
    L0, A0 = s.initial_fill()
    gpu.fill(L0, A0)
    ref.fill(L0, A0)
    launched_for = None  # the oracle's partition of the window the running repartition saw
    for step in range(80):
        L, A = s.arrivals(step)
        Lg, Ag = torch.from_numpy(L).cuda(), torch.from_numpy(A).cuda()
        ref.insert(L, A)
        n_swaps = len(gpu.swaps)
        ids, top, nsel = gpu.step(float(A[-1]), tombstone=False, length=Lg, arrival=Ag)
        took = len(gpu.swaps) > n_swaps
        if took:
            ref.next_table, launched_for = launched_for, None
        rids, rtop, rnsel, rsc = ref.step(float(A[-1]), take_new=took)
        if step % 3 == 0:
            before = gpu.skipped
            gpu.launch_repartition()
            if gpu.skipped == before:
                launched_for = oracle.partition(ref.win, init_queues=16, max_queues=16)
        torch.cuda.synchronize()
        check_admission(ids.cpu().numpy()[0], top.cpu().numpy()[0], nsel.cpu().numpy()[0], rids, rtop, rnsel, rsc)
        gpu.apply_tombstones(rids[:rnsel])  # both sides drop the oracle's admitted set
        ref.tombstone(rids[:rnsel])
        g = ewsjf.read_table(gpu.tables[gpu.cur])
        assert np.array_equal(g["bounds"], ref.table.bounds), f"step {step}: tables differ"
    assert gpu.swaps, "no partition took effect"
    print(f"nonblocking: {len(gpu.swaps)} swaps, {gpu.skipped} skipped", flush=True)


@pytest.mark.gpu
def test_streaming_lockstep_full_size_prefix():
    # the streaming workload at full size (1,048,576-slot ring, 4,096 arrivals
    # and 512 admissions per step, 65,536-length window, 64 queues): the first
    # 101 steps, so two hand-overs (steps 0 and 100) are covered
    _lockstep(capacity=1 << 20, per_step=4096, steps=101, window=65536, rp_every=100, B=512, K=64, label="full",
              tombstone_check_every=25, fused=True)


@pytest.mark.gpu
def test_streaming_lockstep_full_size_late_drift():
    # the streaming workload at full size late in its drift: the ring holds
    # the last 1,048,576 arrivals drawn before step 9,799 of the 10,000-step
    # schedule (short weight ~0.31), then steps 9,799..9,901 run in lockstep,
    # so the partitions of steps 9,800 and 9,900 both take effect
    _lockstep(capacity=1 << 20, per_step=4096, steps=103, window=65536, rp_every=100, B=512, K=64,
              label="full-late", tombstone_check_every=25, fused=True, start=9799, total=10000, report_every=20)


@pytest.mark.gpu
def test_streaming_lockstep_whole_drift_reduced():
    # the whole 10,000-step drift (short weight 0.9 -> 0.3) at reduced size:
    # a 65,536-slot ring, 256 arrivals and B=32 admissions per step, a
    # 4,096-length window partitioned every 100 steps into up to 64 queues;
    # every step's admissions and every partition are compared
    _lockstep(capacity=1 << 16, per_step=256, steps=10000, window=4096, rp_every=100, B=32, K=64,
              label="drift", tombstone_check_every=97, fused=True, report_every=500)
