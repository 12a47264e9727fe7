"""GPU parity of the tactical step (Algorithm 1) against the oracle, in
lockstep over several steps (the admitted slots are emptied on both sides,
queues run dry and are removed)."""
import sys

import numpy as np
import pytest

import oracle
from paper_2601_21758_amd import workloads as W
from parity_util import SCORE_RTOL

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

COST = (0.01, 1e-4, 0.0)


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


def upload(E, t: oracle.Table):
    return E.upload_table(t.bounds, t.mean, 32768, t.lo, t.hi, t.count, t.sum)


def near_tie(a, b, rtol=SCORE_RTOL):
    return abs(float(a) - float(b)) <= rtol * max(abs(float(a)), abs(float(b)), 1e-30)


def compare_step(E, tab, ec_dev, out, ref: oracle.TacticalResult, k0):
    ids, nsel, qp, hs, rm = (host(x) for x in out)
    # head scores: 1e-5 relative, NaN exactly for the empty queues
    g, r = hs[:k0], ref.head_score
    assert np.array_equal(np.isnan(g), np.isnan(r))
    fin = ~np.isnan(r)
    if fin.any():
        err = np.abs(g[fin].astype(np.float64) - r[fin]) / np.maximum(np.abs(r[fin].astype(np.float64)), 1e-30)
        assert err.max() <= SCORE_RTOL, f"head score error {err.max():.3e}"
    if int(qp[0]) != ref.q_prim:
        # allowed only where the oracle's head scores tie within the tolerance
        assert near_tie(r[int(qp[0])], r[ref.q_prim]), f"q_prim {qp[0]} != {ref.q_prim}"
        return False
    n = int(nsel[0])
    assert n == ref.ids.size, f"n_sel {n} != {ref.ids.size}"
    if not np.array_equal(ids[:n], ref.ids):
        # the backfill order may differ only where the neighbours' head scores tie
        p = ref.q_prim
        nb = [j for j in (p - 1, p + 1) if 0 <= j < k0 and not np.isnan(r[j])]
        assert len(nb) == 2 and near_tie(r[nb[0]], r[nb[1]]), "batch differs"
        return False
    assert np.all(ids[n:] == -1)
    assert np.array_equal(rm[:k0].astype(bool), ref.removed)
    gt, rt = E.read_table(tab), ref.table
    assert gt["k"] == rt.k and np.array_equal(gt["bounds"], rt.bounds)
    assert np.array_equal(gt["count"], rt.count) and np.array_equal(gt["sum"], rt.sum)
    assert np.array_equal(gt["lo"], rt.lo) and np.array_equal(gt["hi"], rt.hi)
    assert np.array_equal(gt["mean"].view(np.uint64), rt.mean.view(np.uint64))
    assert np.array_equal(gt["lut"][1:], oracle.route(np.arange(1, gt["max_len"] + 1), ref.table)), "lut"
    assert np.array_equal(E.route_map_queues(gt["route"], gt["max_len"])[1:], gt["lut"][1:]), "compact routing map"
    assert np.array_equal(host(ec_dev)[:ref.table.k], ref.empty_cnt)
    return True


def run_lockstep(E, L, A, now, t, B, thr, steps, theta=None, arrivals=None):
    theta = W.THETA_MID if theta is None else theta
    th = dev(np.asarray(theta, np.float32).reshape(1, 6))
    tab = upload(E, t)
    ec_dev = E.new_empty_counters("cuda")
    ec = np.zeros(t.k, np.int32)
    Ld, Ad = dev(L.astype(np.int32)), dev(A.astype(np.float32))
    Lh = L.astype(np.int32).copy()
    ws = E.Workspace("cuda")
    exact = 0
    for s in range(steps):
        k0 = t.k
        out = E.tactical_step(Ld, Ad, now, tab, th, B, thr, ec_dev, tombstone=True, ws=ws)
        ref = oracle.tactical_step(Lh, A, now, t, ec, theta, B, thr, COST)
        ok = compare_step(E, tab, ec_dev, out, ref, k0)
        if not ok:
            say(f"  step {s}: near-tie, stopping the lockstep")
            break
        exact += 1
        Lh[ref.ids] = 0
        assert np.array_equal(host(Ld), Lh), "tombstones differ"
        t, ec = ref.table, ref.empty_cnt
        if arrivals is not None:
            Lh = arrivals(s, Lh)
            Ld.copy_(dev(Lh))
    return exact


@pytest.mark.parametrize("cfg,B,thr,steps", [(0, 64, 0, 40), (0, 500, 2, 12), (1, 256, 1, 12)])
def test_tactical_lockstep_matches_oracle(E, cfg, B, thr, steps):
    p = W.config(cfg)
    say(f"tactical cfg{cfg} n={p.n} B={B} thr={thr}")
    t = oracle.partition(p.window, init_queues=p.init_queues, max_queues=p.max_queues)
    # thin the pool so that queues run dry within a few steps
    rng = np.random.default_rng(cfg + 7)
    L = np.where(rng.random(p.n) < 0.08, p.length, 0).astype(np.int32)
    exact = run_lockstep(E, L, p.arrival, p.now, t, B, thr, steps)
    assert exact >= steps // 2


def test_tactical_removals_happen_and_match(E):
    # a sparse pool over a 16-queue table: most queues are empty from the start
    p = W.config(0)
    t = oracle.partition(p.window, init_queues=p.init_queues, max_queues=p.max_queues)
    rng = np.random.default_rng(2)
    L = np.where(rng.random(p.n) < 0.01, p.length, 0).astype(np.int32)
    say(f"tactical removals k={t.k} live={int((L > 0).sum())}")
    th = dev(W.THETA_MID.reshape(1, 6))
    tab = upload(E, t)
    ec_dev = E.new_empty_counters("cuda")
    out = E.tactical_step(dev(L), dev(p.arrival), p.now, tab, th, 8, 0, ec_dev)
    ref = oracle.tactical_step(L, p.arrival, p.now, t, np.zeros(t.k, np.int32), W.THETA_MID, 8, 0, COST)
    assert ref.removed.any()
    assert compare_step(E, tab, ec_dev, out, ref, t.k)


def test_tactical_ragged_with_arrivals(E):
    p = W.make_pool("two", 50001, 21, arrivals="poisson", rate=1e4, window=20001, K=32, B=100)
    t = oracle.partition(p.window, init_queues=p.init_queues, max_queues=p.max_queues)
    rng = np.random.default_rng(4)
    L = np.where(rng.random(p.n) < 0.05, p.length, 0).astype(np.int32)
    fresh = p.length.copy()

    def arrivals(s, Lh):  # refill a few emptied slots with their original requests
        idx = rng.choice(p.n, 300, replace=False)
        Lh = Lh.copy()
        Lh[idx] = fresh[idx]
        return Lh

    say("tactical ragged 50001 with arrivals")
    assert run_lockstep(E, L, p.arrival, p.now, t, 100, 1, 15, arrivals=arrivals) >= 7


@pytest.mark.parametrize("kind", W.ADVERSARIAL_KINDS)
def test_tactical_adversarial(E, kind):
    L, A, now = W.adversarial(kind, 4099, 3)
    say(f"tactical adversarial {kind}")
    t = oracle.partition(np.clip(L, 1, None), init_queues=8, max_queues=8)
    run_lockstep(E, L, A, now, t, 300, 1, 6)


def test_tactical_nan_and_equal_arrivals(E):
    rng = np.random.default_rng(9)
    n = 5000
    L = rng.integers(1, 3000, n).astype(np.int32)
    A = rng.integers(0, 50, n).astype(np.float32)
    A[::13] = np.nan
    A[::17] = -0.0
    t = oracle.partition(L, init_queues=8, max_queues=8)
    say("tactical NaN / equal arrivals")
    assert run_lockstep(E, L, A, 60.0, t, 700, 0, 8) >= 4


def test_tactical_all_empty_and_single_queue(E):
    t = oracle.partition(np.array([5, 6, 7], np.int32), init_queues=1, max_queues=1)
    assert t.k == 1
    L = np.zeros(1000, np.int32)
    A = np.zeros(1000, np.float32)
    say("tactical all empty")
    th = dev(W.THETA_MID.reshape(1, 6))
    tab = upload(E, t)
    ec_dev = E.new_empty_counters("cuda")
    ids, nsel, qp, hs, rm = E.tactical_step(dev(L), dev(A), 1.0, tab, th, 16, 0, ec_dev)
    assert int(host(nsel)[0]) == 0 and int(host(qp)[0]) == -1 and np.all(host(ids) == -1)
    assert E.read_table(tab)["k"] == 1 and int(host(ec_dev)[0]) == 1


def test_tactical_full_size_step(E):
    p = W.config(2)
    say(f"tactical full size n={p.n}")
    t = oracle.partition(p.window, init_queues=p.init_queues, max_queues=p.max_queues)
    th = dev(W.THETA_MID.reshape(1, 6))
    tab = upload(E, t)
    ec_dev = E.new_empty_counters("cuda")
    out = E.tactical_step(dev(p.length), dev(p.arrival), p.now, tab, th, p.B, 3, ec_dev)
    ref = oracle.tactical_step(p.length, p.arrival, p.now, t, np.zeros(t.k, np.int32), W.THETA_MID, p.B, 3, COST)
    assert compare_step(E, tab, ec_dev, out, ref, t.k)
