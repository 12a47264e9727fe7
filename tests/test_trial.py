"""GPU parity of trials of batched scoring-parameter proposals
(ewsjf_trial_step / ewsjf_trial_finish) against the trial oracle: every
pool's admitted set at every step, the accumulated statistics (integers and
maxima bit for bit, sums of waits to 1e-12 relative: the GPU reduces them
in another order), the admissions per queue, and the Eq. 5 reward."""
import sys

import numpy as np
import pytest

import oracle
from oracle import trial as OT
from paper_2601_21758_amd import workloads as W

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


def proposals(rng, P):
    th = np.tile(W.THETA_MID.reshape(1, 6), (P, 1)).astype(np.float32)
    th *= rng.uniform(0.3, 3.0, (P, 6)).astype(np.float32)
    th[0] = W.THETA_MID
    return th


def run(E, cap, P, B, steps, per, seed, lam=(0.5, 2.0, 3.0, 0.1), gapped=False, nan=0.0):
    from paper_2601_21758_amd.trial import Trial
    rng = np.random.default_rng(seed)
    pool = W.make_pool("two", cap, seed, arrivals="poisson", rate=1e4, window=min(cap, 20000), K=16, B=B)
    t = oracle.partition(pool.window, init_queues=16, max_queues=16)
    tab = E.upload_table(t.bounds, t.mean, 32768, t.lo, t.hi, t.count, t.sum)
    if gapped:  # the gapped reading (bubble queues' table)
        E.dispatch(torch.zeros(0, dtype=torch.int32, device="cuda"),
                   torch.zeros(0, dtype=torch.float32, device="cuda"), tab, 64, 64)
        t.gapped = True
    length = np.where(rng.random(cap) < 0.6, pool.length, 0).astype(np.int32)
    arrival = pool.arrival.copy()
    arrival[rng.random(cap) < nan] = np.nan
    th = proposals(rng, P)
    t0 = float(np.nanmax(arrival))
    batches = []
    for s in range(steps):
        nl = rng.choice(pool.length, per).astype(np.int32)
        na = (t0 + 0.01 * s + rng.random(per) * 0.01).astype(np.float32)
        batches.append((nl, na, float(np.float32(t0 + 0.01 * (s + 1)))))
    tr = Trial(cap, th, B, tab, COST)
    tr.start(length, arrival)
    say(f"trial cap={cap} P={P} B={B} steps={steps} per={per}")
    got = []
    for nl, na, now in batches:
        ids, top, nsel = tr.step(dev(nl), dev(na), now)
        got.append((host(ids), host(nsel)))
    R = host(tr.finish(lam))
    stats, qad = host(tr.stats), host(tr.queue_admits)
    rs, rq, hist = OT.trial(length, arrival, t, th, batches, B, COST)
    # the admitted sets must agree (the trial's state and statistics depend on
    # the set only; the order within it may differ where scores tie to 1e-5)
    for s, ((ids, nsel), ref) in enumerate(zip(got, hist)):
        for p in range(P):
            assert int(nsel[p]) == ref[p].size and np.array_equal(np.sort(ids[p][:ref[p].size]), np.sort(ref[p])), \
                f"step {s} proposal {p}: admitted sets differ"
    exact = [0, 1, 4, 5, 6, 7]
    assert np.array_equal(stats[:, exact], rs[:, exact])
    assert np.allclose(stats[:, 2:4], rs[:, 2:4], rtol=1e-12, atol=0)
    assert np.array_equal(qad[:, :t.k], rq) and not qad[:, t.k:].any()
    assert np.allclose(R, OT.reward(rs, rq, t, lam), rtol=1e-12, atol=1e-15)
    return stats


@pytest.mark.parametrize("cap,P,B,steps,per,seed", [(4096, 4, 64, 20, 300, 1), (20000, 17, 200, 12, 2000, 2),
                                                    (1000, 1, 1000, 5, 0, 3), (65536, 8, 512, 8, 4096, 4)])
def test_trial_matches_oracle(E, cap, P, B, steps, per, seed):
    stats = run(E, cap, P, B, steps, per, seed)
    assert stats[:, 7].tolist() == [steps] * P


def test_trial_on_a_gapped_table_with_nan_arrivals(E):
    run(E, 8192, 5, 100, 10, 700, 5, gapped=True, nan=0.05)


def test_identical_proposals_agree(E):
    from paper_2601_21758_amd.trial import Trial
    rng = np.random.default_rng(6)
    p = W.config(0)
    t = oracle.partition(p.window, init_queues=16, max_queues=16)
    tab = E.upload_table(t.bounds, t.mean, 32768, t.lo, t.hi, t.count, t.sum)
    th = np.tile(W.THETA_MID.reshape(1, 6), (3, 1))
    cap = p.n - p.n % 4
    tr = Trial(cap, th, 256, tab, COST)
    tr.start(p.length[:cap], p.arrival[:cap])
    say("trial identical proposals")
    for s in range(5):
        nl = rng.choice(p.length, 1000).astype(np.int32)
        tr.step(dev(nl), dev(np.full(1000, p.now + s, np.float32)), p.now + s + 1)
    R = host(tr.finish())
    st = host(tr.stats)
    assert np.array_equal(st[0], st[1]) and np.array_equal(st[0], st[2]) and R[0] == R[1] == R[2]


def test_full_size_trial_prefix(E):
    """The bench's trial at full size (16 proposals on 1,048,576-slot rings,
    4,096 common arrivals and B=512 per step) for three steps."""
    from paper_2601_21758_amd.trial import Trial
    sw = W.Streaming(steps=3)
    L0, A0 = sw.initial_fill()
    t = oracle.partition(L0[-sw.window_size:], init_queues=sw.K, max_queues=sw.K)
    tab = E.upload_table(t.bounds, t.mean, 32768, t.lo, t.hi, t.count, t.sum)
    rng = np.random.default_rng(11)
    th = np.tile(W.THETA_MID.reshape(1, 6), (16, 1)).astype(np.float32)
    th[1:] *= rng.uniform(0.3, 3.0, (15, 6)).astype(np.float32)
    batches = []
    for i in range(3):
        nl, na = sw.arrivals(i)
        batches.append((nl, na, float(na[-1])))
    tr = Trial(sw.capacity, th, sw.B, tab, sw.cost)
    tr.start(L0, A0)
    say("trial full size: 16 x 1,048,576, 3 steps")
    got = []
    for nl, na, now in batches:
        ids, top, nsel = tr.step(dev(nl), dev(na), now)
        got.append((host(ids), host(nsel)))
    R = host(tr.finish((1.0, 1.0, 1.0, 1.0)))
    rs, rq, hist = OT.trial(L0, A0, t, th, batches, sw.B, sw.cost)
    for s, ((ids, nsel), ref) in enumerate(zip(got, hist)):
        for p in range(16):
            assert int(nsel[p]) == ref[p].size and np.array_equal(np.sort(ids[p][:ref[p].size]), np.sort(ref[p])), \
                f"step {s} proposal {p}"
    st = host(tr.stats)
    assert np.array_equal(st[:, [0, 1, 4, 5, 6, 7]], rs[:, [0, 1, 4, 5, 6, 7]])
    assert np.allclose(st[:, 2:4], rs[:, 2:4], rtol=1e-12, atol=0)
    assert np.allclose(R, OT.reward(rs, rq, t, (1.0, 1.0, 1.0, 1.0)), rtol=1e-12, atol=1e-15)
