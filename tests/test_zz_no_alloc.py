"""The allocation-free step, ewsjf_step_static, called through the C ABI:
its outputs against ewsjf_step's on the same inputs, on calls in a row of
decreasing size (the scratch keeps the previous call's contents), its
tombstone flag, and the rejection of sizes beyond its fixed scratch."""
import ctypes as C
import os
import sys

import numpy as np
import pytest

import oracle
from paper_2601_21758_amd import workloads as W

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
from parity_util import check_admission  # noqa: E402

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu
vp = C.c_void_p


def say(*a):
    print(*a, flush=True)


@pytest.fixture(scope="module")
def E():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2601_21758_amd import ewsjf
    ewsjf.table_bytes()  # loads libewsjf.so or raises
    return ewsjf


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def static_step(E, length, arrival, now, table, theta, B, cost, flags=0):
    """ewsjf_step_static through the C ABI; the outputs start as sentinels."""
    from paper_2601_21758_amd import _lib as L
    nt = theta.shape[0]
    ids = torch.full((nt, B), 7, dtype=torch.int32, device="cuda")
    top = torch.full((nt, B), 7.0, dtype=torch.float32, device="cuda")
    nsel = torch.full((nt,), 7, dtype=torch.int32, device="cuda")
    c = L.Cost(*cost)
    st = L.lib().ewsjf_step_static(vp(length.data_ptr()), vp(arrival.data_ptr()), length.numel(), float(now),
                                   vp(table.data_ptr()), vp(theta.data_ptr()), nt, C.byref(c), int(B), int(flags),
                                   vp(ids.data_ptr()), vp(top.data_ptr()), vp(nsel.data_ptr()),
                                   vp(torch.cuda.current_stream().cuda_stream))
    return st, ids, top, nsel


def same(a, b):
    return all(torch.equal(x.view(torch.int32), y.view(torch.int32)) for x, y in zip(a, b))


def case(E, p, theta=None):
    theta = p.theta if theta is None else theta
    t = oracle.partition(p.window, init_queues=p.init_queues, max_queues=p.max_queues)
    tab = E.upload_table(t.bounds, t.mean, 32768, t.lo, t.hi, t.count, t.sum)
    return t, tab, dev(p.length), dev(p.arrival), dev(theta)


def test_static_step_matches_step_on_calls_in_a_row(E):
    from paper_2601_21758_amd import _lib as L
    big = W.config(2)                    # 4,194,304 requests, B = 1,024
    mid = W.config(1)                    # 262,144 requests, B = 256 (smaller, after the big one)
    small = W.make_pool("three", 5001, 33, arrivals="uniform", horizon=300.0, window=None, K=16, B=100, n_theta=3)
    near = 0
    for name, p in (("4M", big), ("256k", mid), ("5001 x 3 vectors", small)):
        say(f"static step {name} n={p.n} n_theta={p.theta.shape[0]} B={p.B}")
        t, tab, Ld, Ad, th = case(E, p)
        st, ids, top, nsel = static_step(E, Ld, Ad, p.now, tab, th, p.B, p.cost)
        assert st == L.OK, L.status_string(st)
        ref = E.step(Ld, Ad, p.now, tab, th, p.B, p.cost)
        torch.cuda.synchronize()
        assert same((ids, top, nsel), ref), f"{name}: ewsjf_step_static differs from ewsjf_step"
        if p.n < 1_000_000:  # and the oracle's admission on the smaller pools
            rids, rtop, rnsel, rs = oracle.step(p.length, p.arrival, p.now, t, p.theta, p.B, p.cost)
            h = [x.cpu().numpy() for x in (ids, top, nsel)]
            for ti in range(p.theta.shape[0]):
                near += check_admission(h[0][ti], h[1][ti], h[2][ti], rids[ti], rtop[ti], rnsel[ti], rs[ti])
    say(f"near-tie differences {near}")


def test_static_step_tombstones_like_step(E):
    from paper_2601_21758_amd import _lib as L
    p = W.config(1)
    say("static step tombstone 256k")
    t, tab, Ld, Ad, th = case(E, p)
    L2 = Ld.clone()
    st, ids, top, nsel = static_step(E, Ld, Ad, p.now, tab, th, p.B, p.cost, flags=L.STEP_TOMBSTONE)
    assert st == L.OK
    ref = E.step(L2, Ad, p.now, tab, th, p.B, p.cost, tombstone=True)
    torch.cuda.synchronize()
    assert same((ids, top, nsel), ref)
    assert torch.equal(Ld, L2)
    assert int((Ld == 0).sum()) == int(nsel[0]) + int((dev(p.length) == 0).sum())


def test_static_step_rejects_sizes_beyond_its_scratch(E):
    from paper_2601_21758_amd import _lib as L
    p = W.make_pool("two", 4096, 5, arrivals="uniform", window=None, K=8, B=64)
    t, tab, Ld, Ad, _ = case(E, p)
    n_big = 4194304
    assert E.workspace_bytes(L.OP_STEP, n_big, 16, 4096) > L.STATIC_SCRATCH_BYTES
    th16 = dev(np.tile(W.THETA_MID, (16, 1)))
    # a 4,194,304-slot view is never read: the size check comes first
    Lbig = torch.zeros(n_big, dtype=torch.int32, device="cuda")
    Abig = torch.zeros(n_big, dtype=torch.float32, device="cuda")
    say("static step too large: 4M x 16 vectors, B=4096")
    st, ids, top, nsel = static_step(E, Lbig, Abig, 1.0, tab, th16, 4096, p.cost)
    torch.cuda.synchronize()
    assert st == L.ERR_WORKSPACE
    assert bool((ids == 7).all()) and bool((nsel == 7).all())  # nothing was enqueued
    # the largest vector count that fits still runs
    st, ids, top, nsel = static_step(E, Ld, Ad, p.now, tab, dev(np.tile(W.THETA_MID, (13, 1))), p.B, p.cost)
    assert st == L.OK
    ref = E.step(Ld, Ad, p.now, tab, dev(np.tile(W.THETA_MID, (13, 1))), p.B, p.cost)
    torch.cuda.synchronize()
    assert same((ids, top, nsel), ref)
