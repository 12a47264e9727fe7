"""Host-side checks of the C ABI: the library loads, exports every function
include/ewsjf.h declares, and rejects bad arguments before touching a device."""
import ctypes as C
import os
import re

import pytest

from paper_2601_21758_amd import _lib as L

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ewsjf.h")

pytestmark = pytest.mark.skipif(not os.path.exists(L.LIB_PATH), reason="libewsjf.so not built")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ewsjf_[a-z_0-9]+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    lib = L.lib()
    names = declared_functions()
    assert set(names) == set(L.EXPORTED)
    for name in names:
        assert hasattr(lib, name), name


def test_struct_layouts_match_header():
    lib = L.lib()
    assert lib.ewsjf_queue_table_bytes() == C.sizeof(L.QueueTable)
    assert C.sizeof(L.PartitionParams) == 40
    assert C.sizeof(L.Cost) == 24
    assert lib.ewsjf_version() >= 10000


def test_status_strings():
    for s in (L.OK, L.ERR_NULL, L.ERR_ARG, L.ERR_WORKSPACE, L.ERR_LAUNCH, L.ERR_ALIGN, L.ERR_DEVICE):
        assert L.status_string(s) and L.status_string(s) != "unknown status"


FAKE = C.c_void_p(0x10000)       # 16-byte aligned, never dereferenced: calls fail validation first
FAKE_MIS = C.c_void_p(0x10004)   # misaligned


def _p(**kw):
    d = dict(init_mode=0, init_queues=16, max_queues=16, min_width=16, max_len=32768, gap_mode=0, alpha=2.0,
             eps=1e-6)
    d.update(kw)
    return L.PartitionParams(**d)


def test_workspace_bytes_rules():
    lib = L.lib()
    assert lib.ewsjf_workspace_bytes(L.OP_STEP, 4 << 20, 1, 1024, None) > 0
    assert lib.ewsjf_workspace_bytes(L.OP_STEP, 1, 1, 0, None) == 0            # B < 1
    assert lib.ewsjf_workspace_bytes(L.OP_STEP, 10, 1, 4097, None) == 0        # B too large
    assert lib.ewsjf_workspace_bytes(L.OP_SELECT, 10, 0, 8, None) == 0         # n_theta < 1
    assert lib.ewsjf_workspace_bytes(L.OP_PARTITION, 10, 0, 0, None) == 0      # params missing
    assert lib.ewsjf_workspace_bytes(L.OP_PARTITION, 10, 0, 0, C.byref(_p())) > 0
    assert lib.ewsjf_workspace_bytes(L.OP_PARTITION, 10, 0, 0, C.byref(_p(alpha=1.0))) == 0
    assert lib.ewsjf_workspace_bytes(99, 10, 1, 1, None) == 0


def test_step_argument_errors():
    lib = L.lib()
    c = L.Cost(0.01, 1e-4, 0.0)
    ws_need = lib.ewsjf_workspace_bytes(L.OP_STEP, 1000, 1, 64, None)

    def step(length=FAKE, arr=FAKE, n=1000, now=60.0, table=FAKE, theta=FAKE, nt=1, cost=c, B=64, flags=0,
             ids=FAKE, top=FAKE, nsel=FAKE, ws=FAKE, wsb=ws_need):
        return lib.ewsjf_step(length, arr, n, now, table, theta, nt, C.byref(cost) if cost is not None else None,
                              B, flags, ids, top, nsel, ws, wsb, None)

    assert step(length=None) == L.ERR_NULL
    assert step(arr=None) == L.ERR_NULL
    assert step(table=None) == L.ERR_NULL
    assert step(cost=None) == L.ERR_NULL
    assert step(ws=None) == L.ERR_NULL
    assert step(n=-1) == L.ERR_ARG
    assert step(n=1 << 31) == L.ERR_ARG
    assert step(B=0) == L.ERR_ARG
    assert step(B=4097) == L.ERR_ARG
    assert step(nt=0) == L.ERR_ARG
    assert step(nt=1025) == L.ERR_ARG
    assert step(now=float("nan")) == L.ERR_ARG
    assert step(cost=L.Cost(0.0, 1e-4, 0.0)) == L.ERR_ARG
    assert step(cost=L.Cost(0.01, -1e-4, 0.0)) == L.ERR_ARG
    assert step(cost=L.Cost(0.01, 1e-4, float("inf"))) == L.ERR_ARG
    # costs the binary32 evaluation cannot hold: c0 rounding to 0 or a
    # subnormal, c0/c1/c2 above FLT_MAX, a subnormal c1 or c2
    for bad in [(1e-50, 0.0, 0.0), (1e-39, 0.0, 0.0), (1e39, 0.0, 0.0), (0.01, 1e39, 0.0), (0.01, 0.0, 1e39),
                (0.01, 1e-40, 0.0), (0.01, 0.0, 1e-45), (float("nan"), 0.0, 0.0), (0.01, 0.0, 1e11),
                (0.01, 1e20, 0.0), (1e29, 0.0, 0.0)]:
        assert step(cost=L.Cost(*bad)) == L.ERR_ARG, bad
    for good in [(1.2e-38, 0.0, 0.0), (1e28, 0.0, 0.0), (0.01, 1.2e-38, 2e-9), (0.01, 1e-4, 1e9)]:
        assert step(cost=L.Cost(*good)) != L.ERR_ARG, good
    assert step(flags=2) == L.ERR_ARG
    assert step(flags=L.STEP_TOMBSTONE, nt=2) == L.ERR_ARG
    assert step(wsb=ws_need - 1) == L.ERR_WORKSPACE
    assert step(length=FAKE_MIS) == L.ERR_ALIGN
    assert step(arr=FAKE_MIS) == L.ERR_ALIGN


def test_step_static_argument_errors():
    lib = L.lib()
    c = L.Cost(0.01, 1e-4, 0.0)

    def st(length=FAKE, arr=FAKE, n=1000, now=60.0, table=FAKE, theta=FAKE, nt=1, cost=c, B=64, flags=0,
           ids=FAKE, top=FAKE, nsel=FAKE):
        return lib.ewsjf_step_static(length, arr, n, now, table, theta, nt, C.byref(cost) if cost is not None else None,
                                     B, flags, ids, top, nsel, None)

    assert st(length=None) == L.ERR_NULL
    assert st(ids=None) == L.ERR_NULL
    assert st(cost=None) == L.ERR_NULL
    assert st(n=-1) == L.ERR_ARG and st(B=0) == L.ERR_ARG and st(nt=0) == L.ERR_ARG
    assert st(flags=L.STEP_TOMBSTONE, nt=2) == L.ERR_ARG
    assert st(cost=L.Cost(1e-50, 0.0, 0.0)) == L.ERR_ARG
    # sizes whose workspace exceeds the fixed scratch are refused before any device work
    assert lib.ewsjf_workspace_bytes(L.OP_STEP, 4194304, 16, 4096, None) > L.STATIC_SCRATCH_BYTES
    assert st(n=4194304, nt=16, B=4096) == L.ERR_WORKSPACE
    assert st(n=1 << 20, nt=56, B=256) == L.ERR_WORKSPACE
    # the largest pools with one vector fit; without a GPU the call stops at the device check
    assert st(n=(1 << 31) - 1, B=4096) == L.ERR_DEVICE
    assert st(n=1 << 20, nt=55, B=256) == L.ERR_DEVICE


def test_select_route_score_argument_errors():
    lib = L.lib()
    c = L.Cost(0.01, 1e-4, 0.0)
    need = lib.ewsjf_workspace_bytes(L.OP_SELECT, 100, 2, 8, None)
    assert lib.ewsjf_select(None, 100, 2, 8, FAKE, FAKE, FAKE, FAKE, need, None) == L.ERR_NULL
    assert lib.ewsjf_select(FAKE, 100, 2, 0, FAKE, FAKE, FAKE, FAKE, need, None) == L.ERR_ARG
    assert lib.ewsjf_select(FAKE, 100, 2, 8, FAKE, FAKE, FAKE, FAKE, need - 1, None) == L.ERR_WORKSPACE
    assert lib.ewsjf_select(FAKE_MIS, 100, 2, 8, FAKE, FAKE, FAKE, FAKE, need, None) == L.ERR_ALIGN
    assert lib.ewsjf_route(None, 10, FAKE, FAKE, None) == L.ERR_NULL
    assert lib.ewsjf_route(FAKE, -5, FAKE, FAKE, None) == L.ERR_ARG
    assert lib.ewsjf_route(FAKE, 10, FAKE, FAKE_MIS, None) == L.ERR_ALIGN
    assert lib.ewsjf_route(FAKE, 0, FAKE, FAKE, None) == L.OK  # nothing to do, no device touched
    assert lib.ewsjf_score(FAKE, FAKE, 10, 1.0, FAKE, FAKE, 1, None, FAKE, None) == L.ERR_NULL
    assert lib.ewsjf_score(FAKE, FAKE, 10, 1.0, FAKE, FAKE, 0, C.byref(c), FAKE, None) == L.ERR_ARG
    assert lib.ewsjf_score(FAKE, FAKE, 10, 1.0, FAKE, FAKE, 1, C.byref(c), FAKE_MIS, None) == L.ERR_ALIGN


def test_ring_insert_argument_errors():
    lib = L.lib()

    def ins(rl=FAKE, ra=FAKE, cap=100, pos=0, w=FAKE, wc=50, wpos=0, nl=FAKE, na=FAKE, n=10):
        return lib.ewsjf_ring_insert(rl, ra, cap, pos, w, wc, wpos, nl, na, n, None)

    assert ins(rl=None) == L.ERR_NULL
    assert ins(na=None) == L.ERR_NULL
    assert ins(w=None) == L.ERR_NULL            # a window size without a window
    assert ins(cap=0) == L.ERR_ARG
    assert ins(pos=100) == L.ERR_ARG            # pos must be a slot
    assert ins(pos=-1) == L.ERR_ARG
    assert ins(n=101) == L.ERR_ARG              # more than the ring holds
    assert ins(n=51) == L.ERR_ARG               # more than the window holds
    assert ins(wpos=50) == L.ERR_ARG
    assert ins(w=None, wc=0, wpos=3) == L.ERR_ARG
    assert ins(n=0) == L.OK                     # nothing to do, no device touched
    assert ins(rl=None, ra=None, nl=None, na=None, n=0) == L.OK


def test_window_histogram_and_partition_hist_argument_errors():
    lib = L.lib()
    p = _p()
    need = lib.ewsjf_workspace_bytes(L.OP_PARTITION, 0, 0, 0, C.byref(p))
    assert 0 < need <= lib.ewsjf_workspace_bytes(L.OP_PARTITION, 100, 0, 0, C.byref(p))

    def wh(ring=FAKE, cap=100, begin=0, n=100, m=4096, h=FAKE):
        return lib.ewsjf_window_histogram(ring, cap, begin, n, m, h, None)

    assert wh(h=None) == L.ERR_NULL
    assert wh(ring=None) == L.ERR_NULL
    assert wh(n=-1) == L.ERR_ARG
    assert wh(n=101) == L.ERR_ARG               # more entries than the ring holds
    assert wh(begin=100) == L.ERR_ARG
    assert wh(begin=-1) == L.ERR_ARG
    assert wh(cap=0, n=0, begin=1) == L.ERR_ARG
    assert wh(m=0) == L.ERR_ARG
    assert wh(m=L.MAX_LEN + 1) == L.ERR_ARG

    def wa(ring=FAKE, cap=100, add=10, sub=60, n=20, m=4096, h=FAKE):
        return lib.ewsjf_window_advance(ring, cap, add, sub, n, m, h, None)

    assert wa(ring=None) == L.ERR_NULL
    assert wa(h=None) == L.ERR_NULL
    assert wa(cap=0) == L.ERR_ARG
    assert wa(add=100) == L.ERR_ARG
    assert wa(sub=-1) == L.ERR_ARG
    assert wa(n=101) == L.ERR_ARG
    assert wa(n=-1) == L.ERR_ARG
    assert wa(m=0) == L.ERR_ARG
    assert wa(n=0) == L.OK                      # nothing to do, no device touched
    assert wa(ring=None, h=None, n=0) == L.OK

    def ph(h=FAKE, p=p, table=FAKE, ws=FAKE, wsb=need):
        return lib.ewsjf_partition_hist(h, C.byref(p) if p is not None else None, table, ws, wsb, None)

    assert ph(h=None) == L.ERR_NULL
    assert ph(p=None) == L.ERR_NULL
    assert ph(table=None) == L.ERR_NULL
    assert ph(ws=None) == L.ERR_NULL
    assert ph(p=_p(alpha=1.0)) == L.ERR_ARG
    assert ph(p=_p(max_len=0)) == L.ERR_ARG
    assert ph(wsb=need - 1) == L.ERR_WORKSPACE
    assert ph(ws=FAKE_MIS) == L.ERR_ALIGN


def test_tactical_step_argument_errors():
    lib = L.lib()
    c = L.Cost(0.01, 1e-4, 0.0)
    need = lib.ewsjf_workspace_bytes(L.OP_TACTICAL, 1000, 1, 64, None)
    assert need > 0 and lib.ewsjf_workspace_bytes(L.OP_TACTICAL, 1000, 1, 0, None) == 0

    def tac(length=FAKE, arr=FAKE, n=1000, now=60.0, table=FAKE, theta=FAKE, cost=c, B=64, thr=2, ec=FAKE, eps=1e-6,
            flags=0, ids=FAKE, nsel=FAKE, qp=FAKE, hs=FAKE, rm=FAKE, ws=FAKE, wsb=need):
        return lib.ewsjf_tactical_step(length, arr, n, now, table, theta, C.byref(cost) if cost is not None else None,
                                       B, thr, ec, eps, flags, ids, nsel, qp, hs, rm, ws, wsb, None)

    assert tac(length=None) == L.ERR_NULL
    assert tac(table=None) == L.ERR_NULL
    assert tac(ec=None) == L.ERR_NULL
    assert tac(qp=None) == L.ERR_NULL
    assert tac(cost=None) == L.ERR_NULL
    assert tac(B=0) == L.ERR_ARG
    assert tac(B=4097) == L.ERR_ARG
    assert tac(thr=-1) == L.ERR_ARG
    assert tac(eps=0.0) == L.ERR_ARG
    assert tac(eps=float("nan")) == L.ERR_ARG
    assert tac(now=float("inf")) == L.ERR_ARG
    assert tac(n=-1) == L.ERR_ARG
    assert tac(flags=4) == L.ERR_ARG
    assert tac(wsb=need - 1) == L.ERR_WORKSPACE
    assert tac(arr=FAKE_MIS) == L.ERR_ALIGN


def test_ring_step_argument_errors():
    lib = L.lib()
    c = L.Cost(0.01, 1e-4, 0.0)
    need = lib.ewsjf_workspace_bytes(L.OP_STEP, 100, 1, 8, None)

    def rs(rl=FAKE, ra=FAKE, cap=100, pos=0, w=FAKE, wc=50, wpos=0, nl=FAKE, na=FAKE, n=10, now=1.0, table=FAKE,
           theta=FAKE, cost=c, B=8, flags=0, ids=FAKE, top=FAKE, nsel=FAKE, ws=FAKE, wsb=need):
        return lib.ewsjf_ring_step(rl, ra, cap, pos, w, wc, wpos, nl, na, n, now, table, theta,
                                   C.byref(cost) if cost is not None else None, B, flags, ids, top, nsel, ws, wsb, None)

    assert rs(rl=None) == L.ERR_NULL
    assert rs(nl=None) == L.ERR_NULL
    assert rs(w=None) == L.ERR_NULL
    assert rs(table=None) == L.ERR_NULL
    assert rs(cap=0) == L.ERR_ARG
    assert rs(pos=100) == L.ERR_ARG
    assert rs(n=101) == L.ERR_ARG
    assert rs(n=51) == L.ERR_ARG
    assert rs(wpos=50) == L.ERR_ARG
    assert rs(B=0) == L.ERR_ARG
    assert rs(flags=2) == L.ERR_ARG
    assert rs(now=float("nan")) == L.ERR_ARG
    assert rs(wsb=need - 1) == L.ERR_WORKSPACE
    assert rs(ra=FAKE_MIS) == L.ERR_ALIGN


def test_partition_argument_errors():
    lib = L.lib()
    need = lib.ewsjf_workspace_bytes(L.OP_PARTITION, 100, 0, 0, C.byref(_p()))

    def part(win=FAKE, n=100, p=_p(), table=FAKE, ws=FAKE, wsb=need):
        return lib.ewsjf_partition(win, n, C.byref(p) if p is not None else None, table, ws, wsb, None)

    assert part(win=None) == L.ERR_NULL
    assert part(p=None) == L.ERR_NULL
    assert part(n=0) == L.ERR_ARG
    assert part(p=_p(alpha=1.0)) == L.ERR_ARG
    assert part(p=_p(eps=0.0)) == L.ERR_ARG
    assert part(p=_p(max_queues=0)) == L.ERR_ARG
    assert part(p=_p(max_queues=257)) == L.ERR_ARG
    assert part(p=_p(max_len=32769)) == L.ERR_ARG
    assert part(p=_p(min_width=-1)) == L.ERR_ARG
    assert part(p=_p(init_mode=2)) == L.ERR_ARG
    assert part(p=_p(gap_mode=3)) == L.ERR_ARG
    assert part(p=_p(init_queues=0)) == L.ERR_ARG
    assert part(wsb=need - 1) == L.ERR_WORKSPACE


def test_table_upload_argument_errors():
    lib = L.lib()
    h = L.QueueTable()
    h.k, h.max_len = 3, 1000
    h.bounds[0], h.bounds[1] = 100, 50   # not increasing
    assert lib.ewsjf_table_upload(C.byref(h), FAKE, None) == L.ERR_ARG
    h.bounds[1] = 2000                   # above max_len
    assert lib.ewsjf_table_upload(C.byref(h), FAKE, None) == L.ERR_ARG
    h.k = 0
    assert lib.ewsjf_table_upload(C.byref(h), FAKE, None) == L.ERR_ARG
    assert lib.ewsjf_table_upload(None, FAKE, None) == L.ERR_NULL
    # the gapped reading: 0 or 1, intervals in [1, max_len], increasing, disjoint
    h.k, h.bounds[0], h.bounds[1] = 3, 100, 500
    for q, (a, b) in enumerate([(10, 50), (100, 300), (500, 900)]):
        h.lo[q], h.hi[q], h.mean[q] = a, b, (a + b) / 2
    h.gapped = 2
    assert lib.ewsjf_table_upload(C.byref(h), FAKE, None) == L.ERR_ARG
    h.gapped = 1
    h.hi[1] = 500                        # overlaps the next interval
    assert lib.ewsjf_table_upload(C.byref(h), FAKE, None) == L.ERR_ARG
    h.hi[1], h.hi[2] = 300, 1001         # beyond max_len
    assert lib.ewsjf_table_upload(C.byref(h), FAKE, None) == L.ERR_ARG
    h.hi[2], h.lo[0] = 900, 0            # below 1
    assert lib.ewsjf_table_upload(C.byref(h), FAKE, None) == L.ERR_ARG
    h.lo[0], h.hi[0] = 60, 50            # empty interval
    assert lib.ewsjf_table_upload(C.byref(h), FAKE, None) == L.ERR_ARG
    # the contiguous reading: queue i > 0 starts at its bound
    h.gapped, h.lo[0], h.hi[0] = 0, 10, 50
    h.lo[1], h.lo[2] = 100, 499          # lo[2] != bounds[1]
    assert lib.ewsjf_table_upload(C.byref(h), FAKE, None) == L.ERR_ARG
    h.lo[1], h.lo[2] = 0, 500            # lo[1] left at 0
    assert lib.ewsjf_table_upload(C.byref(h), FAKE, None) == L.ERR_ARG
    h.lo[1] = 100                        # consistent: passes validation, then needs a device
    assert lib.ewsjf_table_upload(C.byref(h), FAKE, None) == L.ERR_DEVICE


def test_trial_argument_errors():
    lib = L.lib()
    c = L.Cost(0.01, 1e-4, 0.0)
    need = lib.ewsjf_workspace_bytes(L.OP_TRIAL, 1000, 4, 64, None)
    assert need > 0 and lib.ewsjf_workspace_bytes(L.OP_TRIAL, 1000, 0, 64, None) == 0

    def ts(ln=FAKE, ar=FAKE, cap=1000, P=4, pos=0, nl=FAKE, na=FAKE, n=10, now=1.0, table=FAKE, theta=FAKE, cost=c,
           B=64, ids=FAKE, top=FAKE, nsel=FAKE, st=FAKE, qa=FAKE, ws=FAKE, wsb=need):
        return lib.ewsjf_trial_step(ln, ar, cap, P, pos, nl, na, n, now, table, theta,
                                    C.byref(cost) if cost is not None else None, B, ids, top, nsel, st, qa, ws, wsb,
                                    None)

    assert ts(ln=None) == L.ERR_NULL
    assert ts(st=None) == L.ERR_NULL
    assert ts(qa=None) == L.ERR_NULL
    assert ts(nl=None) == L.ERR_NULL
    assert ts(cost=None) == L.ERR_NULL
    assert ts(cap=1002) == L.ERR_ARG           # pools must stay 16-byte aligned
    assert ts(P=0) == L.ERR_ARG
    assert ts(P=L.MAX_THETA + 1) == L.ERR_ARG
    assert ts(pos=1000) == L.ERR_ARG
    assert ts(n=1001) == L.ERR_ARG
    assert ts(B=0) == L.ERR_ARG
    assert ts(now=float("inf")) == L.ERR_ARG
    assert ts(wsb=need - 1) == L.ERR_WORKSPACE
    assert ts(ar=FAKE_MIS) == L.ERR_ALIGN
    lam = (C.c_double * 4)(1, 1, 1, 1)
    bad = (C.c_double * 4)(1, float("nan"), 1, 1)
    assert lib.ewsjf_trial_finish(None, FAKE, 1000, 4, 1.0, FAKE, FAKE, lam, FAKE, FAKE, None) == L.ERR_NULL
    assert lib.ewsjf_trial_finish(FAKE, FAKE, 1000, 4, 1.0, FAKE, FAKE, None, FAKE, FAKE, None) == L.ERR_NULL
    assert lib.ewsjf_trial_finish(FAKE, FAKE, 1000, 4, 1.0, FAKE, FAKE, bad, FAKE, FAKE, None) == L.ERR_ARG
    assert lib.ewsjf_trial_finish(FAKE, FAKE, 1001, 4, 1.0, FAKE, FAKE, lam, FAKE, FAKE, None) == L.ERR_ARG


def test_dispatch_argument_errors():
    lib = L.lib()

    def dsp(length=FAKE, arr=FAKE, n=100, table=FAKE, width=64, mq=32, qid=FAKE):
        return lib.ewsjf_dispatch(length, arr, n, table, width, mq, qid, None)

    assert dsp(table=None) == L.ERR_NULL
    assert dsp(length=None) == L.ERR_NULL
    assert dsp(arr=None) == L.ERR_NULL
    assert dsp(qid=None) == L.ERR_NULL
    assert dsp(n=-1) == L.ERR_ARG
    assert dsp(n=L.MAX_DISPATCH + 1) == L.ERR_ARG
    assert dsp(width=0) == L.ERR_ARG
    assert dsp(mq=0) == L.ERR_ARG
    assert dsp(mq=L.MAX_QUEUES + 1) == L.ERR_ARG


def test_valid_call_without_gpu_reports_no_device():
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    lib = L.lib()
    h = L.QueueTable()
    h.k, h.max_len = 1, 100
    h.mean[0] = 10.0
    assert lib.ewsjf_table_upload(C.byref(h), FAKE, None) == L.ERR_DEVICE
