"""ctypes declarations for libewsjf.so (the C ABI in include/ewsjf.h).

Argument marshalling only.  Loading fails loudly when the library has not
been built: there is no fallback implementation.
"""
from __future__ import annotations

import ctypes as C
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libewsjf.so")

OK, ERR_NULL, ERR_ARG, ERR_WORKSPACE, ERR_LAUNCH, ERR_ALIGN, ERR_DEVICE = 0, -1, -2, -3, -4, -5, -6
MAX_QUEUES, MAX_LEN, MAX_B, MAX_THETA, MAX_DISPATCH = 256, 32768, 4096, 1024, 4096
ROUTE_WORDS = MAX_LEN // 32 + 2
INIT_EQUAL_WIDTH, INIT_KMEANS3 = 0, 1
GAPS_DISTINCT, GAPS_MULTISET = 0, 1
STEP_TOMBSTONE = 1
OP_PARTITION, OP_SELECT, OP_STEP, OP_TACTICAL, OP_TRIAL = 0, 1, 2, 3, 4
TRIAL_STATS = 8

EXPORTED = ("ewsjf_queue_table_bytes", "ewsjf_workspace_bytes", "ewsjf_table_upload", "ewsjf_partition",
            "ewsjf_route", "ewsjf_score", "ewsjf_select", "ewsjf_step", "ewsjf_step_timed", "ewsjf_ring_insert",
            "ewsjf_tactical_step", "ewsjf_ring_step", "ewsjf_window_histogram", "ewsjf_window_advance",
            "ewsjf_partition_hist", "ewsjf_dispatch", "ewsjf_trial_step", "ewsjf_trial_finish",
            "ewsjf_status_string", "ewsjf_version", "ewsjf_step_static")
STATIC_SCRATCH_BYTES = 4 << 20


class PartitionParams(C.Structure):
    _fields_ = [("init_mode", C.c_int32), ("init_queues", C.c_int32), ("max_queues", C.c_int32),
                ("min_width", C.c_int32), ("max_len", C.c_int32), ("gap_mode", C.c_int32),
                ("alpha", C.c_double), ("eps", C.c_double)]


class Cost(C.Structure):
    _fields_ = [("c0", C.c_double), ("c1", C.c_double), ("c2", C.c_double)]


class QueueTable(C.Structure):
    _fields_ = [("k", C.c_int32), ("max_len", C.c_int32), ("n_distinct", C.c_int32), ("n_coarse", C.c_int32),
                ("n_leaves", C.c_int32), ("gapped", C.c_int32), ("n_window", C.c_int64),
                ("bounds", C.c_int32 * MAX_QUEUES), ("lo", C.c_int32 * MAX_QUEUES),
                ("hi", C.c_int32 * MAX_QUEUES), ("count", C.c_int64 * MAX_QUEUES),
                ("sum", C.c_int64 * MAX_QUEUES), ("mean", C.c_double * MAX_QUEUES),
                ("lut", C.c_uint8 * (MAX_LEN + 16)), ("route", C.c_uint64 * ROUTE_WORDS)]


class EwsjfError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(f"{what}: {status_string(status)} ({status})")


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run __graft_entry__.build() "
                               "(python -m paper_2601_21758_amd.build)")
        L = C.CDLL(LIB_PATH)
        vp, i32, i64, f32, sz = C.c_void_p, C.c_int32, C.c_int64, C.c_float, C.c_size_t
        L.ewsjf_queue_table_bytes.argtypes = []
        L.ewsjf_queue_table_bytes.restype = sz
        L.ewsjf_workspace_bytes.argtypes = [C.c_int, i64, i32, i32, C.POINTER(PartitionParams)]
        L.ewsjf_workspace_bytes.restype = sz
        L.ewsjf_table_upload.argtypes = [C.POINTER(QueueTable), vp, vp]
        L.ewsjf_table_upload.restype = C.c_int
        L.ewsjf_partition.argtypes = [vp, i64, C.POINTER(PartitionParams), vp, vp, sz, vp]
        L.ewsjf_partition.restype = C.c_int
        L.ewsjf_route.argtypes = [vp, i64, vp, vp, vp]
        L.ewsjf_route.restype = C.c_int
        L.ewsjf_score.argtypes = [vp, vp, i64, f32, vp, vp, i32, C.POINTER(Cost), vp, vp]
        L.ewsjf_score.restype = C.c_int
        L.ewsjf_select.argtypes = [vp, i64, i32, i32, vp, vp, vp, vp, sz, vp]
        L.ewsjf_select.restype = C.c_int
        L.ewsjf_step.argtypes = [vp, vp, i64, f32, vp, vp, i32, C.POINTER(Cost), i32, i32, vp, vp, vp, vp, sz, vp]
        L.ewsjf_step.restype = C.c_int
        L.ewsjf_step_timed.argtypes = [vp, vp, i64, f32, vp, vp, i32, C.POINTER(Cost), i32, i32, vp, vp, vp, vp, sz,
                                       vp, vp]
        L.ewsjf_step_timed.restype = C.c_int
        L.ewsjf_step_static.argtypes = [vp, vp, i64, f32, vp, vp, i32, C.POINTER(Cost), i32, i32, vp, vp, vp, vp]
        L.ewsjf_step_static.restype = C.c_int
        L.ewsjf_ring_insert.argtypes = [vp, vp, i64, i64, vp, i64, i64, vp, vp, i64, vp]
        L.ewsjf_ring_insert.restype = C.c_int
        L.ewsjf_tactical_step.argtypes = [vp, vp, i64, f32, vp, vp, C.POINTER(Cost), i32, i32, vp, C.c_double, i32,
                                          vp, vp, vp, vp, vp, vp, sz, vp]
        L.ewsjf_tactical_step.restype = C.c_int
        L.ewsjf_ring_step.argtypes = [vp, vp, i64, i64, vp, i64, i64, vp, vp, i64, f32, vp, vp, C.POINTER(Cost), i32,
                                      i32, vp, vp, vp, vp, sz, vp]
        L.ewsjf_ring_step.restype = C.c_int
        L.ewsjf_window_histogram.argtypes = [vp, i64, i64, i64, i32, vp, vp]
        L.ewsjf_window_histogram.restype = C.c_int
        L.ewsjf_window_advance.argtypes = [vp, i64, i64, i64, i64, i32, vp, vp]
        L.ewsjf_window_advance.restype = C.c_int
        L.ewsjf_trial_step.argtypes = [vp, vp, i64, i32, i64, vp, vp, i64, f32, vp, vp, C.POINTER(Cost), i32, vp, vp,
                                       vp, vp, vp, vp, sz, vp]
        L.ewsjf_trial_step.restype = C.c_int
        L.ewsjf_trial_finish.argtypes = [vp, vp, i64, i32, f32, vp, vp, C.POINTER(C.c_double), vp, vp, vp]
        L.ewsjf_trial_finish.restype = C.c_int
        L.ewsjf_dispatch.argtypes = [vp, vp, i64, vp, i32, i32, vp, vp]
        L.ewsjf_dispatch.restype = C.c_int
        L.ewsjf_partition_hist.argtypes = [vp, C.POINTER(PartitionParams), vp, vp, sz, vp]
        L.ewsjf_partition_hist.restype = C.c_int
        L.ewsjf_status_string.argtypes = [C.c_int]
        L.ewsjf_status_string.restype = C.c_char_p
        L.ewsjf_version.argtypes = []
        L.ewsjf_version.restype = i32
        _lib = L
    return _lib


def status_string(s: int) -> str:
    try:
        return lib().ewsjf_status_string(int(s)).decode()
    except RuntimeError:
        return "library not loaded"


def check(status: int, what: str) -> None:
    if status != OK:
        raise EwsjfError(status, what)
