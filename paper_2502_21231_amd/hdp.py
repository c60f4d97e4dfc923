"""Python binding of libbs_hdp.so, the host-side HDP planners (argument marshalling only).

The planning itself runs in the native library; if it has not been built this module raises
instead of planning another way.  Plans are returned as (micro_batches, rank_time) with
micro_batches in assignment order as tuples (seqs, ranks, offload_ratio, start, time).
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libbs_hdp.so")

BS_HDP_OK, BS_HDP_ERR_INVALID_ARG, BS_HDP_ERR_INFEASIBLE, BS_HDP_ERR_CAPACITY = range(4)
NAIVE, DP_BALANCE, PP_BALANCE = range(3)
EXPORTS = ("bs_hdp_offload_ratio", "bs_hdp_plan", "bs_hdp_last_error")


class bs_hdp_cost(ctypes.Structure):
    _fields_ = [("alpha1", ctypes.c_double), ("beta1", ctypes.c_double), ("gamma", ctypes.c_double),
                ("alpha2", ctypes.c_double), ("beta2", ctypes.c_double), ("layers", ctypes.c_int32),
                ("bw_d2h", ctypes.c_double), ("bw_h2d", ctypes.c_double)]


class bs_hdp_microbatch(ctypes.Structure):
    _fields_ = [("seq_offset", ctypes.c_int32), ("n_seqs", ctypes.c_int32),
                ("rank_offset", ctypes.c_int32), ("n_ranks", ctypes.c_int32),
                ("offload_ratio", ctypes.c_double), ("start", ctypes.c_double),
                ("time", ctypes.c_double)]


class HdpError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"bs_hdp status {status}: {message}")
        self.status = status


_LIB = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    global _LIB
    if _LIB is not None:
        return _LIB
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with `python -m paper_2502_21231_amd.build`")
    lib = ctypes.CDLL(path)
    P, I32, I64, D = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_double
    lib.bs_hdp_offload_ratio.restype = ctypes.c_int
    lib.bs_hdp_offload_ratio.argtypes = [ctypes.POINTER(bs_hdp_cost), I64, I64,
                                         ctypes.POINTER(D), ctypes.POINTER(I32)]
    lib.bs_hdp_plan.restype = ctypes.c_int
    lib.bs_hdp_plan.argtypes = [ctypes.c_int, ctypes.POINTER(bs_hdp_cost), P, I32, I64, I32, D, I32,
                                P, I32, P, P, I64, ctypes.POINTER(I32), P]
    lib.bs_hdp_last_error.restype = ctypes.c_char_p
    lib.bs_hdp_last_error.argtypes = []
    _LIB = lib
    return lib


def _check(status: int) -> None:
    if status != BS_HDP_OK:
        raise HdpError(status, load_library().bs_hdp_last_error().decode())


def make_cost(alpha1, beta1, gamma, alpha2, beta2, layers, bw_d2h, bw_h2d) -> bs_hdp_cost:
    return bs_hdp_cost(alpha1, beta1, gamma, alpha2, beta2, layers, bw_d2h, bw_h2d)


def as_cost(c) -> bs_hdp_cost:
    """A bs_hdp_cost from any object with the fields alpha1 .. bw_h2d (or a bs_hdp_cost)."""
    if isinstance(c, bs_hdp_cost):
        return c
    return make_cost(c.alpha1, c.beta1, c.gamma, c.alpha2, c.beta2, c.layers, c.bw_d2h, c.bw_h2d)


def offload_ratio(s: int, capacity: int, cost) -> tuple[float, int]:
    r, d = ctypes.c_double(), ctypes.c_int32()
    c = as_cost(cost)
    _check(load_library().bs_hdp_offload_ratio(ctypes.byref(c), int(s), int(capacity),
                                               ctypes.byref(r), ctypes.byref(d)))
    return r.value, d.value


def plan(algorithm: int, lengths, capacity: int, d_hdp: int, cost, delta: float = 0.0,
         n_buckets: int = 4):
    lens = np.ascontiguousarray(np.asarray(lengths, dtype=np.int64))
    n = int(lens.shape[0])
    c = as_cost(cost)
    mbs = (bs_hdp_microbatch * max(n, 1))()
    seqs = np.empty(max(n, 1), dtype=np.int32)
    max_ranks = max(1, n * d_hdp)
    ranks = np.empty(max_ranks, dtype=np.int32)
    rank_time = np.empty(d_hdp, dtype=np.float64)
    n_mbs = ctypes.c_int32()
    _check(load_library().bs_hdp_plan(
        int(algorithm), ctypes.byref(c), lens.ctypes.data, n, int(capacity), int(d_hdp), float(delta),
        int(n_buckets), ctypes.cast(mbs, ctypes.c_void_p), max(n, 1), seqs.ctypes.data,
        ranks.ctypes.data, max_ranks, ctypes.byref(n_mbs), rank_time.ctypes.data))
    out = []
    for k in range(n_mbs.value):
        m = mbs[k]
        out.append((tuple(int(x) for x in seqs[m.seq_offset:m.seq_offset + m.n_seqs]),
                    tuple(int(x) for x in ranks[m.rank_offset:m.rank_offset + m.n_ranks]),
                    m.offload_ratio, m.start, m.time))
    return out, [float(x) for x in rank_time]
