"""Python binding of ``ls_schedule_round`` (interaction-aware batch selection
of one stage and one round) — argument marshalling only; the ordering and the
budget scan run in the library."""
from __future__ import annotations

import ctypes
from typing import Tuple

import numpy as np

from paper_2606_22983_amd import kv as _kv

_lib = _kv.raw_library()

REQUEST_DTYPE = np.dtype([("playback_buffer_s", "<f8"), ("ready_age_s", "<f8"), ("first_audio_done", "<i4"),
                          ("reserved", "<i4"), ("kv_blocks_held", "<i8"), ("tokens_needed", "<i8"),
                          ("kv_blocks_needed", "<i8")])


class _Stage(ctypes.Structure):
    _fields_ = [("p_safe_s", ctypes.c_double), ("alpha", ctypes.c_double), ("beta", ctypes.c_double),
                ("kv_occupancy", ctypes.c_double), ("token_budget", ctypes.c_int64),
                ("kv_block_budget", ctypes.c_int64)]


_lib.ls_schedule_round.argtypes = [ctypes.POINTER(_Stage), ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p,
                                   ctypes.c_void_p, ctypes.c_void_p, ctypes.POINTER(ctypes.c_int32)]
_lib.ls_schedule_round.restype = ctypes.c_int


def requests(n: int) -> np.ndarray:
    """A zeroed request table (fill its fields, then pass it to ls_schedule_round)."""
    return np.zeros(n, dtype=REQUEST_DTYPE)


def ls_schedule_round(reqs: np.ndarray, p_safe_s: float, alpha: float, beta: float, kv_occupancy: float,
                      token_budget: int, kv_block_budget: int) -> Tuple[np.ndarray, int, np.ndarray, np.ndarray]:
    """(order, num_admitted, classes, utility): order[:num_admitted] is the batch."""
    reqs = np.ascontiguousarray(reqs, dtype=REQUEST_DTYPE)
    n = len(reqs)
    order = np.zeros(max(n, 1), np.int32)
    classes = np.zeros(max(n, 1), np.int32)
    util = np.zeros(max(n, 1), np.float64)
    adm = ctypes.c_int32(0)
    st = _Stage(p_safe_s, alpha, beta, kv_occupancy, token_budget, kv_block_budget)
    _kv._check(_lib.ls_schedule_round(ctypes.byref(st), n, reqs.ctypes.data, order.ctypes.data,
                                      classes.ctypes.data, util.ctypes.data, ctypes.byref(adm)),
               "ls_schedule_round")
    return order[:n], adm.value, classes[:n], util[:n]
