"""Python binding of the library's host-side KV manager (``kv_manager_*``) —
argument marshalling only.

The manager decides which blocks move between the HBM pool and the host store
(next-use-aware eviction with the indexed candidate heap, speech-triggered
preload with admission, cancellation and synchronous fallback); every decision
is made in the C++ library.  Moves come back as int32 arrays of shape (n, 4):
columns (session, position, device_block, host_slot).  The caller runs the
copies with :func:`paper_2606_22983_amd.kv.kv_blocks_stash` /
:func:`~paper_2606_22983_amd.kv.kv_blocks_restore`.
"""
from __future__ import annotations

import ctypes
import math
from typing import Dict, Tuple

import numpy as np

from paper_2606_22983_amd import kv as _kv

_lib = _kv.raw_library()
_p, _i32, _i64, _f64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_double
_pi32 = ctypes.POINTER(ctypes.c_int32)

LS_KV_RESIDENT, LS_KV_OFFLOADED, LS_KV_LOADING = 0, 1, 2
LS_KV_RUNNING, LS_KV_IMMEDIATE, LS_KV_WARM, LS_KV_EVICTABLE = 0x1, 0x2, 0x4, 0x8


class _Desc(ctypes.Structure):
    _fields_ = [("num_device_blocks", ctypes.c_int64), ("num_host_slots", ctypes.c_int64),
                ("max_sessions", ctypes.c_int32), ("reply_prior_s", ctypes.c_double),
                ("reply_ema_alpha", ctypes.c_double), ("seconds_per_token", ctypes.c_double),
                ("warm_ttl_s", ctypes.c_double), ("warm_cap_blocks", ctypes.c_int64)]


class _Move(ctypes.Structure):
    _fields_ = [("session", ctypes.c_int32), ("position", ctypes.c_int32),
                ("device_block", ctypes.c_int32), ("host_slot", ctypes.c_int32)]


_P_MOVE = ctypes.POINTER(_Move)
_SIGS = {
    "kv_manager_create": [ctypes.POINTER(_Desc), ctypes.POINTER(_p)],
    "kv_manager_destroy": [_p],
    "kv_manager_add_session": [_p, _i32],
    "kv_manager_remove_session": [_p, _i32],
    "kv_manager_append_blocks": [_p, _i32, _i32, _p],
    "kv_manager_set_running": [_p, _i32, _i32],
    "kv_manager_set_playback": [_p, _i32, _f64, _i64],
    "kv_manager_observe_reply": [_p, _i32, _f64],
    "kv_manager_speech_start": [_p, _i32],
    "kv_manager_evict": [_p, _i64, _p, _i32, _pi32],
    "kv_manager_preload": [_p, _i32, _f64, _f64, _f64, _p, _i32, _pi32, _p, _i32, _pi32, _pi32],
    "kv_manager_load_sync": [_p, _i32, _p, _i32, _pi32, _p, _i32, _pi32],
    "kv_manager_preload_done": [_p, _i32, _f64],
    "kv_manager_preload_cancel": [_p, _i32],
    "kv_manager_tick": [_p, _f64],
    "kv_manager_session_info": [_p, _i32, ctypes.POINTER(_f64), _pi32, _pi32],
    "kv_manager_table": [_p, _i32, _i32, _p, _p, _p],
    "kv_manager_counts": [_p, ctypes.POINTER(_i64), ctypes.POINTER(_i64), ctypes.POINTER(_i64),
                          ctypes.POINTER(_i64)],
}
for _name, _args in _SIGS.items():
    getattr(_lib, _name).argtypes = _args
    getattr(_lib, _name).restype = ctypes.c_int


def _moves(buf, n: int) -> np.ndarray:
    a = np.ctypeslib.as_array(ctypes.cast(buf, ctypes.POINTER(ctypes.c_int32)), shape=(max(n, 1) * 4,))
    return a[:n * 4].reshape(n, 4).copy()


class KVManager:
    """Handle of one ``ls_kv_manager``; methods are the ``kv_manager_*`` calls."""

    def __init__(self, num_device_blocks: int, num_host_slots: int, max_sessions: int,
                 reply_prior_s: float = 3.0, reply_ema_alpha: float = 0.5,
                 seconds_per_token: float = 0.04, warm_ttl_s: float = 5.0,
                 warm_cap_blocks: int = 1 << 40):
        self.handle = None
        d = _Desc(num_device_blocks, num_host_slots, max_sessions, reply_prior_s, reply_ema_alpha,
                  seconds_per_token, warm_ttl_s, warm_cap_blocks)
        h = _p()
        _kv._check(_lib.kv_manager_create(ctypes.byref(d), ctypes.byref(h)), "kv_manager_create")
        self.handle = h
        self.num_device_blocks = num_device_blocks

    def close(self):
        if self.handle:
            _lib.kv_manager_destroy(self.handle)
            self.handle = None

    def __del__(self):
        self.close()

    def add_session(self, session: int):
        _kv._check(_lib.kv_manager_add_session(self.handle, session), "kv_manager_add_session")

    def remove_session(self, session: int):
        _kv._check(_lib.kv_manager_remove_session(self.handle, session), "kv_manager_remove_session")

    def append_blocks(self, session: int, n: int) -> np.ndarray:
        out = np.zeros(max(n, 1), np.int32)
        _kv._check(_lib.kv_manager_append_blocks(self.handle, session, n, out.ctypes.data),
                   "kv_manager_append_blocks")
        return out[:n]

    def set_running(self, session: int, running: bool):
        _kv._check(_lib.kv_manager_set_running(self.handle, session, int(bool(running))),
                   "kv_manager_set_running")

    def set_playback(self, session: int, t_play_s: float, unfinished_tokens: int = 0):
        _kv._check(_lib.kv_manager_set_playback(self.handle, session, t_play_s, unfinished_tokens),
                   "kv_manager_set_playback")

    def observe_reply(self, session: int, interval_s: float):
        _kv._check(_lib.kv_manager_observe_reply(self.handle, session, interval_s),
                   "kv_manager_observe_reply")

    def speech_start(self, session: int):
        _kv._check(_lib.kv_manager_speech_start(self.handle, session), "kv_manager_speech_start")

    def evict(self, blocks_needed: int) -> np.ndarray:
        cap = max(int(blocks_needed), 1)
        buf = (_Move * cap)()
        n = ctypes.c_int32(0)
        _kv._check(_lib.kv_manager_evict(self.handle, blocks_needed, buf, cap, ctypes.byref(n)),
                   "kv_manager_evict")
        return _moves(buf, n.value)

    def _load(self, fn, session: int, *extra) -> Tuple[int, np.ndarray, np.ndarray]:
        cap = max(self.session_info(session)[2], 1)        # at most one move per table entry
        rb, eb = (_Move * cap)(), (_Move * cap)()
        nr, ne, adm = ctypes.c_int32(0), ctypes.c_int32(0), ctypes.c_int32(1)
        if fn == "kv_manager_preload":
            st = _lib.kv_manager_preload(self.handle, session, *extra, rb, cap, ctypes.byref(nr), eb, cap,
                                         ctypes.byref(ne), ctypes.byref(adm))
        else:
            st = _lib.kv_manager_load_sync(self.handle, session, rb, cap, ctypes.byref(nr), eb, cap,
                                           ctypes.byref(ne))
        _kv._check(st, fn)
        return adm.value, _moves(rb, nr.value), _moves(eb, ne.value)

    def preload(self, session: int, time_available_s: float, bytes_per_block: float,
                bandwidth_bytes_per_s: float) -> Tuple[bool, np.ndarray, np.ndarray]:
        """(admitted, restores, evictions); restores are prefix first."""
        adm, r, e = self._load("kv_manager_preload", session, time_available_s, bytes_per_block,
                               bandwidth_bytes_per_s)
        return bool(adm), r, e

    def load_sync(self, session: int) -> Tuple[np.ndarray, np.ndarray]:
        _, r, e = self._load("kv_manager_load_sync", session)
        return r, e

    def preload_done(self, session: int, now_s: float):
        _kv._check(_lib.kv_manager_preload_done(self.handle, session, now_s), "kv_manager_preload_done")

    def preload_cancel(self, session: int):
        _kv._check(_lib.kv_manager_preload_cancel(self.handle, session), "kv_manager_preload_cancel")

    def tick(self, now_s: float):
        _kv._check(_lib.kv_manager_tick(self.handle, now_s), "kv_manager_tick")

    def session_info(self, session: int) -> Tuple[float, int, int]:
        t, f, n = ctypes.c_double(math.nan), ctypes.c_int32(0), ctypes.c_int32(0)
        _kv._check(_lib.kv_manager_session_info(self.handle, session, ctypes.byref(t), ctypes.byref(f),
                                                ctypes.byref(n)), "kv_manager_session_info")
        return t.value, f.value, n.value

    def table(self, session: int) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
        n = self.session_info(session)[2]
        dev, host, state = (np.zeros(max(n, 1), np.int32) for _ in range(3))
        _kv._check(_lib.kv_manager_table(self.handle, session, n, dev.ctypes.data, host.ctypes.data,
                                         state.ctypes.data), "kv_manager_table")
        return dev[:n], host[:n], state[:n]

    def counts(self) -> Dict[str, int]:
        v = [ctypes.c_int64(0) for _ in range(4)]
        _kv._check(_lib.kv_manager_counts(self.handle, *[ctypes.byref(x) for x in v]), "kv_manager_counts")
        return dict(zip(("free_device_blocks", "free_host_slots", "evictable_blocks", "warm_blocks"),
                        (x.value for x in v)))


def kv_manager_create(num_device_blocks: int, num_host_slots: int, max_sessions: int, **kw) -> KVManager:
    return KVManager(num_device_blocks, num_host_slots, max_sessions, **kw)
