"""CPU oracle for the paged-KV hot path of LiveServe (arXiv 2606.22983).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
benchmark's ``cpu_baseline`` leg may import this package.  It is a plain fp64
CPU reference written from the definitions (see ``oracle.c``); it shares no
code with the GPU library and never imports it.

Entry points (numpy in, numpy out; bf16 arrays are ``uint16`` bit patterns):

* :func:`attend`  — exact softmax attention rows over block-table-addressed keys.
* :func:`append`  — write new tokens' K/V rows into their pool slots.
* :func:`stash` / :func:`restore` — block-granular byte copies between the pool
  and a contiguous staging array (the offload / reload of §5 and §5.2).
* :func:`decode` / :func:`prefill` — the two attention calls of the hot path,
  composed as "append into a private copy of the pool, then attend".
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import time

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile ``oracle.c`` into ``liboracle.so`` with gcc and OpenMP."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-fopenmp", "-shared", "-fPIC", "-std=c11", _SRC, "-o", tmp, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build(force=False)
        lib = ctypes.CDLL(_LIB)
        p, i32, i64, dbl = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_double
        lib.oracle_attend.argtypes = [p, i32, i64, i32, i32, i32, i32, i32, p, i32, i32, p, p, p, p,
                                      dbl, p]
        lib.oracle_append.argtypes = [p, i32, i64, i32, i32, i32, i32, p, i32, i32, p, p, p, p]
        lib.oracle_stash.argtypes = [p, i32, i64, i32, i32, i32, i32, p, p]
        lib.oracle_restore.argtypes = [p, i32, i64, i32, i32, i32, i32, p, p]
        for f in (lib.oracle_attend, lib.oracle_append, lib.oracle_stash, lib.oracle_restore):
            f.restype = ctypes.c_int
        _lib = lib
    return _lib


def _ptr(a: np.ndarray):
    assert a.flags["C_CONTIGUOUS"], "oracle arrays must be C-contiguous"
    return a.ctypes.data_as(ctypes.c_void_p)


def _geometry(pool: np.ndarray):
    """pool shape: [layers][blocks][2][kv_heads][block_size * head_dim] (uint16)."""
    if pool.dtype != np.uint16 or pool.ndim != 5 or pool.shape[2] != 2:
        raise ValueError("pool must be uint16 [layers][blocks][2][kv_heads][tile]")
    return pool.shape[0], pool.shape[1], pool.shape[3], pool.shape[4]


def attend(pool, block_size, head_dim, layer, q, block_tables, row_session, row_keys,
           row_q_index, scale):
    """out[r][h][:] = softmax(scale * q_r,h . K_s[:n]) V_s[:n] with n = row_keys[r].

    ``q`` is uint16 [num_q_rows][Hq][D]; row r reads q[row_q_index[r]].
    Returns fp64 [rows][Hq][D].
    """
    nl, nb, hkv, tile = _geometry(pool)
    assert tile == block_size * head_dim
    q = np.ascontiguousarray(q, dtype=np.uint16)
    hq = q.shape[1]
    bt = np.ascontiguousarray(block_tables, dtype=np.int32)
    rs = np.ascontiguousarray(row_session, dtype=np.int32)
    rk = np.ascontiguousarray(row_keys, dtype=np.int32)
    rq = np.ascontiguousarray(row_q_index, dtype=np.int64)
    out = np.zeros((len(rs), hq, head_dim), dtype=np.float64)
    rc = _load().oracle_attend(_ptr(pool), nl, nb, hkv, head_dim, block_size, layer, hq, _ptr(bt),
                               bt.shape[1], len(rs), _ptr(rs), _ptr(rk), _ptr(rq), _ptr(q),
                               float(scale), _ptr(out))
    if rc != 0:
        raise ValueError("oracle_attend: empty row or block id outside the pool")
    return out


def append(pool, block_size, head_dim, layer, block_tables, tok_session, tok_pos, k_new, v_new):
    """Write k_new/v_new [T][Hkv][D] at (session, position) slots, in place."""
    nl, nb, hkv, tile = _geometry(pool)
    bt = np.ascontiguousarray(block_tables, dtype=np.int32)
    ts = np.ascontiguousarray(tok_session, dtype=np.int32)
    tp = np.ascontiguousarray(tok_pos, dtype=np.int32)
    kn = np.ascontiguousarray(k_new, dtype=np.uint16)
    vn = np.ascontiguousarray(v_new, dtype=np.uint16)
    rc = _load().oracle_append(_ptr(pool), nl, nb, hkv, head_dim, block_size, layer, _ptr(bt),
                               bt.shape[1], len(ts), _ptr(ts), _ptr(tp), _ptr(kn), _ptr(vn))
    if rc != 0:
        raise ValueError("oracle_append: slot outside the block table or pool")
    return pool


def stash(pool, block_size, head_dim, ids):
    """staging[i][layer] = pool[layer][ids[i]] (uint16 [n][layers][2][Hkv][tile])."""
    nl, nb, hkv, tile = _geometry(pool)
    ids = np.ascontiguousarray(ids, dtype=np.int32)
    staging = np.empty((len(ids), nl, 2, hkv, tile), dtype=np.uint16)
    rc = _load().oracle_stash(_ptr(pool), nl, nb, hkv, head_dim, block_size, len(ids), _ptr(ids),
                              _ptr(staging))
    if rc != 0:
        raise ValueError("oracle_stash: block id outside the pool")
    return staging


def restore(pool, block_size, head_dim, ids, staging):
    """pool[layer][ids[i]] = staging[i][layer], in place."""
    nl, nb, hkv, tile = _geometry(pool)
    ids = np.ascontiguousarray(ids, dtype=np.int32)
    staging = np.ascontiguousarray(staging, dtype=np.uint16)
    rc = _load().oracle_restore(_ptr(pool), nl, nb, hkv, head_dim, block_size, len(ids),
                                _ptr(ids), _ptr(staging))
    if rc != 0:
        raise ValueError("oracle_restore: block id outside the pool")
    return pool


def decode(pool, block_size, head_dim, layer, q, block_tables, context_lens, scale,
           k_new=None, v_new=None, sessions=None, pool_out=False):
    """One decode step: optional append of this step's token at position L_s,
    then attention of q[s] over L_s (+1 when appended) keys.

    ``sessions`` selects a subset of sessions to evaluate (all by default).
    Returns fp64 [len(sessions)][Hq][D], and the appended pool if pool_out.
    """
    lens = np.asarray(context_lens, dtype=np.int64)
    work = pool
    if k_new is not None:
        work = pool.copy()
        s_all = np.arange(len(lens), dtype=np.int32)
        append(work, block_size, head_dim, layer, block_tables, s_all, lens.astype(np.int32),
               k_new, v_new)
        lens = lens + 1
    sel = np.arange(len(lens)) if sessions is None else np.asarray(sessions)
    out = attend(work, block_size, head_dim, layer, q, block_tables, sel, lens[sel], sel, scale)
    return (out, work) if pool_out else out


def prefill(pool, block_size, head_dim, layer, q, k_new, v_new, cu_new_lens, reused_lens,
            block_tables, scale, rows=None, pool_out=False):
    """Next-turn prefill: append the turn's n_s tokens at positions c_s .. c_s+n_s-1,
    then new row j of session s attends to keys 0 .. c_s + j.

    ``rows`` selects global new-token indices to evaluate (all by default).
    Returns fp64 [len(rows)][Hq][D], and the appended pool if pool_out.
    """
    cu = np.asarray(cu_new_lens, dtype=np.int64)
    c = np.asarray(reused_lens, dtype=np.int64)
    total = int(cu[-1])
    tok_session = np.repeat(np.arange(len(c)), np.diff(cu)).astype(np.int32)
    tok_pos = (c[tok_session] + np.arange(total) - cu[tok_session]).astype(np.int32)
    work = pool
    if k_new is not None:
        work = pool.copy()
        append(work, block_size, head_dim, layer, block_tables, tok_session, tok_pos, k_new, v_new)
    sel = np.arange(total) if rows is None else np.asarray(rows, dtype=np.int64)
    out = attend(work, block_size, head_dim, layer, q, block_tables, tok_session[sel],
                 tok_pos[sel] + 1, sel, scale)
    return (out, work) if pool_out else out


def timed(fn, *args, **kwargs):
    """Run fn and return (result, seconds) — used by the benchmark's cpu_baseline leg."""
    t0 = time.perf_counter()
    r = fn(*args, **kwargs)
    return r, time.perf_counter() - t0


def num_threads() -> int:
    """Threads OpenMP will use for the oracle (OMP_NUM_THREADS or the affinity set)."""
    env = os.environ.get("OMP_NUM_THREADS")
    if env and env.strip().isdigit():
        return int(env)
    return len(os.sched_getaffinity(0))
