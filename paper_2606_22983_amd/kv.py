"""Python binding of ``libliveserve_kv.so`` — argument marshalling only.

Every function here has the name of the C entry point it calls and passes
device pointers of torch tensors (PyTorch provides device memory and streams)
plus the current HIP stream.  All work runs in the library's HIP kernels; there
is no fallback.  Importing this module raises ``ImportError`` when the library
has not been built (``python -m paper_2606_22983_amd.build``).
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libliveserve_kv.so")
if not os.path.exists(LIB_PATH):
    raise ImportError("libliveserve_kv.so is not built; run `python -m paper_2606_22983_amd.build`")

_lib = ctypes.CDLL(LIB_PATH)

_p, _i32, _i64, _sz, _f32 = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t,
                             ctypes.c_float)


class _PoolDesc(ctypes.Structure):
    _fields_ = [("num_layers", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("block_size", ctypes.c_int32),
                ("num_blocks", ctypes.c_int64), ("kv_base", ctypes.c_void_p),
                ("kv_bytes", ctypes.c_size_t)]


_lib.ls_kv_pool_bytes.argtypes = [_i32, _i64, _i32, _i32, _i32]
_lib.ls_kv_pool_bytes.restype = _sz
_lib.kv_pool_create.argtypes = [ctypes.POINTER(_PoolDesc), ctypes.POINTER(_p)]
_lib.kv_pool_destroy.argtypes = [_p]
_lib.ls_decode_workspace_bytes.argtypes = [_p, _i32, _i32, _i32]
_lib.ls_decode_workspace_bytes.restype = _sz
_lib.paged_attn_decode.argtypes = [_p, _i32, _i32, _i32, _p, _p, _p, _p, _i32, _p, _p, _f32, _p,
                                   _p, _sz, _p]
_lib.ls_decode_schedule.argtypes = [_p, _i32, _i32, _i32, _p, _i32, _p, ctypes.POINTER(_i32),
                                    ctypes.POINTER(_i32), ctypes.POINTER(_i32)]
_lib.ls_decode_schedule.restype = ctypes.c_int
_lib.paged_attn_decode_static.argtypes = [_p, _i32, _i32, _i32, _p, _p, _p, _p, _i32, _p, _p, _f32,
                                          _p, _p]
_lib.paged_attn_prefill.argtypes = [_p, _i32, _i32, _i32, _p, _p, _p, _p, _p, _p, _i32, _i32, _p,
                                    _i32, _f32, _p, _p, _sz, _p]
_f64 = ctypes.c_double
_lib.kv_blocks_stash.argtypes = [_p, _i32, _p, _p, _p, _sz, _i32, _p, _sz, _f64, _p]
_lib.kv_blocks_restore.argtypes = [_p, _i32, _p, _p, _p, _sz, _i32, _p, _sz, _f64, _p]
_lib.kv_blocks_restore_layers.argtypes = [_p, _i32, _i32, _i32, _p, _p, _p, _sz, _i32, _p, _sz,
                                          _f64, _p]
_lib.ls_device_errors.argtypes = [ctypes.POINTER(ctypes.c_uint32)]
_lib.ls_last_error.restype = ctypes.c_char_p
_lib.ls_version.restype = ctypes.c_char_p
for _f in (_lib.kv_pool_create, _lib.kv_pool_destroy, _lib.paged_attn_decode,
           _lib.paged_attn_decode_static,
           _lib.paged_attn_prefill, _lib.kv_blocks_stash, _lib.kv_blocks_restore,
           _lib.kv_blocks_restore_layers,
           _lib.ls_device_errors):
    _f.restype = ctypes.c_int

LS_OK, LS_EINVAL, LS_ENOMEM, LS_EHIP, LS_EUNSUPPORTED = 0, -22, -12, -5, -95
LS_DEVERR_BLOCK_ID, LS_DEVERR_LENGTH, LS_DEVERR_INTERNAL = 0x1, 0x2, 0x4
PREFILL_WORKSPACE_BYTES = 256     # LS_PREFILL_WORKSPACE_BYTES


class LiveServeError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        msg = _lib.ls_last_error().decode(errors="replace")
        super().__init__("%s failed with status %d: %s" % (where, status, msg))


def _check(status: int, where: str):
    if status != LS_OK:
        raise LiveServeError(status, where)


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _shape(t: torch.Tensor, name: str, shape, dtype=None):
    """Check shape (None = any extent) and dtype; no device access."""
    if dtype is not None and t.dtype not in (dtype if isinstance(dtype, tuple) else (dtype,)):
        raise ValueError("%s must have dtype %s (got %s)" % (name, dtype, t.dtype))
    if len(t.shape) != len(shape) or any(e is not None and e != a for e, a in zip(shape, t.shape)):
        want = "[" + "][".join("*" if e is None else str(e) for e in shape) + "]"
        raise ValueError("%s must have shape %s (got %s)" % (name, want, list(t.shape)))
    return t


def _dev(t: torch.Tensor, name: str, dtype=None):
    if dtype is not None and t.dtype not in (dtype if isinstance(dtype, tuple) else (dtype,)):
        raise ValueError("%s must have dtype %s (got %s)" % (name, dtype, t.dtype))
    if not t.is_cuda:
        raise ValueError("%s must be a device tensor" % name)
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    return t


def _nbytes(t: torch.Tensor) -> int:
    return t.numel() * t.element_size()


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


_BF16 = (torch.bfloat16, torch.int16)


def version() -> str:
    return _lib.ls_version().decode()


def ls_kv_pool_bytes(num_layers, num_blocks, num_kv_heads, head_dim, block_size=16) -> int:
    return int(_lib.ls_kv_pool_bytes(num_layers, num_blocks, num_kv_heads, head_dim, block_size))


class KVPool:
    """Handle of a pool created by :func:`kv_pool_create` (keeps its tensor alive)."""

    def __init__(self, handle, kv, num_layers, num_blocks, num_kv_heads, head_dim, block_size):
        self.handle = handle
        self.kv = kv
        self.num_layers = num_layers
        self.num_blocks = num_blocks
        self.num_kv_heads = num_kv_heads
        self.head_dim = head_dim
        self.block_size = block_size

    @property
    def slab_bytes(self) -> int:
        """Bytes of one (layer, block) slab: K and V tiles of every KV head."""
        return 2 * self.num_kv_heads * self.block_size * self.head_dim * 2

    @property
    def block_bytes(self) -> int:
        """Bytes of one block's all-layer staging record."""
        return self.num_layers * self.slab_bytes

    def close(self):
        if self.handle:
            _lib.kv_pool_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def kv_pool_create(kv: torch.Tensor, num_layers: int, num_blocks: int, num_kv_heads: int,
                   head_dim: int, block_size: int = 16) -> KVPool:
    """Wrap ``kv`` (device memory of at least ``ls_kv_pool_bytes`` bytes) as a pool."""
    _dev(kv, "kv")
    desc = _PoolDesc(num_layers, num_kv_heads, head_dim, block_size, num_blocks,
                     kv.data_ptr(), _nbytes(kv))
    handle = ctypes.c_void_p()
    _check(_lib.kv_pool_create(ctypes.byref(desc), ctypes.byref(handle)), "kv_pool_create")
    return KVPool(handle, kv, num_layers, num_blocks, num_kv_heads, head_dim, block_size)


def decode_workspace_bytes(pool: KVPool, num_sessions: int, num_q_heads: int,
                           max_blocks_per_session: int) -> int:
    return int(_lib.ls_decode_workspace_bytes(pool.handle, num_sessions, num_q_heads,
                                              max_blocks_per_session))


def _host_i32(a, name: str, n: int):
    """Host int32 copy (kept alive by the caller) of an optional length array."""
    if a is None:
        return None, None
    arr = np.ascontiguousarray(np.asarray(a).reshape(-1), dtype=np.int32)
    if arr.size != n:
        raise ValueError("%s must hold %d values (got %d)" % (name, n, arr.size))
    return arr, ctypes.c_void_p(arr.ctypes.data)


def paged_attn_decode(pool: KVPool, layer: int, q: torch.Tensor, block_tables: torch.Tensor,
                      context_lens: torch.Tensor, scale: float, out: torch.Tensor,
                      workspace: torch.Tensor, k_new: Optional[torch.Tensor] = None,
                      v_new: Optional[torch.Tensor] = None, context_lens_host=None,
                      stream=None) -> torch.Tensor:
    """q/out: [S][Hq][D] bf16; block_tables int32 [S][maxb]; context_lens int32 [S];
    k_new/v_new [S][Hkv][D] bf16; context_lens_host: optional host copy of context_lens."""
    if q.dim() != 3:
        raise ValueError("q must be [S][Hq][D]")
    s, hq = q.shape[0], q.shape[1]
    d, hkv = pool.head_dim, pool.num_kv_heads
    _shape(q, "q", (s, hq, d), _BF16)
    _shape(out, "out", (s, hq, d), _BF16)
    _shape(block_tables, "block_tables", (s, None), torch.int32)
    _shape(context_lens, "context_lens", (s,), torch.int32)
    for t, name in ((k_new, "k_new"), (v_new, "v_new")):
        if t is not None:
            _shape(t, name, (s, hkv, d), _BF16)
    for t, name in ((q, "q"), (out, "out"), (block_tables, "block_tables"),
                    (context_lens, "context_lens"), (workspace, "workspace"), (k_new, "k_new"),
                    (v_new, "v_new")):
        if t is not None:
            _dev(t, name)
    keep, hl = _host_i32(context_lens_host, "context_lens_host", s)
    _check(_lib.paged_attn_decode(pool.handle, layer, s, hq, _ptr(q), _ptr(k_new), _ptr(v_new),
                                  _ptr(block_tables), block_tables.shape[1], _ptr(context_lens), hl,
                                  float(scale), _ptr(out), _ptr(workspace), _nbytes(workspace),
                                  _stream(stream)),
           "paged_attn_decode")
    del keep
    return out


def ls_decode_schedule(pool: KVPool, num_sessions: int, num_q_heads: int, max_blocks_per_session: int,
                       context_lens_host=None, appended: bool = False, stream=None) -> dict:
    """How paged_attn_decode will run this batch: split size, host-planned, merge."""
    keep, hl = _host_i32(context_lens_host, "context_lens_host", num_sessions)
    t, h, m = _i32(), _i32(), _i32()
    _check(_lib.ls_decode_schedule(pool.handle, num_sessions, num_q_heads, max_blocks_per_session, hl,
                                   1 if appended else 0, _stream(stream), ctypes.byref(t), ctypes.byref(h),
                                   ctypes.byref(m)), "ls_decode_schedule")
    del keep
    return {"split_tokens": t.value, "host_planned": bool(h.value), "merge": bool(m.value)}


def paged_attn_decode_static(pool: KVPool, layer: int, q: torch.Tensor, block_tables: torch.Tensor,
                             context_lens: torch.Tensor, scale: float, out: torch.Tensor,
                             k_new: Optional[torch.Tensor] = None, v_new: Optional[torch.Tensor] = None,
                             context_lens_host=None, stream=None) -> torch.Tensor:
    """paged_attn_decode with the library's static split scratch (no workspace)."""
    if q.dim() != 3:
        raise ValueError("q must be [S][Hq][D]")
    s, hq = q.shape[0], q.shape[1]
    d, hkv = pool.head_dim, pool.num_kv_heads
    _shape(q, "q", (s, hq, d), _BF16)
    _shape(out, "out", (s, hq, d), _BF16)
    _shape(block_tables, "block_tables", (s, None), torch.int32)
    _shape(context_lens, "context_lens", (s,), torch.int32)
    for t, name in ((k_new, "k_new"), (v_new, "v_new")):
        if t is not None:
            _shape(t, name, (s, hkv, d), _BF16)
    for t, name in ((q, "q"), (out, "out"), (block_tables, "block_tables"),
                    (context_lens, "context_lens"), (k_new, "k_new"), (v_new, "v_new")):
        if t is not None:
            _dev(t, name)
    keep, hl = _host_i32(context_lens_host, "context_lens_host", s)
    _check(_lib.paged_attn_decode_static(pool.handle, layer, s, hq, _ptr(q), _ptr(k_new), _ptr(v_new),
                                         _ptr(block_tables), block_tables.shape[1], _ptr(context_lens),
                                         hl, float(scale), _ptr(out), _stream(stream)),
           "paged_attn_decode_static")
    del keep
    return out


def paged_attn_prefill(pool: KVPool, layer: int, q: torch.Tensor, cu_new_lens: torch.Tensor,
                       reused_lens: torch.Tensor, max_new_len: int, block_tables: torch.Tensor,
                       scale: float, out: torch.Tensor, k_new: Optional[torch.Tensor] = None,
                       v_new: Optional[torch.Tensor] = None, lens_host=None,
                       workspace: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """q/out: [T][Hq][D] bf16; cu_new_lens int32 [S+1]; reused_lens int32 [S];
    k_new/v_new [T][Hkv][D] bf16; lens_host: optional host [S][2] of (n_s, c_s);
    workspace: optional device tensor of PREFILL_WORKSPACE_BYTES bytes (item
    counters that let faster XCDs take over the slower ones' last tiles; used
    with lens_host)."""
    if q.dim() != 3:
        raise ValueError("q must be [T][Hq][D]")
    total, hq = q.shape[0], q.shape[1]
    s = reused_lens.shape[0] if reused_lens.dim() == 1 else -1
    d, hkv = pool.head_dim, pool.num_kv_heads
    _shape(q, "q", (total, hq, d), _BF16)
    _shape(out, "out", (total, hq, d), _BF16)
    _shape(reused_lens, "reused_lens", (None,), torch.int32)
    _shape(cu_new_lens, "cu_new_lens", (s + 1,), torch.int32)
    _shape(block_tables, "block_tables", (s, None), torch.int32)
    for t, name in ((k_new, "k_new"), (v_new, "v_new")):
        if t is not None:
            _shape(t, name, (total, hkv, d), _BF16)
    for t, name in ((q, "q"), (out, "out"), (cu_new_lens, "cu_new_lens"),
                    (reused_lens, "reused_lens"), (block_tables, "block_tables"), (k_new, "k_new"),
                    (v_new, "v_new")):
        if t is not None:
            _dev(t, name)
    keep, hl = _host_i32(lens_host, "lens_host", 2 * s)
    if workspace is not None:
        _dev(workspace, "workspace")
    _check(_lib.paged_attn_prefill(pool.handle, layer, s, hq, _ptr(q), _ptr(k_new), _ptr(v_new),
                                   _ptr(cu_new_lens), _ptr(reused_lens), hl, total,
                                   int(max_new_len), _ptr(block_tables), block_tables.shape[1],
                                   float(scale), _ptr(out), _ptr(workspace),
                                   0 if workspace is None else _nbytes(workspace), _stream(stream)),
           "paged_attn_prefill")
    del keep
    return out


def _host_ids(ids):
    """Host int32 copy of the ids (kept alive by the caller) and its address."""
    if ids is None:
        return None, None
    arr = np.ascontiguousarray(ids, dtype=np.int32)
    return arr, ctypes.c_void_p(arr.ctypes.data)


def _copy_args(pool: KVPool, block_ids: torch.Tensor, staging: torch.Tensor, ring, max_gbps):
    """Checks shared by the block copies; returns (on_host, ring pointer, ring bytes)."""
    _shape(block_ids, "block_ids", (None,), torch.int32)
    if not staging.is_contiguous():
        raise ValueError("staging must be contiguous")
    if _nbytes(staging) < block_ids.numel() * pool.block_bytes:
        raise ValueError("staging holds %d bytes; %d blocks need %d" % (
            _nbytes(staging), block_ids.numel(), block_ids.numel() * pool.block_bytes))
    if not max_gbps >= 0:
        raise ValueError("max_gbps must be >= 0")
    _dev(block_ids, "block_ids")
    on_host = not staging.is_cuda
    if on_host and not staging.is_pinned():
        raise ValueError("host staging must be pinned memory")
    if ring is not None:
        _dev(ring, "ring")
    return on_host, _ptr(ring), 0 if ring is None else _nbytes(ring)


def kv_blocks_stash(pool: KVPool, block_ids: torch.Tensor, staging: torch.Tensor,
                    block_ids_host=None, ring: Optional[torch.Tensor] = None,
                    max_gbps: float = 0.0, stream=None) -> torch.Tensor:
    """Copy every layer's slab of ``block_ids`` into ``staging`` (device, or pinned host
    through the device ``ring``); ``max_gbps`` > 0 paces it to that payload rate."""
    on_host, rp, rb = _copy_args(pool, block_ids, staging, ring, max_gbps)
    keep, hp = _host_ids(block_ids_host)
    _check(_lib.kv_blocks_stash(pool.handle, block_ids.numel(), _ptr(block_ids), hp, _ptr(staging),
                                _nbytes(staging), 1 if on_host else 0, rp, rb, max_gbps,
                                _stream(stream)),
           "kv_blocks_stash")
    del keep
    return staging


def kv_blocks_restore(pool: KVPool, block_ids: torch.Tensor, staging: torch.Tensor,
                      block_ids_host=None, ring: Optional[torch.Tensor] = None,
                      max_gbps: float = 0.0, stream=None):
    """Copy ``staging`` (device, or pinned host through the device ``ring``) back into
    pool blocks ``block_ids``."""
    on_host, rp, rb = _copy_args(pool, block_ids, staging, ring, max_gbps)
    keep, hp = _host_ids(block_ids_host)
    _check(_lib.kv_blocks_restore(pool.handle, block_ids.numel(), _ptr(block_ids), hp,
                                  _ptr(staging), _nbytes(staging), 1 if on_host else 0, rp, rb,
                                  max_gbps, _stream(stream)),
           "kv_blocks_restore")
    del keep


def kv_blocks_restore_layers(pool: KVPool, layer_begin: int, layer_count: int, block_ids: torch.Tensor,
                             staging: torch.Tensor, block_ids_host=None,
                             ring: Optional[torch.Tensor] = None, max_gbps: float = 0.0,
                             stream=None):
    """Restore layers [layer_begin, layer_begin + layer_count) of ``block_ids`` from an
    all-layer ``staging`` (device, or pinned host through the device ``ring``)."""
    on_host, rp, rb = _copy_args(pool, block_ids, staging, ring, max_gbps)
    keep, hp = _host_ids(block_ids_host)
    _check(_lib.kv_blocks_restore_layers(pool.handle, layer_begin, layer_count, block_ids.numel(),
                                         _ptr(block_ids), hp, _ptr(staging), _nbytes(staging),
                                         1 if on_host else 0, rp, rb, max_gbps,
                                         _stream(stream)), "kv_blocks_restore_layers")
    del keep


def ls_device_errors() -> int:
    """Wait for all work on the device, then read and clear its error word."""
    bits = ctypes.c_uint32()
    _check(_lib.ls_device_errors(ctypes.byref(bits)), "ls_device_errors")
    return int(bits.value)


def raw_library():
    """The ctypes handle of the C library (tests call entry points through it)."""
    return _lib
