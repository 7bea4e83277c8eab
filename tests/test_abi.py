"""The C-ABI library loads, exports every entry point its header declares, and
rejects invalid arguments on the host before touching a device (no GPU needed)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "liveserve_kv.h")

LS_OK, LS_EINVAL, LS_ENOMEM, LS_EUNSUPPORTED = 0, -22, -12, -95


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"^\s*(?:const\s+)?[A-Za-z_][\w\s\*]*?\b([a-z_][a-z0-9_]*)\s*\(", text, flags=re.M)
    return sorted(set(n for n in names if n not in ("defined",)))


class Desc(ctypes.Structure):
    _fields_ = [("num_layers", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("block_size", ctypes.c_int32),
                ("num_blocks", ctypes.c_int64), ("kv_base", ctypes.c_void_p),
                ("kv_bytes", ctypes.c_size_t), ("staging_ring", ctypes.c_void_p),
                ("staging_ring_bytes", ctypes.c_size_t)]


@pytest.fixture(scope="module")
def lib(built_lib):
    L = ctypes.CDLL(built_lib)
    L.ls_last_error.restype = ctypes.c_char_p
    L.ls_version.restype = ctypes.c_char_p
    L.ls_kv_pool_bytes.restype = ctypes.c_size_t
    L.ls_kv_pool_bytes.argtypes = [ctypes.c_int32, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                                   ctypes.c_int32]
    L.kv_pool_create.argtypes = [ctypes.POINTER(Desc), ctypes.POINTER(ctypes.c_void_p)]
    L.ls_decode_workspace_bytes.restype = ctypes.c_size_t
    L.ls_decode_workspace_bytes.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
                                            ctypes.c_int32]
    return L


def test_header_declares_the_five_entry_points():
    names = declared_functions()
    for n in ("kv_pool_create", "paged_attn_decode", "paged_attn_prefill", "kv_blocks_restore",
              "kv_blocks_stash"):
        assert n in names
    assert len(names) >= 10


def test_every_declared_symbol_is_exported(lib):
    for n in declared_functions():
        assert hasattr(lib, n), "missing export: " + n


def test_version_and_pool_bytes(lib):
    assert b"gfx950" in lib.ls_version()
    assert lib.ls_kv_pool_bytes(48, 65536, 4, 128, 16) == 48 * 65536 * 2 * 4 * 16 * 128 * 2
    assert lib.ls_kv_pool_bytes(0, 10, 4, 128, 16) == 0


def _desc(**kw):
    d = dict(num_layers=2, num_kv_heads=4, head_dim=128, block_size=16, num_blocks=100,
             kv_base=0x100000, kv_bytes=2 * 100 * 2 * 4 * 16 * 128 * 2, staging_ring=None,
             staging_ring_bytes=0)
    d.update(kw)
    return Desc(**d)


@pytest.mark.parametrize("kw,status", [
    (dict(block_size=32), LS_EUNSUPPORTED),
    (dict(head_dim=96), LS_EUNSUPPORTED),
    (dict(num_layers=0), LS_EINVAL),
    (dict(kv_base=None), LS_EINVAL),
    (dict(kv_base=0x100010), LS_EINVAL),
    (dict(kv_bytes=1000), LS_ENOMEM),
    (dict(num_blocks=1 << 40), LS_EINVAL),
])
def test_pool_create_rejects(lib, kw, status):
    h = ctypes.c_void_p()
    assert lib.kv_pool_create(ctypes.byref(_desc(**kw)), ctypes.byref(h)) == status
    assert h.value is None
    assert lib.ls_last_error() != b""


@pytest.fixture()
def pool(lib):
    h = ctypes.c_void_p()
    assert lib.kv_pool_create(ctypes.byref(_desc()), ctypes.byref(h)) == LS_OK
    yield h
    lib.kv_pool_destroy(h)


F = 0x200000  # a fake, never dereferenced, device address


def _decode(lib, pool, **kw):
    a = dict(layer=0, S=4, hq=32, q=F, kn=None, vn=None, bt=F, maxb=8, lens=F, scale=0.088,
             out=F, ws=F, wsb=1 << 30)
    a.update(kw)
    return lib.paged_attn_decode(pool, a["layer"], a["S"], a["hq"], ctypes.c_void_p(a["q"]),
                                 ctypes.c_void_p(a["kn"]), ctypes.c_void_p(a["vn"]),
                                 ctypes.c_void_p(a["bt"]), a["maxb"], ctypes.c_void_p(a["lens"]),
                                 ctypes.c_float(a["scale"]), ctypes.c_void_p(a["out"]),
                                 ctypes.c_void_p(a["ws"]), ctypes.c_size_t(a["wsb"]), None)


@pytest.mark.parametrize("kw,status", [
    (dict(layer=2), LS_EINVAL),
    (dict(hq=30), LS_EINVAL),
    (dict(hq=64), LS_EUNSUPPORTED),
    (dict(q=None), LS_EINVAL),
    (dict(kn=F), LS_EINVAL),
    (dict(maxb=0), LS_EINVAL),
    (dict(scale=0.0), LS_EINVAL),
    (dict(scale=float("nan")), LS_EINVAL),
    (dict(wsb=16), LS_ENOMEM),
])
def test_decode_rejects_before_launch(lib, pool, kw, status):
    assert _decode(lib, pool, **kw) == status


def test_decode_zero_sessions_is_noop(lib, pool):
    assert _decode(lib, pool, S=0, q=None) == LS_OK


def test_decode_null_pool(lib):
    assert _decode(lib, None) == LS_EINVAL


def test_workspace_query(lib, pool):
    ws = lib.ls_decode_workspace_bytes(pool, 64, 32, 1024)
    assert ws > 64 * 32 * 128 * 4
    assert lib.ls_decode_workspace_bytes(pool, 0, 32, 1024) == 0


def _prefill(lib, pool, **kw):
    a = dict(layer=0, S=2, hq=32, q=F, kn=None, vn=None, cu=F, ctx=F, total=100, maxn=60, bt=F,
             maxb=8, scale=0.088, out=F)
    a.update(kw)
    return lib.paged_attn_prefill(pool, a["layer"], a["S"], a["hq"], ctypes.c_void_p(a["q"]),
                                  ctypes.c_void_p(a["kn"]), ctypes.c_void_p(a["vn"]),
                                  ctypes.c_void_p(a["cu"]), ctypes.c_void_p(a["ctx"]), a["total"],
                                  a["maxn"], ctypes.c_void_p(a["bt"]), a["maxb"],
                                  ctypes.c_float(a["scale"]), ctypes.c_void_p(a["out"]), None)


@pytest.mark.parametrize("kw,status", [
    (dict(layer=-1), LS_EINVAL),
    (dict(hq=33), LS_EINVAL),
    (dict(cu=None), LS_EINVAL),
    (dict(vn=F), LS_EINVAL),
    (dict(maxn=200), LS_EINVAL),
    (dict(total=-1), LS_EINVAL),
])
def test_prefill_rejects_before_launch(lib, pool, kw, status):
    assert _prefill(lib, pool, **kw) == status


def test_prefill_empty_is_noop(lib, pool):
    assert _prefill(lib, pool, total=0, maxn=0, q=None) == LS_OK


@pytest.mark.parametrize("fn", ["kv_blocks_restore", "kv_blocks_stash"])
@pytest.mark.parametrize("ids,status", [([3, 7, 3], LS_EINVAL), ([3, 100], LS_EINVAL),
                                        ([-1], LS_EINVAL)])
def test_copy_rejects_bad_host_ids(lib, pool, fn, ids, status):
    arr = (ctypes.c_int32 * len(ids))(*ids)
    r = getattr(lib, fn)(pool, len(ids), ctypes.c_void_p(F), arr, ctypes.c_void_p(F), 0, None)
    assert r == status
    msg = lib.ls_last_error()
    assert b"twice" in msg or b"outside" in msg


@pytest.mark.parametrize("fn", ["kv_blocks_restore", "kv_blocks_stash"])
def test_copy_host_staging_needs_ring(lib, pool, fn):
    arr = (ctypes.c_int32 * 2)(1, 2)
    assert getattr(lib, fn)(pool, 2, ctypes.c_void_p(F), arr, ctypes.c_void_p(F), 1, None) == LS_ENOMEM


@pytest.mark.parametrize("fn", ["kv_blocks_restore", "kv_blocks_stash"])
def test_copy_zero_blocks_is_noop(lib, pool, fn):
    assert getattr(lib, fn)(pool, 0, None, None, None, 0, None) == LS_OK
    assert getattr(lib, fn)(pool, -1, None, None, None, 0, None) == LS_EINVAL
