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
                ("kv_bytes", ctypes.c_size_t)]


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
             kv_base=0x100000, kv_bytes=2 * 100 * 2 * 4 * 16 * 128 * 2)
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


def _i32s(v):
    return None if v is None else (ctypes.c_int32 * len(v))(*v)


def _decode(lib, pool, **kw):
    a = dict(layer=0, S=4, hq=32, q=F, kn=None, vn=None, bt=F, maxb=8, lens=F, lens_host=None,
             scale=0.088, out=F, ws=F, wsb=1 << 30)
    a.update(kw)
    return lib.paged_attn_decode(pool, a["layer"], a["S"], a["hq"], ctypes.c_void_p(a["q"]),
                                 ctypes.c_void_p(a["kn"]), ctypes.c_void_p(a["vn"]),
                                 ctypes.c_void_p(a["bt"]), a["maxb"], ctypes.c_void_p(a["lens"]),
                                 _i32s(a["lens_host"]), ctypes.c_float(a["scale"]),
                                 ctypes.c_void_p(a["out"]), ctypes.c_void_p(a["ws"]),
                                 ctypes.c_size_t(a["wsb"]), None)


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
    # past the batch limits: 2049 sessions, 16385 blocks per session
    (dict(S=2049), LS_EUNSUPPORTED),
    (dict(maxb=16385), LS_EUNSUPPORTED),
    # host lengths: an empty context, a negative one, keys past the 8-block table
    (dict(lens_host=[5, 0, 7, 9]), LS_EINVAL),
    (dict(lens_host=[5, -1, 7, 9], kn=F, vn=F), LS_EINVAL),
    (dict(lens_host=[5, 129, 7, 9]), LS_EINVAL),
    (dict(lens_host=[5, 128, 7, 9], kn=F, vn=F), LS_EINVAL),
])
def test_decode_rejects_before_launch(lib, pool, kw, status):
    assert _decode(lib, pool, **kw) == status
    assert lib.ls_last_error() != b""


def test_decode_zero_sessions_is_noop(lib, pool):
    assert _decode(lib, pool, S=0, q=None) == LS_OK


def test_decode_null_pool(lib):
    assert _decode(lib, None) == LS_EINVAL


def test_workspace_query(lib, pool):
    ws = lib.ls_decode_workspace_bytes(pool, 64, 32, 1024)
    assert ws > 64 * 32 * 128 * 4
    assert lib.ls_decode_workspace_bytes(pool, 0, 32, 1024) == 0


def _prefill(lib, pool, **kw):
    a = dict(layer=0, S=2, hq=32, q=F, kn=None, vn=None, cu=F, ctx=F, lens_host=None, total=100,
             maxn=60, bt=F, maxb=8, scale=0.088, out=F, ws=None, wsb=0)
    a.update(kw)
    return lib.paged_attn_prefill(pool, a["layer"], a["S"], a["hq"], ctypes.c_void_p(a["q"]),
                                  ctypes.c_void_p(a["kn"]), ctypes.c_void_p(a["vn"]),
                                  ctypes.c_void_p(a["cu"]), ctypes.c_void_p(a["ctx"]),
                                  _i32s(a["lens_host"]), a["total"], a["maxn"],
                                  ctypes.c_void_p(a["bt"]), a["maxb"], ctypes.c_float(a["scale"]),
                                  ctypes.c_void_p(a["out"]), ctypes.c_void_p(a["ws"]),
                                  ctypes.c_size_t(a["wsb"]), None)


@pytest.mark.parametrize("kw,status", [
    (dict(layer=-1), LS_EINVAL),
    (dict(hq=33), LS_EINVAL),
    (dict(cu=None), LS_EINVAL),
    (dict(vn=F), LS_EINVAL),
    (dict(maxn=200), LS_EINVAL),
    (dict(total=-1), LS_EINVAL),
    # host (n, c) pairs: a turn above max_new_len, lengths not adding up to the
    # total, keys past the 8-block table, a negative context
    (dict(lens_host=[61, 0, 39, 5]), LS_EINVAL),
    (dict(lens_host=[60, 0, 39, 5]), LS_EINVAL),
    (dict(lens_host=[60, 70, 40, 5]), LS_EINVAL),
    (dict(lens_host=[60, 0, 40, -1]), LS_EINVAL),
    # the item-counter workspace: too small, misaligned
    (dict(ws=F, wsb=255), LS_ENOMEM),
    (dict(ws=F + 8, wsb=256), LS_EINVAL),
])
def test_prefill_rejects_before_launch(lib, pool, kw, status):
    assert _prefill(lib, pool, **kw) == status
    assert lib.ls_last_error() != b""


def test_prefill_empty_is_noop(lib, pool):
    assert _prefill(lib, pool, total=0, maxn=0, q=None) == LS_OK


BLOCK = 2 * 2 * 4 * 16 * 128 * 2        # all-layer bytes of one block of the test pool


def _copy(lib, fn, pool, n, ids=F, ids_host=None, staging=F, staging_bytes=None, on_host=0,
          ring=None, ring_bytes=0, rate=0.0):
    if staging_bytes is None:
        staging_bytes = max(n, 0) * BLOCK
    return getattr(lib, fn)(pool, n, ctypes.c_void_p(ids), ids_host, ctypes.c_void_p(staging),
                            ctypes.c_size_t(staging_bytes), on_host, ctypes.c_void_p(ring),
                            ctypes.c_size_t(ring_bytes), ctypes.c_double(rate), None)


@pytest.mark.parametrize("fn", ["kv_blocks_restore", "kv_blocks_stash"])
@pytest.mark.parametrize("ids,status", [([3, 7, 3], LS_EINVAL), ([3, 100], LS_EINVAL),
                                        ([-1], LS_EINVAL)])
def test_copy_rejects_bad_host_ids(lib, pool, fn, ids, status):
    arr = (ctypes.c_int32 * len(ids))(*ids)
    assert _copy(lib, fn, pool, len(ids), ids_host=arr) == status
    msg = lib.ls_last_error()
    assert b"twice" in msg or b"outside" in msg


@pytest.mark.parametrize("fn", ["kv_blocks_restore", "kv_blocks_stash"])
@pytest.mark.parametrize("kw,status,word", [
    (dict(on_host=1), LS_ENOMEM, b"ring"),                                   # no ring
    (dict(on_host=1, ring=F, ring_bytes=BLOCK - 16), LS_ENOMEM, b"ring"),    # ring below one block
    (dict(on_host=1, ring=F + 8, ring_bytes=BLOCK), LS_EINVAL, b"aligned"),
    (dict(staging_bytes=2 * BLOCK - 1), LS_ENOMEM, b"staging_bytes"),       # staging short of 2 blocks
    (dict(rate=-1.0), LS_EINVAL, b"max_gbps"),
    (dict(rate=float("nan")), LS_EINVAL, b"max_gbps"),
])
def test_copy_rejects_staging_ring_and_rate(lib, pool, fn, kw, status, word):
    arr = (ctypes.c_int32 * 2)(1, 2)
    assert _copy(lib, fn, pool, 2, ids_host=arr, **kw) == status
    assert word in lib.ls_last_error()


def test_restore_layers_checks_range_and_staging(lib, pool):
    arr = (ctypes.c_int32 * 2)(1, 2)
    L = lib.kv_blocks_restore_layers

    def call(lb, lc, staging_bytes=2 * BLOCK, on_host=0, ring_bytes=0):
        return L(pool, lb, lc, 2, ctypes.c_void_p(F), arr, ctypes.c_void_p(F),
                 ctypes.c_size_t(staging_bytes), on_host, ctypes.c_void_p(F),
                 ctypes.c_size_t(ring_bytes), ctypes.c_double(0.0), None)
    assert call(1, 2) == LS_EINVAL                   # layers [1, 3) of 2
    assert call(-1, 1) == LS_EINVAL
    assert call(1, 1, staging_bytes=2 * BLOCK - 2) == LS_ENOMEM   # all-layer stride even for one layer
    assert call(1, 1, on_host=1, ring_bytes=BLOCK // 2 - 1) == LS_ENOMEM   # ring below one layer slab


@pytest.mark.parametrize("fn", ["kv_blocks_restore", "kv_blocks_stash"])
def test_copy_zero_blocks_is_noop(lib, pool, fn):
    assert _copy(lib, fn, pool, 0, ids=None, staging=None) == LS_OK
    assert _copy(lib, fn, pool, -1, ids=None, staging=None) == LS_EINVAL


# ---- the Python binding checks every tensor's shape before any device access
@pytest.fixture()
def binding():
    try:
        from paper_2606_22983_amd import kv
    except ImportError as e:  # the library is built by the session fixture in other tests
        pytest.skip(str(e))
    return kv


def _fake_pool(kv, nl=1, hkv=4, d=128):
    return kv.KVPool(None, None, nl, 100, hkv, d, 16)


def _bf(*shape):
    import torch
    return torch.zeros(shape, dtype=torch.bfloat16)


def _i32(*shape):
    import torch
    return torch.zeros(shape, dtype=torch.int32)


@pytest.mark.parametrize("bad", ["out", "k_new", "v_new", "tables", "lens", "head_dim", "lens_host"])
def test_binding_decode_shape_checks(built_lib, binding, bad):
    kv = binding
    S, hq, hkv, d = 4, 32, 4, 128
    a = dict(q=_bf(S, hq, d), out=_bf(S, hq, d), k_new=_bf(S, hkv, d), v_new=_bf(S, hkv, d),
             tables=_i32(S, 8), lens=_i32(S), lens_host=[5, 6, 7, 8])
    a[{"out": "out", "k_new": "k_new", "v_new": "v_new", "tables": "tables", "lens": "lens",
       "head_dim": "q", "lens_host": "lens_host"}[bad]] = {
        "out": _bf(S, hq + 1, d), "k_new": _bf(S, hkv, d + 1), "v_new": _bf(S - 1, hkv, d),
        "tables": _i32(S + 1, 8), "lens": _i32(S, 1), "head_dim": _bf(S, hq, 64),
        "lens_host": [5, 6, 7]}[bad]
    if bad == "head_dim":
        a["out"] = _bf(S, hq, 64)
    with pytest.raises(ValueError):
        kv.paged_attn_decode(_fake_pool(kv), 0, a["q"], a["tables"], a["lens"], 0.1, a["out"],
                             _bf(16), a["k_new"], a["v_new"], context_lens_host=a["lens_host"])


@pytest.mark.parametrize("bad", ["cu", "out", "k_new", "tables"])
def test_binding_prefill_shape_checks(built_lib, binding, bad):
    kv = binding
    S, T, hq, hkv, d = 3, 50, 32, 4, 128
    a = dict(q=_bf(T, hq, d), out=_bf(T, hq, d), k_new=_bf(T, hkv, d), cu=_i32(S + 1),
             tables=_i32(S, 8))
    a[bad] = {"cu": _i32(S), "out": _bf(T - 1, hq, d), "k_new": _bf(T, hkv + 1, d),
              "tables": _i32(S - 1, 8)}[bad]
    with pytest.raises(ValueError):
        kv.paged_attn_prefill(_fake_pool(kv), 0, a["q"], a["cu"], _i32(S), 30, a["tables"], 0.1,
                              a["out"], a["k_new"], _bf(T, hkv, d))


def test_binding_copy_checks_staging_size(built_lib, binding):
    kv = binding
    pool = _fake_pool(kv, nl=2)
    with pytest.raises(ValueError, match="staging"):
        kv.kv_blocks_restore(pool, _i32(3), _bf(3 * pool.block_bytes // 2 - 1))
    with pytest.raises(ValueError, match="max_gbps"):
        kv.kv_blocks_stash(pool, _i32(3), _bf(3 * pool.block_bytes // 2), max_gbps=-2.0)


# ---- the decode schedule planned on the host (pure host code: no GPU needed)
def _sched(lib, hkv, hq, lens, maxb, appended=0, host=True):
    import numpy as np
    h = ctypes.c_void_p()
    d = _desc(num_layers=1, num_kv_heads=hkv, num_blocks=1 << 20, kv_bytes=1 << 40)
    assert lib.kv_pool_create(ctypes.byref(d), ctypes.byref(h)) == LS_OK
    arr = np.ascontiguousarray(lens, dtype=np.int32)
    t, hp, m = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
    r = lib.ls_decode_schedule(h, len(arr), hq, maxb, arr.ctypes.data_as(ctypes.c_void_p) if host else None,
                               appended, None, ctypes.byref(t), ctypes.byref(hp), ctypes.byref(m))
    lib.kv_pool_destroy(h)
    return r, t.value, bool(hp.value), bool(m.value)


def test_schedule_talker_batch_is_planned_on_host_without_merge(lib):
    """256 talker sessions (512-4128 keys, 2 KV heads): whole sessions balance the
    GPU, so the host plans one split per session and no merge kernel runs."""
    from paper_2606_22983_amd import workloads as W
    l0 = W.talker_lengths()
    maxb = int(((l0 + 32 + 15) // 16).max())
    for t in (0, 31):
        r, split, host, merge = _sched(lib, 2, 16, l0 + t, maxb, appended=1)
        assert r == LS_OK and host and not merge
        assert split >= int(l0.max()) + t + 1 and split % 1024 == 0


def test_schedule_thinker_batch_splits_long_sessions(lib):
    """The lognormal thinker batch (64 sessions up to 16k keys): 2048-token splits
    (856 items, in the 16-bit item form) with the merge, planned on the host;
    without host lengths the kernel deals 2048-token splits itself."""
    from paper_2606_22983_amd import workloads as W
    lens = W.thinker_lengths()
    maxb = int(((lens + 15) // 16).max())
    assert _sched(lib, 4, 32, lens, maxb) == (LS_OK, 2048, True, True)
    assert _sched(lib, 4, 32, lens, maxb, host=False) == (LS_OK, 2048, False, True)


def test_schedule_mixed_batch_splits_long_sessions(lib):
    """Mostly ~2k-key sessions and ten of 8000 keys: the host splits the long ones
    (a multiple of 1024 below 8000) and the merge runs."""
    import numpy as np
    rng = np.random.default_rng(1)
    lens = np.concatenate([rng.integers(1500, 2040, 200), np.full(10, 8000)])
    r, split, host, merge = _sched(lib, 2, 16, lens, 600)
    assert r == LS_OK and host and merge and split % 1024 == 0 and 2048 <= split < 8000


def test_schedule_eight_heads_uses_wide_items(lib):
    """Eight KV heads (beyond the 16-bit item form): still planned on the host,
    split at 2048 tokens with the merge; the same lengths the GPU test runs."""
    import numpy as np
    rng = np.random.default_rng(225)
    lens = np.concatenate([rng.integers(1, 3000, 20), [6000, 6001, 1, 2048]])
    maxb = int(((lens + 1 + 15) // 16).max())
    assert _sched(lib, 8, 16, lens, maxb, appended=1) == (LS_OK, 2048, True, True)


def test_schedule_rejects_bad_host_lengths(lib):
    assert _sched(lib, 2, 16, [5, 0, 7], 10)[0] == LS_EINVAL          # an empty context
    assert _sched(lib, 2, 16, [5, 0, 7], 10, appended=1)[0] == LS_OK
    assert _sched(lib, 2, 16, [5, 161, 7], 10)[0] == LS_EINVAL        # past a 10-block table


def test_binding_constants_match_the_header(built_lib, binding):
    """The binding's copies of the header's constants (error codes, device error
    bits, the prefill workspace size) agree with the header."""
    kv = binding
    text = open(HEADER).read()

    def define(name):
        m = re.search(r"#define\s+%s\s+\(?\s*(?:\(size_t\))?\s*(0x[0-9a-fA-F]+|-?\d+)u?\s*\)?" % name, text)
        assert m, name
        return int(m.group(1), 0)

    assert kv.PREFILL_WORKSPACE_BYTES == define("LS_PREFILL_WORKSPACE_BYTES")
    assert kv.LS_DEVERR_BLOCK_ID == define("LS_DEVERR_BLOCK_ID")
    assert kv.LS_DEVERR_LENGTH == define("LS_DEVERR_LENGTH")
    assert kv.LS_DEVERR_INTERNAL == define("LS_DEVERR_INTERNAL")


def test_schedule_at_the_batch_limits(lib):
    """2048 sessions and 16384-block tables are accepted; one more of either is
    not.  A 262,144-token session is planned on the host, split into 1024-token
    multiples of at least 2048 tokens, with the merge."""
    assert _sched(lib, 2, 8, [1] * 2048, 16384, host=False)[0] == LS_OK
    assert _sched(lib, 2, 8, [1] * 2049, 8, host=False)[0] == LS_EUNSUPPORTED
    assert _sched(lib, 2, 8, [1] * 4, 16385, host=False)[0] == LS_EUNSUPPORTED
    r, split, host, merge = _sched(lib, 1, 8, [262143, 261444, 9000], 16384, appended=1)
    assert r == LS_OK and host and merge and split % 1024 == 0 and split >= 2048


def test_schedule_large_batches_are_planned_on_host(lib):
    """Batches beyond the small argument block (1280 items) take the large one:
    512 sessions x 4 KV heads (2048 items) and 1000 sessions x 4 (4000) are
    planned on the host; 2048 sessions x 4 KV heads (8192 32-bit items) are
    more than either holds and run the kernel's own schedule."""
    assert _sched(lib, 4, 32, [1536] * 512, 96)[:3] == (LS_OK, 2048, True)
    r, split, host, _ = _sched(lib, 4, 32, [1000 + (7 * s) % 2000 for s in range(1000)], 192)
    assert r == LS_OK and host
    r, split, host, _ = _sched(lib, 4, 32, [1536] * 2048, 96)
    assert r == LS_OK and not host
