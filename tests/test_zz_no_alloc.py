"""paged_attn_decode_static (the entry point that allocates nothing: its split
partials live in a static device buffer of the library) gives bit for bit the
outputs of paged_attn_decode with a caller workspace, on two calls in a row,
the second smaller; and refuses a shape whose partials exceed the buffer."""
import math

import numpy as np
import pytest
import torch

from paper_2606_22983_amd import workloads as W
from tests.gpu_util import DevicePool, assert_attn_close, bf16_dev, i32_dev, log

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def kv():
    from paper_2606_22983_amd import kv as kv_mod
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return kv_mod


def _case(rng, lens, hq, hkv, d, append):
    lens = np.asarray(lens, np.int64)
    need = np.maximum((lens + (1 if append else 0) + 15) // 16, 1)
    nb = int(need.sum()) + 4
    perm = rng.permutation(nb).astype(np.int32)
    tables = np.full((len(lens), int(need.max())), -1, np.int32)
    pos = 0
    for s, k in enumerate(need):
        tables[s, :k] = perm[pos:pos + k]
        pos += k
    pool = W.normal_bf16(rng, (1, nb, 2, hkv, 16 * d))
    W._poison(pool, d, tables, lens, int(need.sum()))
    q = W.normal_bf16(rng, (len(lens), hq, d))
    kn = W.normal_bf16(rng, (len(lens), hkv, d)) if append else None
    vn = W.normal_bf16(rng, (len(lens), hkv, d)) if append else None
    return pool, tables, q, kn, vn


def _both(kv, pool, tables, q, kn, vn, lens, d):
    """(static-scratch output, workspace output) of the same call on separate pool copies."""
    outs = []
    for static in (True, False):
        dp = DevicePool(kv, pool, d)
        out = torch.empty(q.shape, dtype=torch.bfloat16, device="cuda")
        args = (dp.pool, 0, bf16_dev(q), i32_dev(tables), i32_dev(lens), 1 / math.sqrt(d), out)
        new = (None if kn is None else bf16_dev(kn), None if vn is None else bf16_dev(vn))
        if static:
            kv.paged_attn_decode_static(*args, *new)
        else:
            ws = torch.zeros(kv.decode_workspace_bytes(dp.pool, q.shape[0], q.shape[1], tables.shape[1]),
                             dtype=torch.uint8, device="cuda")
            kv.paged_attn_decode(*args, ws, *new)
        torch.cuda.synchronize()
        outs.append((out, dp.host()))
    return outs


def test_static_scratch_decode_matches_workspace_decode(kv, oracle_lib):
    rng = np.random.default_rng(777)
    # first call: 48 thinker-shaped sessions, up to 9 splits each
    lens1 = rng.integers(300, 9000, size=48)
    pool, tables, q, kn, vn = _case(rng, lens1, 32, 4, 128, append=False)
    (a, _), (b, _) = _both(kv, pool, tables, q, kn, vn, lens1, 128)
    log("static scratch decode, call 1: %d sessions, %d tokens" % (len(lens1), int(lens1.sum())))
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    ref = oracle_lib.decode(pool, 16, 128, 0, q, tables, lens1, 1 / math.sqrt(128))
    assert_attn_close(a, ref, "static scratch decode, call 1")
    # second call, right after, smaller: 7 sessions with append, other geometry
    lens2 = np.array([0, 5, 1023, 1024, 2100, 64, 3])
    pool2, tables2, q2, kn2, vn2 = _case(rng, lens2, 8, 2, 64, append=True)
    (a2, pa), (b2, pb) = _both(kv, pool2, tables2, q2, kn2, vn2, lens2, 64)
    assert torch.equal(a2.view(torch.int16), b2.view(torch.int16))
    assert np.array_equal(pa, pb)
    ref2 = oracle_lib.decode(pool2, 16, 64, 0, q2, tables2, lens2, 1 / math.sqrt(64), k_new=kn2, v_new=vn2)
    assert_attn_close(a2, ref2, "static scratch decode, call 2")
    assert kv.ls_device_errors() == 0


def test_static_scratch_refuses_oversized_batch(kv):
    rng = np.random.default_rng(5)
    pool = W.normal_bf16(rng, (1, 64, 2, 4, 16 * 128))
    dp = DevicePool(kv, pool, 128)
    S, maxb = 2048, 1024                       # partials of 2048 sessions x 16k tokens: far above 32 MiB
    assert kv.decode_workspace_bytes(dp.pool, S, 32, maxb) > (32 << 20)
    q = torch.zeros((S, 32, 128), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(kv.LiveServeError, match="static"):
        kv.paged_attn_decode_static(dp.pool, 0, q, torch.zeros((S, maxb), dtype=torch.int32, device="cuda"),
                                    torch.ones(S, dtype=torch.int32, device="cuda"), 0.088, q.clone())
