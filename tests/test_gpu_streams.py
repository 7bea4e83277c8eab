"""Kernels on CU-masked streams: the persistent grids are sized to the CUs the
stream may use, and the results do not depend on it."""
import numpy as np
import pytest
import torch

from paper_2606_22983_amd import workloads as W
from tests.gpu_util import (DevicePool, bf16_dev, cu_masked_stream, destroy_stream, host_bits,
                            i32_dev, log)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def kv():
    from paper_2606_22983_amd import kv as kv_mod
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return kv_mod


def _decode(kv, dp, case, q, tables, lens, stream, ws=None):
    s, hq, d = q.shape
    out = torch.empty((s, hq, d), dtype=torch.bfloat16, device="cuda")
    if ws is None:
        ws = torch.zeros(kv.decode_workspace_bytes(dp.pool, s, hq, tables.shape[1]),
                         dtype=torch.uint8, device="cuda")
    kv.paged_attn_decode(dp.pool, 0, q, tables, lens, case.scale, out, ws, stream=stream)
    return out, ws


@pytest.mark.parametrize("lo,hi", [(0, 24), (40, 256)])
def test_decode_on_cu_masked_stream_is_bit_identical(kv, lo, hi):
    n_cus = torch.cuda.get_device_properties(0).multi_processor_count
    hi = min(hi, n_cus)
    made = cu_masked_stream(lo, hi)
    if made is None:
        pytest.skip("runtime has no hipExtStreamCreateWithCUMask")
    stream, handle = made
    try:
        case = W.thinker_decode(num_sessions=24)
        dp = DevicePool(kv, case.pool.data, 128)
        q, tables, lens = bf16_dev(case.q[0]), i32_dev(case.block_tables), i32_dev(case.context_lens)
        full, ws = _decode(kv, dp, case, q, tables, lens, torch.cuda.current_stream())
        torch.cuda.synchronize()
        for _ in range(2):      # the workspace's counters are reused across grids
            part, _ = _decode(kv, dp, case, q, tables, lens, stream, ws)
            stream.synchronize()
            assert torch.equal(full.view(torch.int16), part.view(torch.int16))
        assert kv.ls_device_errors() == 0
        log("decode on CUs %d..%d bit-identical to the full-device run" % (lo, hi - 1))
    finally:
        torch.cuda.synchronize()
        destroy_stream(handle)


def test_restore_on_cu_masked_stream_is_bit_exact(kv):
    made = cu_masked_stream(0, 8)
    if made is None:
        pytest.skip("runtime has no hipExtStreamCreateWithCUMask")
    stream, handle = made
    try:
        rng = np.random.default_rng(11)
        nl, nb, hkv, d = 3, 96, 2, 64
        pool = W.normal_bf16(rng, (nl, nb, 2, hkv, 16 * d))
        dp = DevicePool(kv, pool, d)
        ids = rng.permutation(nb)[:40].astype(np.int32)
        staging = bf16_dev(W.normal_bf16(rng, (40, nl, 2, hkv, 16 * d)))
        kv.kv_blocks_restore(dp.pool, i32_dev(ids), staging, stream=stream)
        stream.synchronize()
        got = dp.host()
        st = host_bits(staging)
        assert np.array_equal(got[:, ids], st.transpose(1, 0, 2, 3, 4))
        others = np.setdiff1d(np.arange(nb), ids)
        assert np.array_equal(got[:, others], pool[:, others])
        back = torch.empty_like(staging)
        kv.kv_blocks_stash(dp.pool, i32_dev(ids), back, stream=stream)
        stream.synchronize()
        assert torch.equal(back.view(torch.int16), staging.view(torch.int16))
        assert kv.ls_device_errors() == 0
    finally:
        torch.cuda.synchronize()
        destroy_stream(handle)
