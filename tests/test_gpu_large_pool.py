"""Decode and prefill over a layer larger than 4 GiB.

With 4 KV heads at head_dim 128 a block's slab is 32 KiB, so block ids past
131,072 put its tiles more than 2^32 bytes past the layer's base.  The device
pool (140,000 blocks, 4.6 GB) is filled on the device; the oracle gets only the
blocks a case uses, relabelled 0 .. m-1, since attention does not depend on
which ids hold the keys.  Appended rows are compared in the same relabelled
form."""
import math

import numpy as np
import pytest
import torch

from paper_2606_22983_amd import workloads as W
from tests.gpu_util import assert_attn_close, bf16_dev, host_bits, i32_dev

pytestmark = pytest.mark.gpu

HKV, D, NB = 4, 128, 140000
HIGH = NB - 9000                      # ids drawn from [131000, 140000): both sides of 2^32 bytes


@pytest.fixture(scope="module")
def kv():
    from paper_2606_22983_amd import kv as kv_mod
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return kv_mod


@pytest.fixture(scope="module")
def big(kv):
    gen = torch.Generator(device="cuda")
    gen.manual_seed(4242)
    data = torch.empty((1, NB, 2, HKV, 16 * D), dtype=torch.bfloat16, device="cuda")
    data.normal_(generator=gen)
    pool = kv.kv_pool_create(data, 1, NB, HKV, D, 16)
    yield data, pool
    del pool, data
    torch.cuda.empty_cache()


def _ids(rng, k):
    """k distinct block ids in [HIGH, NB), 131071 and 131072 (the slabs on either
    side of 2^32 bytes) among them, in random order."""
    rest = np.setdiff1d(np.arange(HIGH, NB), [131071, 131072])
    ids = np.concatenate([[131071, 131072], rng.choice(rest, size=k - 2, replace=False)])
    return rng.permutation(ids).astype(np.int32)


def _tables(ids, need):
    tables = np.full((len(need), int(max(need))), -1, np.int32)
    pos = 0
    for s, k in enumerate(need):
        tables[s, :k] = ids[pos:pos + k]
        pos += k
    return tables


def _compact(data, tables):
    """Host copy of the used blocks and the tables relabelled onto it."""
    used = np.unique(tables[tables >= 0]).astype(np.int64)
    lut = np.full(NB, -1, np.int32)
    lut[used] = np.arange(len(used), dtype=np.int32)
    relabelled = np.where(tables >= 0, lut[np.clip(tables, 0, NB - 1)], -1).astype(np.int32)
    idx = torch.from_numpy(used).cuda()
    torch.cuda.synchronize()
    return host_bits(data.index_select(1, idx)), relabelled, idx


def test_decode_with_block_ids_past_4gib(kv, oracle_lib, big):
    data, pool = big
    rng = np.random.default_rng(131072)
    S, hq = 8, 32
    lens = rng.integers(1500, 2500, size=S)
    need = (lens + 1 + 15) // 16
    ids = _ids(rng, int(need.sum()))
    tables = _tables(ids, need)
    host_pool, relabelled, idx = _compact(data, tables)
    q = W.normal_bf16(rng, (S, hq, D))
    kn = W.normal_bf16(rng, (S, HKV, D))
    vn = W.normal_bf16(rng, (S, HKV, D))
    scale = 1 / math.sqrt(D)
    ref, ref_pool = oracle_lib.decode(host_pool, 16, D, 0, q, relabelled, lens, scale, k_new=kn, v_new=vn,
                                      pool_out=True)
    ws = torch.zeros(kv.decode_workspace_bytes(pool, S, hq, tables.shape[1]), dtype=torch.uint8, device="cuda")
    for host in (False, True):
        out = torch.empty((S, hq, D), dtype=torch.bfloat16, device="cuda")
        kv.paged_attn_decode(pool, 0, bf16_dev(q), i32_dev(tables), i32_dev(lens), scale, out, ws,
                             bf16_dev(kn), bf16_dev(vn), context_lens_host=lens if host else None)
        assert_attn_close(out, ref, "decode, block ids past 4 GiB, host lengths %s" % host)
        torch.cuda.synchronize()
        assert np.array_equal(host_bits(data.index_select(1, idx)), ref_pool), "appended rows differ"
    assert kv.ls_device_errors() == 0


def test_prefill_with_block_ids_past_4gib(kv, oracle_lib, big):
    data, pool = big
    rng = np.random.default_rng(262144)
    hq = 8
    n = np.array([100, 37, 256])
    c = np.array([1500, 16, 700])
    need = (c + n + 15) // 16
    ids = _ids(rng, int(need.sum()))
    tables = _tables(ids, need)
    host_pool, relabelled, idx = _compact(data, tables)
    total = int(n.sum())
    q = W.normal_bf16(rng, (total, hq, D))
    kn = W.normal_bf16(rng, (total, HKV, D))
    vn = W.normal_bf16(rng, (total, HKV, D))
    cu = np.concatenate([[0], np.cumsum(n)]).astype(np.int32)
    scale = 1 / math.sqrt(D)
    ref, ref_pool = oracle_lib.prefill(host_pool, 16, D, 0, q, kn, vn, cu, c, relabelled, scale, pool_out=True)
    for mode in ("device-lengths", "host-lengths-counters"):
        host = mode != "device-lengths"
        ws = torch.zeros((kv.PREFILL_WORKSPACE_BYTES,), dtype=torch.uint8, device="cuda") if host else None
        out = torch.empty((total, hq, D), dtype=torch.bfloat16, device="cuda")
        kv.paged_attn_prefill(pool, 0, bf16_dev(q), i32_dev(cu), i32_dev(c), int(n.max()), i32_dev(tables),
                              scale, out, bf16_dev(kn), bf16_dev(vn),
                              lens_host=np.stack([n, c], 1) if host else None, workspace=ws)
        assert_attn_close(out, ref, "prefill, block ids past 4 GiB, %s" % mode)
        torch.cuda.synchronize()
        assert np.array_equal(host_bits(data.index_select(1, idx)), ref_pool), "appended rows differ"
    assert kv.ls_device_errors() == 0
