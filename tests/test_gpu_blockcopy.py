"""GPU parity of kv_blocks_stash / kv_blocks_restore: bit-exact against the
oracle's byte copies, device and pinned-host staging, cancelled-preload
fallback, canaries, bad ids, and decode undisturbed by a concurrent restore."""
import math

import numpy as np
import pytest
import torch

from paper_2606_22983_amd import workloads as W
from tests.gpu_util import DevicePool, bf16_dev, host_bits, i32_dev, log, run_decode

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def kv():
    from paper_2606_22983_amd import kv as kv_mod
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return kv_mod


def _random_pool(rng, nl, nb, hkv, d):
    return rng.integers(0, 1 << 16, size=(nl, nb, 2, hkv, 16 * d), dtype=np.uint16)


def test_tiny_restore_8_blocks(kv, oracle_lib):
    """8 blocks restored from a contiguous device staging buffer into a 256-block pool."""
    case = W.tiny_decode()
    pool = case.pool.data
    rng = np.random.default_rng(26061)
    ids = rng.permutation(pool.shape[1])[:8].astype(np.int32)
    staging = _random_pool(rng, 8, 1, 2, 64).reshape(8, 1, 2, 2, 16 * 64)
    dp = DevicePool(kv, pool, 64)
    kv.kv_blocks_restore(dp.pool, i32_dev(ids), bf16_dev(staging), block_ids_host=ids)
    ref = oracle_lib.restore(pool.copy(), 16, 64, ids, staging)
    assert np.array_equal(dp.host(), ref)
    st = torch.empty((8, 1, 2, 2, 16 * 64), dtype=torch.bfloat16, device="cuda")
    kv.kv_blocks_stash(dp.pool, i32_dev(ids), st, block_ids_host=ids)
    assert np.array_equal(host_bits(st), staging)
    assert kv.ls_device_errors() == 0


@pytest.mark.parametrize("nl,hkv,d,nb,n", [(48, 4, 128, 160, 96), (3, 2, 64, 64, 64),
                                           (1, 4, 128, 40, 1)])
def test_stash_then_restore_into_permutation(kv, oracle_lib, nl, hkv, d, nb, n):
    """Stash slot set A, poison the pool, restore into slots B: pool[B[i]] == old pool[A[i]],
    every other block untouched."""
    rng = np.random.default_rng(nl * 100 + nb)
    pool = _random_pool(rng, nl, nb, hkv, d)
    a = rng.permutation(nb)[:n].astype(np.int32)
    b = rng.permutation(nb)[:n].astype(np.int32)
    dp = DevicePool(kv, pool, d)
    st = torch.empty((n, nl, 2, hkv, 16 * d), dtype=torch.bfloat16, device="cuda")
    kv.kv_blocks_stash(dp.pool, i32_dev(a), st, block_ids_host=a)
    st_host = host_bits(st)
    assert np.array_equal(st_host, oracle_lib.stash(pool, 16, d, a))
    dp.data.view(torch.int16).fill_(0x7FC0)                 # poison the pool
    kv.kv_blocks_restore(dp.pool, i32_dev(b), st, block_ids_host=b)
    expect = np.full_like(pool, 0x7FC0)
    oracle_lib.restore(expect, 16, d, b, st_host)
    assert np.array_equal(dp.host(), expect)
    assert kv.ls_device_errors() == 0


def test_pinned_host_staging_through_ring(kv, oracle_lib):
    """Host-pinned staging goes through a 3-block device ring in several chunks."""
    rng = np.random.default_rng(5)
    nl, hkv, d, nb, n = 4, 4, 128, 50, 11
    pool = _random_pool(rng, nl, nb, hkv, d)
    ids = rng.permutation(nb)[:n].astype(np.int32)
    dp = DevicePool(kv, pool, d, ring_blocks=3)
    host = torch.empty((n, nl, 2, hkv, 16 * d), dtype=torch.int16, pin_memory=True)
    kv.kv_blocks_stash(dp.pool, i32_dev(ids), host, block_ids_host=ids, ring=dp.ring)
    torch.cuda.synchronize()
    assert np.array_equal(host.numpy().view(np.uint16), oracle_lib.stash(pool, 16, d, ids))
    fresh = _random_pool(rng, n, nl, hkv, d).reshape(n, nl, 2, hkv, 16 * d)
    host.copy_(torch.from_numpy(fresh.view(np.int16)))
    ids2 = rng.permutation(nb)[:n].astype(np.int32)
    kv.kv_blocks_restore(dp.pool, i32_dev(ids2), host, block_ids_host=ids2, ring=dp.ring)
    torch.cuda.synchronize()
    assert np.array_equal(dp.host(), oracle_lib.restore(pool.copy(), 16, d, ids2, fresh))


def test_cancelled_preload_then_synchronous_fallback(kv):
    """Restore k of n blocks, stop, restore the rest: same pool as one full restore."""
    rng = np.random.default_rng(6)
    nl, hkv, d, nb, n = 8, 4, 128, 64, 30
    pool = _random_pool(rng, nl, nb, hkv, d)
    ids = rng.permutation(nb)[:n].astype(np.int32)
    staging = bf16_dev(_random_pool(rng, n, nl, hkv, d).reshape(n, nl, 2, hkv, 16 * d))
    full = DevicePool(kv, pool, d)
    kv.kv_blocks_restore(full.pool, i32_dev(ids), staging)
    part = DevicePool(kv, pool, d)
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):
        kv.kv_blocks_restore(part.pool, i32_dev(ids[:11]), staging[:11])
    side.synchronize()
    kv.kv_blocks_restore(part.pool, i32_dev(ids[11:]), staging[11:])
    assert np.array_equal(full.host(), part.host())


def test_device_ids_out_of_range_are_skipped_and_flagged(kv):
    rng = np.random.default_rng(7)
    pool = _random_pool(rng, 2, 20, 2, 64)
    dp = DevicePool(kv, pool, 64)
    kv.ls_device_errors()
    ids = np.array([3, 25, 5], np.int32)          # 25 is outside the pool; no host copy given
    staging = bf16_dev(_random_pool(rng, 3, 2, 2, 64).reshape(3, 2, 2, 2, 16 * 64))
    kv.kv_blocks_restore(dp.pool, i32_dev(ids), staging)
    assert kv.ls_device_errors() & kv.LS_DEVERR_BLOCK_ID
    got = dp.host()
    st = host_bits(staging)
    assert np.array_equal(got[:, 3], st[0]) and np.array_equal(got[:, 5], st[2])
    others = np.setdiff1d(np.arange(20), [3, 5])
    assert np.array_equal(got[:, others], pool[:, others])


def test_decode_unchanged_by_concurrent_restore(kv):
    """Thinker-shaped decode on the main stream, a restore into disjoint blocks on a
    side stream at the same time: decode output bit-identical to the solo run."""
    case = W.thinker_decode(num_sessions=16)
    pool = case.pool.data
    used = np.unique(case.block_tables[case.block_tables >= 0])
    free = np.setdiff1d(np.arange(pool.shape[1]), used).astype(np.int32)
    dp = DevicePool(kv, pool, 128)
    q = bf16_dev(case.q[0])
    tables = i32_dev(case.block_tables)
    lens = i32_dev(case.context_lens)
    solo, ws = run_decode(kv, dp, q, tables, lens, case.scale)
    torch.cuda.synchronize()
    rng = np.random.default_rng(8)
    n = len(free)
    staging = bf16_dev(_random_pool(rng, n, 1, 4, 128).reshape(n, 1, 2, 4, 16 * 128))
    side = torch.cuda.Stream()
    ids = i32_dev(free)
    torch.cuda.synchronize()
    outs = []
    with torch.cuda.stream(side):
        for _ in range(3):
            kv.kv_blocks_restore(dp.pool, ids, staging)
    for _ in range(3):
        o, _ = run_decode(kv, dp, q, tables, lens, case.scale, workspace=ws)
        outs.append(o)
    torch.cuda.synchronize()
    for o in outs:
        assert torch.equal(o.view(torch.int16), solo.view(torch.int16))
    got = dp.host()
    assert np.array_equal(got[:, free], host_bits(staging).transpose(1, 0, 2, 3, 4))
    log("decode bit-identical under a concurrent restore of %d blocks" % n)


@pytest.mark.parametrize("on_host", [False, True])
def test_restore_by_layer_ranges_equals_full_restore(kv, oracle_lib, on_host):
    """Layer ranges [0,1), [1,4), [4,5) restored one by one (device staging, or
    pinned host staging through a ring narrower than a whole block) give the
    oracle's full restore, byte for byte."""
    rng = np.random.default_rng(31 + on_host)
    nl, hkv, d, nb, n = 5, 2, 64, 40, 13
    pool = _random_pool(rng, nl, nb, hkv, d)
    ids = rng.permutation(nb)[:n].astype(np.int32)
    staging = _random_pool(rng, n, nl, hkv, d).reshape(n, nl, 2, hkv, 16 * d)
    expect = oracle_lib.restore(pool.copy(), 16, d, ids, staging)
    layer_bytes = 2 * hkv * 16 * d * 2
    dp = DevicePool(kv, pool, d, ring_blocks=0)
    ring = None
    if on_host:
        ring = torch.empty(5 * layer_bytes, dtype=torch.uint8, device="cuda")   # 5 layer slabs
        st = torch.from_numpy(staging.view(np.int16)).pin_memory()
    else:
        st = bf16_dev(staging)
    for lb, lc in ((0, 1), (1, 3), (4, 1)):
        kv.kv_blocks_restore_layers(dp.pool, lb, lc, i32_dev(ids), st, block_ids_host=ids, ring=ring)
    torch.cuda.synchronize()
    assert np.array_equal(dp.host(), expect)
    with pytest.raises(kv.LiveServeError):
        kv.kv_blocks_restore_layers(dp.pool, 4, 2, i32_dev(ids), st, ring=ring)
    assert kv.ls_device_errors() == 0


def test_host_staged_stash_and_restore_on_two_streams(kv, oracle_lib):
    """An eviction stash to pinned host memory on one stream and a preload restore
    from pinned host memory on another, at the same time, on disjoint blocks, each
    through its own ring (a ring narrower than either copy, so both cycle it):
    both bit-exact against the oracle."""
    rng = np.random.default_rng(51)
    nl, hkv, d, nb, n = 6, 4, 128, 120, 40
    pool = _random_pool(rng, nl, nb, hkv, d)
    perm = rng.permutation(nb).astype(np.int32)
    out_ids, in_ids = perm[:n], perm[n:2 * n]
    incoming = _random_pool(rng, n, nl, hkv, d).reshape(n, nl, 2, hkv, 16 * d)
    dp = DevicePool(kv, pool, d)
    per_block = nl * 2 * hkv * 16 * d * 2
    rings = [torch.empty(3 * per_block, dtype=torch.uint8, device="cuda") for _ in range(2)]
    evicted = torch.empty((n, nl, 2, hkv, 16 * d), dtype=torch.int16, pin_memory=True)
    preload = torch.from_numpy(incoming.view(np.int16)).pin_memory()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    torch.cuda.synchronize()
    for rep in range(3):
        with torch.cuda.stream(streams[0]):
            kv.kv_blocks_stash(dp.pool, i32_dev(out_ids), evicted, block_ids_host=out_ids, ring=rings[0])
        with torch.cuda.stream(streams[1]):
            kv.kv_blocks_restore(dp.pool, i32_dev(in_ids), preload, block_ids_host=in_ids, ring=rings[1])
        torch.cuda.synchronize()
        assert np.array_equal(evicted.numpy().view(np.uint16), oracle_lib.stash(pool, 16, d, out_ids)), rep
        assert np.array_equal(dp.host(), oracle_lib.restore(pool.copy(), 16, d, in_ids, incoming)), rep
    assert kv.ls_device_errors() == 0


@pytest.mark.parametrize("gbps", [0.5, 40.0, 1e6])
def test_rate_bounded_copies_are_bit_exact(kv, oracle_lib, gbps):
    """A rate-bounded copy (full-rate bursts at clock-window boundaries) moves the
    same bytes; at 0.5 GB/s the 11 MB stash takes at least ~20 ms, at 40 GB/s at
    least ~0.3 ms."""
    rng = np.random.default_rng(60 + int(gbps) % 97)
    nl, hkv, d, nb, n = 5, 4, 128, 90, 70
    pool = _random_pool(rng, nl, nb, hkv, d)
    ids = rng.permutation(nb)[:n].astype(np.int32)
    dp = DevicePool(kv, pool, d, ring_blocks=4)
    st = torch.empty((n, nl, 2, hkv, 16 * d), dtype=torch.int16, device="cuda")
    torch.cuda.synchronize()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record()
    kv.kv_blocks_stash(dp.pool, i32_dev(ids), st, max_gbps=gbps)
    t1.record()
    assert np.array_equal(host_bits(st), oracle_lib.stash(pool, 16, d, ids))
    ms = t0.elapsed_time(t1)
    payload = n * nl * 2 * hkv * 16 * d * 2
    log("stash of %.1f MB at a %.1f GB/s cap: %.3f ms (%.1f GB/s)" % (payload / 1e6, gbps, ms,
                                                                       payload / ms / 1e6))
    if gbps < 100:
        assert payload / (ms * 1e-3) <= 1.15 * gbps * 1e9, "the copy ran faster than its cap"
    fresh = _random_pool(rng, n, nl, hkv, d).reshape(n, nl, 2, hkv, 16 * d)
    host = torch.from_numpy(fresh.view(np.int16)).pin_memory()
    ids2 = rng.permutation(nb)[:n].astype(np.int32)
    kv.kv_blocks_restore(dp.pool, i32_dev(ids2), host, block_ids_host=ids2, ring=dp.ring, max_gbps=gbps)
    assert np.array_equal(dp.host(), oracle_lib.restore(pool.copy(), 16, d, ids2, fresh))
    assert kv.ls_device_errors() == 0


def test_restore_at_preload_geometry_10k_blocks(kv, oracle_lib):
    """The preload workload's geometry (48 layers x 4 KV heads x D = 128, 1.5 MiB
    per block) at 10,000 blocks (15 GiB; byte offsets far past 2^32): stash a
    random slot set, poison the pool, restore into a fresh permutation, bit-exact
    against the oracle's byte copies.  Contents come from a seeded device generator
    and are copied to the host for the oracle."""
    nl, hkv, d, n, nb = 48, 4, 128, 10000, 10240
    elems = nl * nb * 2 * hkv * 16 * d
    gen = torch.Generator(device="cuda")
    gen.manual_seed(26065)
    data = torch.empty(elems, dtype=torch.int16, device="cuda")
    data.random_(-32768, 32767, generator=gen)
    pool = data.cpu().numpy().view(np.uint16).reshape(nl, nb, 2, hkv, 16 * d)
    rng = np.random.default_rng(26065)
    a = rng.permutation(nb)[:n].astype(np.int32)
    b = rng.permutation(nb)[:n].astype(np.int32)
    log("restore at the preload geometry: %d of %d blocks, %.1f GiB" % (n, nb, n * nl * 32768 / 2 ** 30))
    p = kv.kv_pool_create(data, nl, nb, hkv, d, 16)
    st = torch.empty((n, nl, 2, hkv, 16 * d), dtype=torch.int16, device="cuda")
    kv.kv_blocks_stash(p, i32_dev(a), st, block_ids_host=a)
    st_host = st.cpu().numpy().view(np.uint16)
    assert np.array_equal(st_host, oracle_lib.stash(pool, 16, d, a))
    data.fill_(0x7FC0)                                   # poison every block
    kv.kv_blocks_restore(p, i32_dev(b), st, block_ids_host=b)
    del st
    torch.cuda.synchronize()
    expect = np.full_like(pool, 0x7FC0)
    del pool
    oracle_lib.restore(expect, 16, d, b, st_host)
    del st_host
    got = data.cpu().numpy().view(np.uint16).reshape(expect.shape)
    assert np.array_equal(got, expect)
    assert kv.ls_device_errors() == 0

