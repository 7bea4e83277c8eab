"""The KV manager driving the block copies on the GPU: evict (stash to a pinned
host store), let other data take the freed blocks, preload (restore into the
blocks the manager assigns), and decode over the manager's new block tables
gives bit-for-bit the output of decode before the eviction (§5.1, §5.2)."""
import math

import numpy as np
import pytest
import torch

from paper_2606_22983_amd import workloads as W
from tests.gpu_util import DevicePool, bf16_dev, i32_dev, run_decode

pytestmark = pytest.mark.gpu

NL, HKV, D, HQ = 2, 2, 64, 8
BLOCK_BYTES = NL * 2 * HKV * 16 * D * 2


@pytest.fixture(scope="module")
def kv():
    from paper_2606_22983_amd import kv as kv_mod
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return kv_mod


def _runs(moves: np.ndarray):
    """Group moves into runs of consecutive host slots: (first slot, device ids)."""
    out = []
    for _, _, dev, host in sorted((tuple(int(x) for x in r) for r in moves), key=lambda r: r[3]):
        if out and host == out[-1][0] + len(out[-1][1]):
            out[-1][1].append(dev)
        else:
            out.append((host, [dev]))
    return [(h, np.array(d, np.int32)) for h, d in out]


def _stash(kv, dp, store, moves):
    for h, ids in _runs(moves):
        kv.kv_blocks_stash(dp.pool, i32_dev(ids), store[h:h + len(ids)], block_ids_host=ids,
                           ring=dp.ring)


def _restore(kv, dp, store, moves):
    for h, ids in _runs(moves):
        kv.kv_blocks_restore(dp.pool, i32_dev(ids), store[h:h + len(ids)], block_ids_host=ids,
                             ring=dp.ring)


def _tables(m, sessions, maxb):
    t = np.full((len(sessions), maxb), -1, np.int32)
    for i, s in enumerate(sessions):
        dev, _, state = m.table(s)
        assert (state == 0).all(), "every block must be resident before attention"
        t[i, :len(dev)] = dev
    return t


def _decode_all_layers(kv, dp, q, tables, lens):
    return [run_decode(kv, dp, q, i32_dev(tables), i32_dev(lens), 1 / math.sqrt(D), layer=l)[0].clone()
            for l in range(NL)]


def test_manager_drives_stash_reuse_preload_restore(kv):
    from paper_2606_22983_amd.kv_manager import KVManager
    rng = np.random.default_rng(21)
    nb, slots = 40, 64
    sessions, lens = [0, 1, 2, 3], np.array([100, 70, 40, 90], np.int32)
    m = KVManager(nb, slots, 8, reply_prior_s=1.0)
    for s, L in zip(sessions, lens):
        m.add_session(s)
        m.append_blocks(s, (int(L) + 15) // 16)
    for s, t in zip(sessions, [5.0, 20.0, 1.0, 12.0]):
        m.set_playback(s, t)
    pool = W.normal_bf16(rng, (NL, nb, 2, HKV, 16 * D))
    dp = DevicePool(kv, pool, D, ring_blocks=3)
    store = torch.empty((slots, NL, 2, HKV, 16 * D), dtype=torch.int16, pin_memory=True)
    q = bf16_dev(W.normal_bf16(rng, (len(sessions), HQ, D)))
    maxb = 8
    before = _decode_all_layers(kv, dp, q, _tables(m, sessions, maxb), lens)

    # Evict 10 blocks: all 5 of session 1 (T_next 21), then the last 5... of session 3 (13).
    ev = m.evict(10)
    assert [tuple(r[:2]) for r in ev] == [(1, p) for p in range(4, -1, -1)] + [(3, p) for p in range(5, 0, -1)]
    _stash(kv, dp, store, ev)
    # Other work takes the freed blocks: overwrite them.
    freed = torch.from_numpy(ev[:, 2].astype(np.int64)).cuda()
    dp.data.view(NL, nb, -1)[:, freed] = bf16_dev(W.normal_bf16(rng, (NL, len(ev), 2 * HKV * 16 * D)))

    # Session 3 speaks: preload admitted (5 x 16 KiB at 50 GB/s fits in 1 ms).
    ok, r, e = m.preload(3, 1e-3, BLOCK_BYTES, 50e9)
    assert ok and len(e) == 0 and [int(x) for x in r[:, 1]] == [1, 2, 3, 4, 5]
    _restore(kv, dp, store, r)
    torch.cuda.synchronize()
    m.preload_done(3, 0.0)
    # Session 1: a preload cut short after its first run, cancelled, then the
    # synchronous fallback restores everything.
    ok, r, e = m.preload(1, 1e-3, BLOCK_BYTES, 50e9)
    assert ok and len(r) == 5
    first = _runs(r)[0]
    kv.kv_blocks_restore(dp.pool, i32_dev(first[1][:2]), store[first[0]:first[0] + 2],
                         block_ids_host=first[1][:2], ring=dp.ring)
    torch.cuda.synchronize()
    m.preload_cancel(1)
    r, e = m.load_sync(1)
    _stash(kv, dp, store, e)
    _restore(kv, dp, store, r)
    torch.cuda.synchronize()
    m.preload_done(1, 0.0)

    after = _decode_all_layers(kv, dp, q, _tables(m, sessions, maxb), lens)
    for l in range(NL):
        assert torch.equal(before[l].view(torch.int16), after[l].view(torch.int16)), "layer %d" % l
    assert kv.ls_device_errors() == 0


def test_preload_evicting_for_room_keeps_every_session_exact(kv):
    """A full pool: the preload itself must evict later-use KV; both the evicted
    and the preloaded sessions decode exactly as before once resident again."""
    from paper_2606_22983_amd.kv_manager import KVManager
    rng = np.random.default_rng(22)
    nb, slots = 12, 32
    sessions, lens = [0, 1, 2], np.array([64, 64, 64], np.int32)       # 4 blocks each
    m = KVManager(nb, slots, 4, reply_prior_s=0.0)
    for s, t in zip(sessions, [3.0, 9.0, 6.0]):
        m.add_session(s)
        m.append_blocks(s, 4)
        m.set_playback(s, t)
    pool = W.normal_bf16(rng, (NL, nb, 2, HKV, 16 * D))
    dp = DevicePool(kv, pool, D, ring_blocks=2)
    store = torch.empty((slots, NL, 2, HKV, 16 * D), dtype=torch.int16, pin_memory=True)
    q = bf16_dev(W.normal_bf16(rng, (3, HQ, D)))
    before = _decode_all_layers(kv, dp, q, _tables(m, sessions, 4), lens)
    ev = m.evict(4)                                  # session 1 out
    _stash(kv, dp, store, ev)
    m.add_session(3)
    taken = m.append_blocks(3, 4)                    # a new session fills the pool
    dp.data.view(NL, nb, -1)[:, torch.from_numpy(taken.astype(np.int64)).cuda()] = 0
    ok, r, e = m.preload(1, 1.0, BLOCK_BYTES, 1e9)
    assert ok and [int(x) for x in e[:, 0]] == [2, 2, 2, 2]          # session 2 (T_next 6) makes room
    _stash(kv, dp, store, e)
    _restore(kv, dp, store, r)
    torch.cuda.synchronize()
    m.preload_done(1, 0.0)
    # Session 2's turn: session 0 (T_next 3) makes room before session 3 (T_next 0).
    r2, e2 = m.load_sync(2)
    assert [int(x) for x in e2[:, 0]] == [0, 0, 0, 0]
    _stash(kv, dp, store, e2)
    _restore(kv, dp, store, r2)
    # Then session 0 comes back: session 3 is the only candidate left.
    r3, e3 = m.load_sync(0)
    assert [int(x) for x in e3[:, 0]] == [3, 3, 3, 3]
    _stash(kv, dp, store, e3)
    _restore(kv, dp, store, r3)
    torch.cuda.synchronize()
    m.preload_done(2, 0.0)
    m.preload_done(0, 0.0)
    after = _decode_all_layers(kv, dp, q, _tables(m, sessions, 4), lens)
    for l in range(NL):
        assert torch.equal(before[l].view(torch.int16), after[l].view(torch.int16)), "layer %d" % l
    assert kv.ls_device_errors() == 0
