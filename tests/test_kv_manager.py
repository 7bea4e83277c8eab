"""KV manager (host policy of LiveServe §5.1, §5.2, §6): pins derived by hand
from the paper's rules, checked on both the brute-force oracle and the
library's C++ manager, and randomized parity between the two."""
import math

import numpy as np
import pytest

from oracle.kv_manager import RefKVManager


def _lib_manager(*args, **kw):
    from paper_2606_22983_amd.kv_manager import KVManager
    return KVManager(*args, **kw)


IMPLS = {"oracle": RefKVManager, "library": _lib_manager}


def _moves(m):
    return [tuple(int(x) for x in row) for row in m]


@pytest.fixture(params=sorted(IMPLS))
def make(request):
    return IMPLS[request.param]


def _four_sessions(make, **kw):
    """A, B, C idle with 4 blocks each (device blocks 0-3, 4-7, 8-11), D running
    with blocks 12-15.  T_next: A = 2 + 3 (prior) = 5, B = 10 + 3 = 13,
    C = 0 + 1 (one observed reply of 1 s) = 1, D pinned."""
    m = make(32, 32, 8, reply_prior_s=3.0, reply_ema_alpha=0.5, seconds_per_token=0.04, **kw)
    for s in range(4):
        m.add_session(s)
        assert list(m.append_blocks(s, 4)) == list(range(4 * s, 4 * s + 4))
    m.set_playback(0, 2.0)
    m.set_playback(1, 10.0)
    m.set_playback(2, 0.0)
    m.observe_reply(2, 1.0)
    m.set_running(3, True)
    return m


def test_next_use_estimate(make):
    m = _four_sessions(make)
    assert [m.session_info(s)[0] for s in range(3)] == [5.0, 13.0, 1.0]
    m.set_playback(0, -1.0, 100)            # horizon unknown: 100 tokens x 0.04 s
    assert math.isclose(m.session_info(0)[0], 100 * 0.04 + 3.0)
    m.observe_reply(2, 4.0)                 # moving average: 0.5 * 4 + 0.5 * 1
    m.observe_reply(2, 2.0)                 # 0.5 * 2 + 0.5 * 2.5
    assert m.session_info(2)[0] == 2.25


def test_eviction_order_farthest_next_use_first_suffix_first(make):
    m = _four_sessions(make)
    # B (T_next 13) gives all 4 blocks, last position first; then A (5) its last two.
    assert _moves(m.evict(6)) == [(1, 3, 7, 0), (1, 2, 6, 1), (1, 1, 5, 2), (1, 0, 4, 3),
                                  (0, 3, 3, 4), (0, 2, 2, 5)]
    dev, host, state = m.table(0)
    assert list(dev) == [0, 1, -1, -1] and list(host) == [-1, -1, 5, 4] and list(state) == [0, 0, 1, 1]
    assert m.counts()["free_device_blocks"] == 16 + 6
    # A's remaining prefix goes next, then C; the running session D never.
    assert _moves(m.evict(3)) == [(0, 1, 1, 6), (0, 0, 0, 7), (2, 3, 11, 8)]
    assert _moves(m.evict(100)) == [(2, 2, 10, 9), (2, 1, 9, 10), (2, 0, 8, 11)]
    assert m.counts()["evictable_blocks"] == 0


def test_speech_start_protects_and_ties_break_by_id(make):
    m = _four_sessions(make)
    m.speech_start(1)
    assert m.session_info(1)[1] & 0x2
    assert _moves(m.evict(6)) == [(0, 3, 3, 0), (0, 2, 2, 1), (0, 1, 1, 2), (0, 0, 0, 3),
                                  (2, 3, 11, 4), (2, 2, 10, 5)]
    m2 = make(8, 8, 4, reply_prior_s=1.0)
    for s in (2, 1):
        m2.add_session(s)
        m2.append_blocks(s, 2)
    assert _moves(m2.evict(3)) == [(1, 1, 3, 0), (1, 0, 2, 1), (2, 1, 1, 2)]


def test_preload_admission_and_prefix_first(make):
    m = _four_sessions(make)
    m.evict(4)                               # B offloaded: host slots 0..3 hold positions 3..0
    # 4 blocks x 1e6 B at 1e9 B/s = 4 ms
    ok, r, e = m.preload(1, 0.0039, 1e6, 1e9)
    assert not ok and len(r) == 0 and len(e) == 0
    assert m.session_info(1)[1] & 0x2       # protected even when not admitted
    ok, r, e = m.preload(1, 0.0040, 1e6, 1e9)
    assert ok and len(e) == 0
    assert _moves(r) == [(1, 0, 4, 3), (1, 1, 5, 2), (1, 2, 6, 1), (1, 3, 7, 0)]
    assert list(m.table(1)[2]) == [2, 2, 2, 2]
    m.preload_done(1, 10.0)
    dev, host, state = m.table(1)
    assert list(dev) == [4, 5, 6, 7] and list(host) == [-1] * 4 and list(state) == [0] * 4
    assert m.session_info(1)[1] == 0x4       # warm, not a candidate
    m.tick(14.9)
    assert m.session_info(1)[1] == 0x4
    m.tick(15.0)                              # warm_ttl_s = 5
    assert m.session_info(1)[1] == 0x8


def test_preload_evicts_later_use_kv_for_room(make):
    m = make(8, 16, 4, reply_prior_s=0.0)
    for s, t in ((0, 1.0), (1, 9.0), (2, 5.0)):
        m.add_session(s)
        m.append_blocks(s, 2)                 # blocks 0-1, 2-3, 4-5
        m.set_playback(s, t)
    m.evict(2)                                # session 1 (T_next 9) -> host 0, 1
    m.add_session(3)
    m.append_blocks(3, 4)                     # fills the pool: blocks 2, 3, 6, 7
    ok, r, e = m.preload(1, 10.0, 1.0, 1.0)   # needs 2 blocks: evicts session 2 (5) before 0 (1) and 3 (0)
    assert ok
    assert _moves(e) == [(2, 1, 5, 2), (2, 0, 4, 3), ]
    assert _moves(r) == [(1, 0, 4, 1), (1, 1, 5, 0)]
    # not admitted when the others cannot make room (everything else protected)
    m2 = make(2, 4, 2)
    m2.add_session(0)
    m2.append_blocks(0, 2)
    m2.evict(2)
    m2.add_session(1)
    m2.append_blocks(1, 2)
    m2.set_running(1, True)
    ok, r, e = m2.preload(0, 1e9, 1.0, 1.0)
    assert not ok and len(r) == 0 and len(e) == 0


def test_cancel_then_synchronous_fallback(make):
    m = _four_sessions(make)
    m.evict(4)
    ok, r, _ = m.preload(1, 1.0, 0.0, 1.0)
    assert ok and len(r) == 4
    m.preload_cancel(1)
    assert list(m.table(1)[2]) == [1, 1, 1, 1]
    assert m.counts()["free_device_blocks"] == 20
    r, e = m.load_sync(1)
    assert _moves(r) == [(1, 0, 4, 3), (1, 1, 5, 2), (1, 2, 6, 1), (1, 3, 7, 0)] and len(e) == 0
    m.set_running(1, True)                   # the turn starts: pinned
    m.preload_done(1, 0.0)
    assert m.session_info(1)[1] == 0x1


def test_warm_cap_releases_oldest(make):
    m = make(16, 16, 4, warm_cap_blocks=6)
    for s in range(2):
        m.add_session(s)
        m.append_blocks(s, 4)
        m.preload(s, 1.0, 0.0, 1.0)           # nothing offloaded: admitted, protected
    m.preload_done(0, 1.0)
    assert m.counts()["warm_blocks"] == 4
    m.preload_done(1, 2.0)                    # 8 > 6: session 0 (older) loses protection
    assert m.session_info(0)[1] == 0x8 and m.session_info(1)[1] == 0x4
    assert m.counts()["warm_blocks"] == 4


def _random_run(seed, steps=400):
    rng = np.random.default_rng(seed)
    # small pools, so that appends run out, evictions empty sessions and
    # preloads must evict to make room or are refused
    nd, nh, ns = int(rng.integers(12, 48)), int(rng.integers(10, 120)), 12
    kw = dict(reply_prior_s=float(rng.choice([0.0, 2.0, 3.0])), reply_ema_alpha=float(rng.choice([0.25, 0.5, 1.0])),
              seconds_per_token=0.04, warm_ttl_s=3.0, warm_cap_blocks=int(rng.integers(0, 40)))
    ref, lib = RefKVManager(nd, nh, ns, **kw), _lib_manager(nd, nh, ns, **kw)
    now = 0.0
    for step in range(steps):
        op = int(rng.choice(12, p=[0.2] + [0.8 / 11] * 11))
        s = int(rng.integers(0, ns))
        have = s in ref.sessions
        what = "step %d op %d session %d" % (step, op, s)
        if not have:
            ref.add_session(s)
            lib.add_session(s)
        elif op == 0:
            n = int(rng.integers(0, 9))
            if len(ref.free_dev) >= n:
                assert list(ref.append_blocks(s, n)) == list(lib.append_blocks(s, n)), what
        elif op == 1:
            r = bool(rng.integers(0, 2))
            ref.set_running(s, r)
            lib.set_running(s, r)
        elif op == 2:
            t = float(rng.choice([-1.0, 0.0, rng.uniform(0, 20)]))
            k = int(rng.integers(0, 300))
            ref.set_playback(s, t, k)
            lib.set_playback(s, t, k)
        elif op == 3:
            x = float(rng.uniform(0, 10))
            ref.observe_reply(s, x)
            lib.observe_reply(s, x)
        elif op == 4:
            ref.speech_start(s)
            lib.speech_start(s)
        elif op in (5, 6):
            n = int(rng.integers(0, 15))
            assert ref.evict(n) == _moves(lib.evict(n)), what
        elif op == 7:
            if any(e[2] == 2 for e in ref.sessions[s]["table"]):
                continue
            t = float(rng.uniform(0, 2))
            a, r, e = ref.preload(s, t, 1.0, 10.0)
            b, r2, e2 = lib.preload(s, t, 1.0, 10.0)
            assert (a, r, e) == (b, _moves(r2), _moves(e2)), what
        elif op == 8:
            now += float(rng.uniform(0, 2))
            ref.preload_done(s, now)
            lib.preload_done(s, now)
        elif op == 9:
            ref.preload_cancel(s)
            lib.preload_cancel(s)
        elif op == 10:
            now += float(rng.uniform(0, 2))
            ref.tick(now)
            lib.tick(now)
        else:
            if rng.integers(0, 4) == 0:
                ref.remove_session(s)
                lib.remove_session(s)
        for j in ref.sessions:
            assert ref.session_info(j) == lib.session_info(j), (what, j)
            d, h, st = lib.table(j)
            assert ref.table(j) == (list(d), list(h), list(st)), (what, j)
        assert ref.counts() == lib.counts(), what


@pytest.mark.parametrize("seed", range(24))
def test_library_matches_oracle_on_random_event_sequences(seed):
    _random_run(seed)


def test_errors_leave_state_unchanged():
    from paper_2606_22983_amd.kv import LiveServeError
    m = _lib_manager(4, 4, 2)
    m.add_session(0)
    with pytest.raises(LiveServeError):
        m.add_session(0)
    with pytest.raises(LiveServeError):
        m.add_session(2)
    with pytest.raises(LiveServeError):
        m.append_blocks(0, 5)
    assert m.counts()["free_device_blocks"] == 4
    with pytest.raises(LiveServeError):
        m.observe_reply(0, -1.0)
    with pytest.raises(LiveServeError):
        _lib_manager(4, 4, 2, reply_ema_alpha=0.0)
