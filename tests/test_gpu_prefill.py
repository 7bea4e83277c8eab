"""GPU parity of paged_attn_prefill (next-turn prefill over reused context)."""
import math

import numpy as np
import pytest
import torch

from paper_2606_22983_amd import workloads as W
from tests.gpu_util import DevicePool, assert_attn_close, bf16_dev, i32_dev, log, scale_keys

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def kv():
    from paper_2606_22983_amd import kv as kv_mod
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return kv_mod


def _case(rng, n, c, hq, hkv, d, spare=3):
    n = np.asarray(n, np.int64)
    c = np.asarray(c, np.int64)
    need = (c + n + 15) // 16
    nb = int(need.sum()) + spare
    perm = rng.permutation(nb).astype(np.int32)
    tables = np.full((len(n), int(need.max())), -1, np.int32)
    pos = 0
    for s, k in enumerate(need):
        tables[s, :k] = perm[pos:pos + k]
        pos += k
    pool = W.normal_bf16(rng, (1, nb, 2, hkv, 16 * d))
    W._poison(pool, d, tables, c, int(need.sum()))
    total = int(n.sum())
    q = W.normal_bf16(rng, (total, hq, d))
    kn = W.normal_bf16(rng, (total, hkv, d))
    vn = W.normal_bf16(rng, (total, hkv, d))
    return pool, tables, q, kn, vn


def _run(kv, dp, q, kn, vn, n, c, tables, scale, host=False, queue=False):
    """host: lengths also on the host (host-dealt schedule); queue: with the
    item-counter workspace (XCDs take over each other's last tiles)."""
    cu = np.concatenate([[0], np.cumsum(n)]).astype(np.int32)
    out = torch.empty((q.shape[0], q.shape[1], q.shape[2]), dtype=torch.bfloat16, device="cuda")
    lens_host = np.stack([np.asarray(n), np.asarray(c)], 1) if host else None
    ws = torch.full((kv.PREFILL_WORKSPACE_BYTES,), 0x5A, dtype=torch.uint8, device="cuda") if queue else None
    kv.paged_attn_prefill(dp.pool, 0, bf16_dev(q), i32_dev(cu), i32_dev(c), int(np.max(n)),
                          i32_dev(tables), scale, out, bf16_dev(kn), bf16_dev(vn), lens_host=lens_host,
                          workspace=ws)
    return out, cu


@pytest.mark.parametrize("mode", ["device-lengths", "host-lengths", "host-lengths-counters"])
@pytest.mark.parametrize("d,hq,hkv", [(128, 32, 4), (64, 8, 2), (128, 8, 8), (128, 16, 8),
                                      (64, 4, 1)])
def test_prefill_ragged(kv, oracle_lib, d, hq, hkv, mode):
    """Turn lengths and contexts around tile and block boundaries, c = 0 included;
    the schedule dealt in the kernel, or on the host from host lengths, with or
    without the item counters (a workspace filled with garbage first)."""
    rng = np.random.default_rng(d + hq * 3 + hkv)
    n = [1, 17, 16, 130, 37, 255, 64]
    c = [0, 5, 300, 0, 1000, 77, 16]
    pool, tables, q, kn, vn = _case(rng, n, c, hq, hkv, d)
    dp = DevicePool(kv, pool, d)
    out, cu = _run(kv, dp, q, kn, vn, np.array(n), np.array(c), tables, 1 / math.sqrt(d),
                   host=mode != "device-lengths", queue=mode.endswith("counters"))
    ref, ref_pool = oracle_lib.prefill(pool, 16, d, 0, q, kn, vn, cu, c, tables, 1 / math.sqrt(d),
                                       pool_out=True)
    assert_attn_close(out, ref, "prefill D=%d G=%d" % (d, hq // hkv))
    assert np.array_equal(dp.host(), ref_pool), "appended pool differs from the oracle's"
    assert kv.ls_device_errors() == 0


@pytest.mark.parametrize("hkv", [2, 4])
def test_prefill_many_sessions(kv, oracle_lib, hkv):
    """140 sessions with empty turns mixed in.  With 2 KV heads (280 session/KV-head
    pairs) the in-kernel longest-first XCD schedule runs; with 4 KV heads (560
    pairs, above the 512 it orders) the workgroups take their items in index order."""
    rng = np.random.default_rng(140 + hkv)
    d, hq = 64, 8
    n = rng.integers(0, 40, size=140)
    n[0] = 39
    c = rng.integers(0, 200, size=140)
    assert (140 * hkv > 512) == (hkv == 4)
    pool, tables, q, kn, vn = _case(rng, n, c, hq, hkv, d)
    dp = DevicePool(kv, pool, d)
    out, cu = _run(kv, dp, q, kn, vn, n, c, tables, 0.125)
    ref = oracle_lib.prefill(pool, 16, d, 0, q, kn, vn, cu, c, tables, 0.125)
    assert_attn_close(out, ref, "prefill, 140 sessions x %d KV heads" % hkv)
    assert kv.ls_device_errors() == 0


def test_prefill_index_order_long_turns(kv, oracle_lib):
    """The index-order schedule (600 pairs) with turns spanning several query
    tiles and contexts spanning several key tiles, ragged tails everywhere."""
    rng = np.random.default_rng(600)
    d, hq, hkv = 128, 16, 4
    S = 150
    n = rng.integers(0, 200, size=S)
    n[:3] = [199, 64, 65]
    c = rng.integers(0, 700, size=S)
    pool, tables, q, kn, vn = _case(rng, n, c, hq, hkv, d)
    dp = DevicePool(kv, pool, d)
    out, cu = _run(kv, dp, q, kn, vn, n, c, tables, 1 / math.sqrt(d))
    ref = oracle_lib.prefill(pool, 16, d, 0, q, kn, vn, cu, c, tables, 1 / math.sqrt(d))
    assert_attn_close(out, ref, "prefill, %d pairs in index order" % (S * hkv))
    assert kv.ls_device_errors() == 0


def test_prefill_turn_longer_than_max_new_len_is_flagged(kv, oracle_lib):
    """max_new_len understated: the grid has tiles for max_new_len tokens only.
    The device flags LS_DEVERR_LENGTH; rows inside the tiles are still right, and
    the whole turn is appended."""
    rng = np.random.default_rng(41)
    d, hq, hkv = 128, 32, 4                   # 256 rows / G = 32 tokens per query tile
    n, c = np.array([100, 40]), np.array([70, 300])
    pool, tables, q, kn, vn = _case(rng, n, c, hq, hkv, d)
    dp = DevicePool(kv, pool, d)
    kv.ls_device_errors()
    cu = np.concatenate([[0], np.cumsum(n)]).astype(np.int32)
    out = torch.zeros((q.shape[0], hq, d), dtype=torch.bfloat16, device="cuda")
    kv.paged_attn_prefill(dp.pool, 0, bf16_dev(q), i32_dev(cu), i32_dev(c), 40, i32_dev(tables),
                          0.0884, out, bf16_dev(kn), bf16_dev(vn))
    assert kv.ls_device_errors() & kv.LS_DEVERR_LENGTH
    covered = np.concatenate([np.arange(0, 64), np.arange(100, 140)])   # 2 tiles of 32 tokens
    ref, ref_pool = oracle_lib.prefill(pool, 16, d, 0, q, kn, vn, cu, c, tables, 0.0884, rows=covered,
                                       pool_out=True)
    assert_attn_close(out[torch.from_numpy(covered).cuda()], ref, "prefill rows inside the tiles")
    assert np.array_equal(dp.host(), ref_pool)
    with pytest.raises(kv.LiveServeError):     # with host lengths it is refused before launch
        kv.paged_attn_prefill(dp.pool, 0, bf16_dev(q), i32_dev(cu), i32_dev(c), 40, i32_dev(tables),
                              0.0884, out, bf16_dev(kn), bf16_dev(vn),
                              lens_host=np.stack([n, c], 1))


def test_prefill_host_lengths_same_result(kv):
    """Host (n, c) pairs change validation and the schedule (dealt on the host),
    not the arithmetic of any row: same bits, empty turns included."""
    rng = np.random.default_rng(43)
    d, hq, hkv = 128, 32, 4
    n, c = np.array([300, 1, 77, 0, 150]), np.array([900, 16, 0, 40, 333])
    pool, tables, q, kn, vn = _case(rng, n, c, hq, hkv, d)
    cu = np.concatenate([[0], np.cumsum(n)]).astype(np.int32)
    outs = []
    ws = torch.empty(kv.PREFILL_WORKSPACE_BYTES, dtype=torch.uint8, device="cuda")
    for lens_host, w in ((None, None), (np.stack([n, c], 1), None), (np.stack([n, c], 1), ws)):
        dp = DevicePool(kv, pool, d)
        out = torch.empty((q.shape[0], hq, d), dtype=torch.bfloat16, device="cuda")
        kv.paged_attn_prefill(dp.pool, 0, bf16_dev(q), i32_dev(cu), i32_dev(c), int(n.max()),
                              i32_dev(tables), 0.0884, out, bf16_dev(kn), bf16_dev(vn),
                              lens_host=lens_host, workspace=w)
        outs.append(out)
    assert torch.equal(outs[0].view(torch.int16), outs[1].view(torch.int16))
    assert torch.equal(outs[0].view(torch.int16), outs[2].view(torch.int16))
    assert kv.ls_device_errors() == 0


@pytest.mark.parametrize("queue", [False, True], ids=["fixed", "counters"])
@pytest.mark.parametrize("S", [64, 65])
def test_prefill_host_plan_capacity(kv, oracle_lib, S, queue):
    """Host lengths with 4 KV heads: 64 sessions (256 session/KV-head pairs) fill
    the host-dealt schedule; 65 sessions (260 pairs) exceed it and the kernel
    deals the schedule itself.  Empty turns mixed in."""
    rng = np.random.default_rng(900 + S)
    d, hq, hkv = 64, 8, 4
    n = rng.integers(0, 40, size=S)
    n[1] = 0
    n[S - 1] = 39
    c = rng.integers(0, 200, size=S)
    pool, tables, q, kn, vn = _case(rng, n, c, hq, hkv, d)
    dp = DevicePool(kv, pool, d)
    out, cu = _run(kv, dp, q, kn, vn, n, c, tables, 0.125, host=True, queue=queue)
    ref = oracle_lib.prefill(pool, 16, d, 0, q, kn, vn, cu, c, tables, 0.125)
    assert_attn_close(out, ref, "prefill, %d sessions x %d KV heads, host lengths" % (S, hkv))
    assert kv.ls_device_errors() == 0


def test_prefill_device_turn_longer_than_host_is_flagged(kv, oracle_lib):
    """Host lengths that pass every host check but understate a turn on the
    device: the host-dealt schedule has 8 query tiles (256 tokens) for a turn of
    300.  The device flags LS_DEVERR_LENGTH; rows inside the planned tiles are
    still right."""
    rng = np.random.default_rng(44)
    d, hq, hkv = 128, 32, 4                   # 32 tokens per query tile
    n, c = np.array([300, 100]), np.array([500, 50])
    pool, tables, q, kn, vn = _case(rng, n, c, hq, hkv, d)
    assert tables.shape[1] * 16 >= 150 + 50       # the claimed lengths fit the table
    dp = DevicePool(kv, pool, d)
    kv.ls_device_errors()
    cu = np.concatenate([[0], np.cumsum(n)]).astype(np.int32)
    out = torch.zeros((q.shape[0], hq, d), dtype=torch.bfloat16, device="cuda")
    claimed = np.stack([[250, 150], c], 1)    # adds up to the same 400 tokens
    kv.paged_attn_prefill(dp.pool, 0, bf16_dev(q), i32_dev(cu), i32_dev(c), 300, i32_dev(tables),
                          0.0884, out, bf16_dev(kn), bf16_dev(vn), lens_host=claimed)
    assert kv.ls_device_errors() & kv.LS_DEVERR_LENGTH
    covered = np.concatenate([np.arange(0, 256), np.arange(300, 400)])
    ref = oracle_lib.prefill(pool, 16, d, 0, q, kn, vn, cu, c, tables, 0.0884, rows=covered)
    assert_attn_close(out[torch.from_numpy(covered).cuda()], ref, "prefill rows inside the planned tiles")


@pytest.mark.parametrize("shape", ["rising", "spike", "falling"])
@pytest.mark.parametrize("d,hq,hkv", [(128, 32, 4), (64, 8, 8)])
def test_prefill_peaky_scores(kv, oracle_lib, shape, d, hq, hkv):
    """Large, uneven scores: key norms that rise along the context (the running
    max is raised many times), one block of much larger keys late in the context,
    or norms that fall (the first keys hold the max).  Scores reach tens of log2
    units, so the rescale path and the exactness of the scaled scores are tested."""
    rng = np.random.default_rng({"rising": 71, "spike": 72, "falling": 73}[shape] + d)
    n, c = [200, 70, 33], [1500, 700, 0]
    pool, tables, q, kn, vn = _case(rng, n, c, hq, hkv, d)
    scale_keys(pool, tables, c, shape)
    if shape == "rising":               # the turn's own keys continue the ramp
        kn = W.to_bf16(W.from_bf16(kn) * np.float32(10.0))
    dp = DevicePool(kv, pool, d)
    out, cu = _run(kv, dp, q, kn, vn, np.array(n), np.array(c), tables, 1 / math.sqrt(d))
    ref = oracle_lib.prefill(pool, 16, d, 0, q, kn, vn, cu, c, tables, 1 / math.sqrt(d))
    assert_attn_close(out, ref, "prefill %s keys D=%d G=%d" % (shape, d, hq // hkv))
    assert kv.ls_device_errors() == 0


@pytest.mark.parametrize("mode", ["device-lengths", "host-lengths-counters"])
def test_prefill_over_a_262144_token_context(kv, oracle_lib, mode):
    """A turn over the longest context a decode call takes (16384 blocks):
    4096 key tiles per query tile, fp32 row sums over 262,144 keys; a second
    session with an empty context beside it."""
    rng = np.random.default_rng(16384)
    d, hq, hkv = 64, 2, 1
    n = np.array([16, 300])
    c = np.array([262144 - 16, 0])
    pool, tables, q, kn, vn = _case(rng, n, c, hq, hkv, d)
    assert tables.shape[1] == 16384
    dp = DevicePool(kv, pool, d)
    out, cu = _run(kv, dp, q, kn, vn, n, c, tables, 0.125, host=mode != "device-lengths",
                   queue=mode.endswith("counters"))
    ref, ref_pool = oracle_lib.prefill(pool, 16, d, 0, q, kn, vn, cu, c, tables, 0.125, pool_out=True)
    assert_attn_close(out, ref, "prefill over 262,144 keys, %s" % mode)
    assert np.array_equal(dp.host(), ref_pool), "appended pool differs from the oracle's"
    assert kv.ls_device_errors() == 0


def test_prefill_chunked_equals_whole_turn(kv):
    """Two chunks (c advanced by the first) give the same rows as one call."""
    rng = np.random.default_rng(12)
    d, hq, hkv = 128, 32, 4
    n, c, n1 = 300, 517, 133
    pool, tables, q, kn, vn = _case(rng, [n], [c], hq, hkv, d)
    dp1 = DevicePool(kv, pool, d)
    whole, _ = _run(kv, dp1, q, kn, vn, np.array([n]), np.array([c]), tables, 0.0884)
    dp2 = DevicePool(kv, pool, d)
    a, _ = _run(kv, dp2, q[:n1], kn[:n1], vn[:n1], np.array([n1]), np.array([c]), tables, 0.0884)
    b, _ = _run(kv, dp2, q[n1:], kn[n1:], vn[n1:], np.array([n - n1]), np.array([c + n1]), tables,
                0.0884)
    assert torch.equal(torch.cat([a, b]).view(torch.int16), whole.view(torch.int16))
    assert np.array_equal(dp1.host(), dp2.host())


def test_next_turn_prefill_full_sampled(kv, oracle_lib):
    case = W.next_turn_prefill()
    n = case.new_lens.astype(np.int64)
    log("next-turn prefill: %d sessions, %d new tokens, %d reused, pool %.2f GB" % (
        case.num_sessions, int(n.sum()), int(case.reused_lens.sum()), case.pool.nbytes / 1e9))
    dp = DevicePool(kv, case.pool.data, 128)
    out, cu = _run(kv, dp, case.q, case.k_new, case.v_new, n, case.reused_lens, case.block_tables,
                   case.scale)
    torch.cuda.synchronize()
    # Sampled rows: the first and last row of every query tile of every session
    # (a tile holds 256 / G = 32 new tokens), plus random rows.
    qtok = 256 // (case.num_q_heads // case.pool.num_kv_heads)
    rng = np.random.default_rng(33)
    rows = set()
    for s in range(case.num_sessions):
        for j0 in range(0, int(n[s]), qtok):
            rows.update([int(cu[s]) + j0, int(cu[s]) + min(j0 + qtok, int(n[s])) - 1])
    rows.update(rng.integers(0, int(cu[-1]), size=40).tolist())
    rows = np.array(sorted(rows))
    ref = oracle_lib.prefill(case.pool.data, 16, 128, 0, case.q, case.k_new, case.v_new, cu,
                             case.reused_lens, case.block_tables, case.scale, rows=rows)
    assert_attn_close(out[torch.from_numpy(rows).cuda()], ref,
                      "next-turn prefill (%d sampled rows)" % len(rows))
    assert kv.ls_device_errors() == 0
    # The timed form of the call (host lengths: schedule dealt on the host)
    # computes every row with the same arithmetic: all rows, same bits.
    for queue in (False, True):
        out_h, _ = _run(kv, dp, case.q, case.k_new, case.v_new, n, case.reused_lens, case.block_tables,
                        case.scale, host=True, queue=queue)
        assert torch.equal(out_h.view(torch.int16), out.view(torch.int16)), "counters=%s" % queue
    assert kv.ls_device_errors() == 0


@pytest.mark.parametrize("n,c", [(1, 0), (700, 1500)])
def test_prefill_counters_single_pair(kv, oracle_lib, n, c):
    """One session and one KV head: the host deals every query tile to one XCD,
    so with the item counters the other XCDs' workgroups take all their tiles
    from that list (or, for a single tile, find nothing and end)."""
    rng = np.random.default_rng(300 + n)
    d, hq, hkv = 128, 8, 1
    pool, tables, q, kn, vn = _case(rng, [n], [c], hq, hkv, d)
    dp = DevicePool(kv, pool, d)
    out, cu = _run(kv, dp, q, kn, vn, np.array([n]), np.array([c]), tables, 1 / math.sqrt(d), host=True,
                   queue=True)
    ref = oracle_lib.prefill(pool, 16, d, 0, q, kn, vn, cu, np.array([c]), tables, 1 / math.sqrt(d))
    assert_attn_close(out, ref, "prefill, one pair, %d new tokens, counters" % n)
    assert kv.ls_device_errors() == 0


def test_prefill_with_counters_captured_and_replayed(kv, oracle_lib):
    """The call with host lengths and the counter workspace (a clearing kernel,
    then the prefill) captured in a graph: every replay, with eager calls
    between them, gives the eager result bit for bit."""
    rng = np.random.default_rng(77)
    d, hq, hkv = 128, 32, 4
    n, c = np.array([300, 45, 129, 1, 200]), np.array([1200, 0, 400, 31, 900])
    pool, tables, q, kn, vn = _case(rng, n, c, hq, hkv, d)
    dp = DevicePool(kv, pool, d)
    cu = np.concatenate([[0], np.cumsum(n)]).astype(np.int32)
    args = [bf16_dev(q), i32_dev(cu), i32_dev(c), int(n.max()), i32_dev(tables), 0.0884]
    kn_d, vn_d = bf16_dev(kn), bf16_dev(vn)
    lens_host = np.stack([n, c], 1)
    ws = torch.empty(kv.PREFILL_WORKSPACE_BYTES, dtype=torch.uint8, device="cuda")
    eager = torch.empty((q.shape[0], hq, d), dtype=torch.bfloat16, device="cuda")
    kv.paged_attn_prefill(dp.pool, 0, *args, eager, kn_d, vn_d, lens_host=lens_host, workspace=ws)
    out = torch.empty_like(eager)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        kv.paged_attn_prefill(dp.pool, 0, *args, out, kn_d, vn_d, lens_host=lens_host, workspace=ws)
    torch.cuda.synchronize()
    for rep in range(3):
        out.fill_(0)
        ws.fill_(0x77)                        # garbage counters: the replay clears them
        kv.paged_attn_prefill(dp.pool, 0, *args, eager, kn_d, vn_d, lens_host=lens_host)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int16), eager.view(torch.int16)), "replay %d" % rep
    ref = oracle_lib.prefill(pool, 16, d, 0, q, kn, vn, cu, c, tables, 0.0884)
    assert_attn_close(out, ref, "prefill replayed from a graph")
    assert kv.ls_device_errors() == 0
