"""GPU parity of paged_attn_decode (through the C ABI) against the CPU oracle."""
import math

import numpy as np
import pytest
import torch

from paper_2606_22983_amd import workloads as W
from tests.gpu_util import (DevicePool, assert_attn_close, bf16_dev, host_bits, i32_dev, log,
                            run_decode, scale_keys)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def kv():
    from paper_2606_22983_amd import kv as kv_mod
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return kv_mod


def _decode_case(kv, oracle_lib, case, step=0, append=False, label=""):
    dp = DevicePool(kv, case.pool.data, case.pool.head_dim)
    lens = case.lens_at(step)
    q = bf16_dev(case.q[step])
    tables = i32_dev(case.block_tables)
    kn = bf16_dev(case.k_new[step]) if append else None
    vn = bf16_dev(case.v_new[step]) if append else None
    out, _ = run_decode(kv, dp, q, tables, i32_dev(lens), case.scale, kn, vn)
    ref, ref_pool = oracle_lib.decode(case.pool.data, 16, case.pool.head_dim, 0, case.q[step],
                                      case.block_tables, lens, case.scale,
                                      k_new=case.k_new[step] if append else None,
                                      v_new=case.v_new[step] if append else None, pool_out=True)
    assert_attn_close(out, ref, label or case.name)
    if append:
        assert np.array_equal(dp.host(), ref_pool), "appended pool differs from the oracle's"
    assert kv.ls_device_errors() == 0
    return out


@pytest.mark.parametrize("append", [False, True])
def test_tiny_decode(kv, oracle_lib, append):
    _decode_case(kv, oracle_lib, W.tiny_decode(append=append), append=append,
                 label="tiny decode append=%s" % append)


def _synthetic(rng, lens, hq, hkv, d, append, spare=5):
    """Random paged case with given lengths (block ids shuffled, tails NaN)."""
    lens = np.asarray(lens, dtype=np.int64)
    final = lens + (1 if append else 0)
    need = np.maximum((final + 15) // 16, 1)
    nb = int(need.sum()) + spare
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


@pytest.mark.parametrize("d,hq,hkv", [(128, 32, 4), (128, 16, 2), (64, 8, 2), (128, 8, 8),
                                      (64, 4, 2), (128, 4, 4)])
@pytest.mark.parametrize("append", [False, True])
def test_decode_lengths_and_groups(kv, oracle_lib, d, hq, hkv, append):
    """Ragged lengths around block and split boundaries, every supported group size."""
    rng = np.random.default_rng(hq * 7 + d + append)
    lens = [1, 2, 15, 16, 17, 63, 64, 65, 127, 128, 129, 255, 256, 257, 511, 512, 513, 1023, 1024,
            1025, 2047, 3001]
    if append:
        lens = [0] + lens
    pool, tables, q, kn, vn = _synthetic(rng, lens, hq, hkv, d, append)
    dp = DevicePool(kv, pool, d)
    out, _ = run_decode(kv, dp, bf16_dev(q), i32_dev(tables), i32_dev(lens), 1 / math.sqrt(d),
                        None if kn is None else bf16_dev(kn), None if vn is None else bf16_dev(vn))
    ref, ref_pool = oracle_lib.decode(pool, 16, d, 0, q, tables, np.array(lens), 1 / math.sqrt(d),
                                      k_new=kn, v_new=vn, pool_out=True)
    assert_attn_close(out, ref, "decode D=%d G=%d append=%s" % (d, hq // hkv, append))
    if append:
        assert np.array_equal(dp.host(), ref_pool)
    assert kv.ls_device_errors() == 0


@pytest.mark.parametrize("num_sessions", [255, 256, 257, 512, 513, 700])
def test_decode_batch_sizes_and_equal_short_splits(kv, oracle_lib, num_sessions):
    """Batches around the schedule's limits: up to 512 sessions the short
    splits are ranked by block count (many equal counts here), beyond that
    they run in session order; every item must run exactly once."""
    rng = np.random.default_rng(num_sessions)
    lens = rng.choice([1, 16, 17, 100, 1024, 1025, 1100, 2048, 2100], size=num_sessions)
    pool, tables, q, _, _ = _synthetic(rng, lens, 8, 2, 64, False)
    dp = DevicePool(kv, pool, 64)
    out, _ = run_decode(kv, dp, bf16_dev(q), i32_dev(tables), i32_dev(lens), 0.125)
    ref = oracle_lib.decode(pool, 16, 64, 0, q, tables, lens, 0.125)
    assert_attn_close(out, ref, "decode %d sessions" % num_sessions)
    assert kv.ls_device_errors() == 0


@pytest.mark.parametrize("limit", ["sessions", "tokens"])
def test_decode_at_the_size_limits(kv, oracle_lib, limit):
    """The largest batch a call takes (2048 sessions) and the longest context
    (16384 blocks, 262,144 keys: 256 splits of 1024 tokens, the merge kernel's
    full capacity), with device lengths and with host lengths; appended rows at
    the table's last slot included."""
    rng = np.random.default_rng(2048 if limit == "sessions" else 262144)
    if limit == "sessions":
        lens = rng.integers(1, 400, size=2048)
        lens[[0, 700, 2047]] = [5000, 4096, 1]
        hq, hkv, append = 8, 2, False
    else:
        lens = np.array([262144 - 1, 262144 - 700, 9000])
        hq, hkv, append = 8, 1, True
    pool, tables, q, kn, vn = _synthetic(rng, lens, hq, hkv, 64, append)
    if limit == "tokens":
        assert tables.shape[1] == 16384
    S = len(lens)
    dp = DevicePool(kv, pool, 64)
    ref, ref_pool = oracle_lib.decode(pool, 16, 64, 0, q, tables, lens, 0.125, k_new=kn, v_new=vn,
                                      pool_out=True)
    for host in (False, True):
        dp.data.copy_(bf16_dev(pool))
        ws = torch.zeros(kv.decode_workspace_bytes(dp.pool, S, hq, tables.shape[1]), dtype=torch.uint8,
                         device="cuda")
        out = torch.empty((S, hq, 64), dtype=torch.bfloat16, device="cuda")
        kv.paged_attn_decode(dp.pool, 0, bf16_dev(q), i32_dev(tables), i32_dev(lens), 0.125, out, ws,
                             None if kn is None else bf16_dev(kn), None if vn is None else bf16_dev(vn),
                             context_lens_host=lens if host else None)
        assert_attn_close(out, ref, "decode at the %s limit, host lengths %s" % (limit, host))
        if append:
            assert np.array_equal(dp.host(), ref_pool), "appended pool differs from the oracle's"
        assert kv.ls_device_errors() == 0


@pytest.mark.parametrize("append", [False, True])
def test_host_planned_batch_beyond_the_small_argument_block(kv, oracle_lib, append):
    """700 sessions x 2 KV heads with contexts up to 4500 tokens: more items than
    the small plan block holds (1280), so the plan goes in the large one."""
    rng = np.random.default_rng(700 + append)
    lens = rng.integers(1, 4500, size=700)
    lens[:3] = [1, 2048, 4499]
    pool, tables, q, kn, vn = _synthetic(rng, lens, 16, 2, 64, append)
    dp = DevicePool(kv, pool, 64)
    sc = _host_planned(kv, dp, 700, 16, tables.shape[1], lens, append)
    assert sc["host_planned"], sc
    ws = torch.zeros(kv.decode_workspace_bytes(dp.pool, 700, 16, tables.shape[1]), dtype=torch.uint8,
                     device="cuda")
    out = torch.empty((700, 16, 64), dtype=torch.bfloat16, device="cuda")
    kv.paged_attn_decode(dp.pool, 0, bf16_dev(q), i32_dev(tables), i32_dev(lens), 0.125, out, ws,
                         None if kn is None else bf16_dev(kn), None if vn is None else bf16_dev(vn),
                         context_lens_host=lens)
    ref, ref_pool = oracle_lib.decode(pool, 16, 64, 0, q, tables, lens, 0.125, k_new=kn, v_new=vn,
                                      pool_out=True)
    assert_attn_close(out, ref, "decode, 700 sessions host-planned in the large block, append=%s" % append)
    if append:
        assert np.array_equal(dp.host(), ref_pool)
    assert kv.ls_device_errors() == 0


@pytest.mark.parametrize("shape", ["rising", "spike", "falling"])
def test_decode_peaky_scores(kv, oracle_lib, shape):
    """Large, uneven scores (key norms rising along the context, one late block of
    much larger keys, or falling norms): the running-max raise and its rescale of
    (l, O), within a split and across the split merge."""
    rng = np.random.default_rng({"rising": 81, "spike": 82, "falling": 83}[shape])
    lens = [3001, 1025, 513, 77, 16]
    pool, tables, q, _, _ = _synthetic(rng, lens, 32, 4, 128, False)
    scale_keys(pool, tables, lens, shape)
    dp = DevicePool(kv, pool, 128)
    out, _ = run_decode(kv, dp, bf16_dev(q), i32_dev(tables), i32_dev(lens), 1 / math.sqrt(128))
    ref = oracle_lib.decode(pool, 16, 128, 0, q, tables, np.array(lens), 1 / math.sqrt(128))
    assert_attn_close(out, ref, "decode %s keys" % shape)
    assert kv.ls_device_errors() == 0


def test_one_key_returns_v_bit_exactly(kv):
    rng = np.random.default_rng(3)
    pool, tables, q, _, _ = _synthetic(rng, [1, 1, 1, 1], 32, 4, 128, False)
    dp = DevicePool(kv, pool, 128)
    out, _ = run_decode(kv, dp, bf16_dev(q), i32_dev(tables), i32_dev([1] * 4), 0.0884)
    got = host_bits(out)
    for s in range(4):
        vt = pool[0, tables[s, 0], 1].reshape(4, 128, 16)[:, :, 0]     # V of token 0, per KV head
        for h in range(32):
            assert np.array_equal(got[s, h], vt[h // 8]), (s, h)


def test_thinker_decode_full(kv, oracle_lib):
    case = W.thinker_decode()
    log("thinker decode: %d sessions, %d tokens, pool %.2f GB" % (
        case.num_sessions, int(case.context_lens.sum()), case.pool.nbytes / 1e9))
    _decode_case(kv, oracle_lib, case, label="thinker decode (64 sessions, full)")


def test_talker_decode_32_steps(kv, oracle_lib):
    case = W.talker_decode()
    log("talker decode: %d sessions, %d steps, pool %.2f GB" % (
        case.num_sessions, case.steps, case.pool.nbytes / 1e9))
    dp = DevicePool(kv, case.pool.data, 128)
    tables = i32_dev(case.block_tables)
    ws = None
    ref_pool = case.pool.data.copy()
    checked = {0, 1, 15, 16, 31}
    for t in range(case.steps):
        lens = case.lens_at(t)
        out, ws = run_decode(kv, dp, bf16_dev(case.q[t]), tables, i32_dev(lens), case.scale,
                             bf16_dev(case.k_new[t]), bf16_dev(case.v_new[t]), workspace=ws)
        if t in checked:
            ref, ref_pool = oracle_lib.decode(ref_pool, 16, 128, 0, case.q[t], case.block_tables,
                                              lens, case.scale, k_new=case.k_new[t],
                                              v_new=case.v_new[t], pool_out=True)
            assert_attn_close(out, ref, "talker step %d" % t)
        else:
            oracle_lib.append(ref_pool, 16, 128, 0, case.block_tables,
                              np.arange(case.num_sessions), lens, case.k_new[t], case.v_new[t])
    assert np.array_equal(dp.host(), ref_pool), "pool after 32 appends differs"
    assert kv.ls_device_errors() == 0


def test_decode_bitwise_deterministic_and_block_permutation_invariant(kv):
    case = W.tiny_decode()
    pool = case.pool.data
    dp = DevicePool(kv, pool, 64)
    q = bf16_dev(case.q[0])
    lens = i32_dev(case.context_lens)
    a, ws = run_decode(kv, dp, q, i32_dev(case.block_tables), lens, case.scale)
    b, _ = run_decode(kv, dp, q, i32_dev(case.block_tables), lens, case.scale, workspace=ws)
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    rng = np.random.default_rng(9)
    sigma = rng.permutation(pool.shape[1])
    moved = np.empty_like(pool)
    moved[:, sigma] = pool
    tables = np.where(case.block_tables >= 0, sigma[np.maximum(case.block_tables, 0)], -1)
    dp2 = DevicePool(kv, moved, 64)
    c, _ = run_decode(kv, dp2, q, i32_dev(tables), lens, case.scale)
    assert torch.equal(a.view(torch.int16), c.view(torch.int16))


def test_out_of_range_block_id_is_flagged_not_read(kv):
    rng = np.random.default_rng(4)
    pool, tables, q, _, _ = _synthetic(rng, [100, 40], 8, 2, 64, False)
    bad = tables.copy()
    bad[0, 2] = pool.shape[1] + 1000          # outside the pool
    bad[1, 0] = -7
    dp = DevicePool(kv, pool, 64)
    kv.ls_device_errors()
    out, _ = run_decode(kv, dp, bf16_dev(q), i32_dev(bad), i32_dev([100, 40]), 0.125)
    assert kv.ls_device_errors() & kv.LS_DEVERR_BLOCK_ID
    torch.cuda.synchronize()


def test_empty_context_is_flagged_with_zero_output(kv, oracle_lib):
    """A session with no key (length 0, no append) gets a zero output row and
    LS_DEVERR_LENGTH; the other sessions are unaffected.  With host lengths the
    call is refused before anything is enqueued."""
    rng = np.random.default_rng(10)
    lens = [40, 0, 1100, 3]
    pool, tables, q, _, _ = _synthetic(rng, lens, 32, 4, 128, False)
    dp = DevicePool(kv, pool, 128)
    kv.ls_device_errors()
    out, ws = run_decode(kv, dp, bf16_dev(q), i32_dev(tables), i32_dev(lens), 0.0884)
    assert kv.ls_device_errors() & kv.LS_DEVERR_LENGTH
    got = out.float().cpu().numpy()
    assert (got[1] == 0).all()
    keep = [0, 2, 3]
    ref = oracle_lib.decode(pool, 16, 128, 0, q, tables, np.array(lens), 0.0884, sessions=keep)
    assert_attn_close(out[keep], ref, "decode beside an empty context")
    with pytest.raises(kv.LiveServeError):
        kv.paged_attn_decode(dp.pool, 0, bf16_dev(q), i32_dev(tables), i32_dev(lens), 0.0884, out, ws,
                             context_lens_host=np.array(lens))
    # the same session with its own token appended has one key: fine
    kn, vn = W.normal_bf16(rng, (4, 4, 128)), W.normal_bf16(rng, (4, 4, 128))
    out2, _ = run_decode(kv, dp, bf16_dev(q), i32_dev(tables), i32_dev(lens), 0.0884, bf16_dev(kn),
                         bf16_dev(vn))
    ref2 = oracle_lib.decode(pool, 16, 128, 0, q, tables, np.array(lens), 0.0884, k_new=kn, v_new=vn)
    assert_attn_close(out2, ref2, "decode with append, context 0 included")
    assert kv.ls_device_errors() == 0


@pytest.mark.parametrize("append", [False, True])
def test_decode_with_host_lengths_matches_oracle(kv, oracle_lib, append):
    """context_lens_host given (host-side checks and split planning)."""
    rng = np.random.default_rng(20 + append)
    lens = rng.integers(1, 5000, size=96)
    lens[:4] = [1, 16, 1024, 4097]
    pool, tables, q, kn, vn = _synthetic(rng, lens, 16, 2, 128, append)
    dp = DevicePool(kv, pool, 128)
    ws = torch.zeros(kv.decode_workspace_bytes(dp.pool, 96, 16, tables.shape[1]), dtype=torch.uint8,
                     device="cuda")
    out = torch.empty((96, 16, 128), dtype=torch.bfloat16, device="cuda")
    kv.paged_attn_decode(dp.pool, 0, bf16_dev(q), i32_dev(tables), i32_dev(lens), 0.0884, out, ws,
                         None if kn is None else bf16_dev(kn), None if vn is None else bf16_dev(vn),
                         context_lens_host=lens)
    ref, ref_pool = oracle_lib.decode(pool, 16, 128, 0, q, tables, lens, 0.0884, k_new=kn, v_new=vn,
                                      pool_out=True)
    assert_attn_close(out, ref, "decode with host lengths, append=%s" % append)
    if append:
        assert np.array_equal(dp.host(), ref_pool)
    assert kv.ls_device_errors() == 0


def _host_planned(kv, dp, S, hq, maxb, lens, appended):
    return kv.ls_decode_schedule(dp.pool, S, hq, maxb, context_lens_host=lens, appended=appended)


def test_talker_32_steps_host_planned(kv, oracle_lib):
    """The talker loop with host lengths: the host plans one item per (session, KV
    head) and no merge runs; steps checked against the oracle, pool bit-exact."""
    case = W.talker_decode()
    dp = DevicePool(kv, case.pool.data, 128)
    tables = i32_dev(case.block_tables)
    ws = None
    ref_pool = case.pool.data.copy()
    checked = {0, 7, 16, 31}
    for t in range(case.steps):
        lens = case.lens_at(t)
        sc = _host_planned(kv, dp, case.num_sessions, case.num_q_heads, case.block_tables.shape[1], lens, True)
        assert sc["host_planned"] and not sc["merge"], sc
        if ws is None:
            ws = torch.zeros(kv.decode_workspace_bytes(dp.pool, case.num_sessions, case.num_q_heads,
                                                       case.block_tables.shape[1]), dtype=torch.uint8, device="cuda")
        out = torch.empty((case.num_sessions, case.num_q_heads, 128), dtype=torch.bfloat16, device="cuda")
        kv.paged_attn_decode(dp.pool, 0, bf16_dev(case.q[t]), tables, i32_dev(lens), case.scale, out, ws,
                             bf16_dev(case.k_new[t]), bf16_dev(case.v_new[t]), context_lens_host=lens)
        if t in checked:
            ref, ref_pool = oracle_lib.decode(ref_pool, 16, 128, 0, case.q[t], case.block_tables, lens, case.scale,
                                              k_new=case.k_new[t], v_new=case.v_new[t], pool_out=True)
            assert_attn_close(out, ref, "host-planned talker step %d (split %d)" % (t, sc["split_tokens"]))
        else:
            oracle_lib.append(ref_pool, 16, 128, 0, case.block_tables, np.arange(case.num_sessions), lens,
                              case.k_new[t], case.v_new[t])
    assert np.array_equal(dp.host(), ref_pool), "pool after 32 host-planned appends differs"
    assert kv.ls_device_errors() == 0


@pytest.mark.parametrize("append", [False, True])
def test_host_planned_with_splits_and_merge(kv, oracle_lib, append):
    """Mostly ~2k-key sessions and a few of 8000: the host splits the long sessions
    (items of several 1024-token chunks) and the merge runs."""
    rng = np.random.default_rng(90 + append)
    lens = np.concatenate([rng.integers(1500, 2040, 200), np.full(10, 8000), [1, 2047, 2048, 4097]])
    pool, tables, q, kn, vn = _synthetic(rng, lens, 16, 2, 128, append)
    dp = DevicePool(kv, pool, 128)
    sc = _host_planned(kv, dp, len(lens), 16, tables.shape[1], lens, append)
    log("schedule: %s" % sc)
    assert sc["host_planned"] and sc["merge"] and sc["split_tokens"] >= 2048
    ws = torch.zeros(kv.decode_workspace_bytes(dp.pool, len(lens), 16, tables.shape[1]), dtype=torch.uint8,
                     device="cuda")
    out = torch.empty((len(lens), 16, 128), dtype=torch.bfloat16, device="cuda")
    kv.paged_attn_decode(dp.pool, 0, bf16_dev(q), i32_dev(tables), i32_dev(lens), 0.0884, out, ws,
                         None if kn is None else bf16_dev(kn), None if vn is None else bf16_dev(vn),
                         context_lens_host=lens)
    ref, ref_pool = oracle_lib.decode(pool, 16, 128, 0, q, tables, lens, 0.0884, k_new=kn, v_new=vn, pool_out=True)
    assert_attn_close(out, ref, "host-planned with splits, append=%s" % append)
    if append:
        assert np.array_equal(dp.host(), ref_pool)
    assert kv.ls_device_errors() == 0


def test_host_plan_device_lengths_disagree(kv, oracle_lib):
    """Device lengths shorter than the host's: the plan covers them and the result
    is that of the device lengths.  Longer: the keys past the plan are flagged
    (LS_DEVERR_LENGTH), and nothing faults."""
    rng = np.random.default_rng(95)
    lens = rng.integers(600, 3000, size=256)
    pool, tables, q, _, _ = _synthetic(rng, lens, 16, 2, 128, False)
    dp = DevicePool(kv, pool, 128)
    host = lens.copy()
    assert _host_planned(kv, dp, 256, 16, tables.shape[1], host, False)["host_planned"]
    shorter = lens - rng.integers(0, 500, size=256)
    kv.ls_device_errors()
    out, ws = run_decode(kv, dp, bf16_dev(q), i32_dev(tables), i32_dev(shorter), 0.0884)
    out2 = torch.empty_like(out)
    kv.paged_attn_decode(dp.pool, 0, bf16_dev(q), i32_dev(tables), i32_dev(shorter), 0.0884, out2, ws,
                         context_lens_host=host)
    ref = oracle_lib.decode(pool, 16, 128, 0, q, tables, shorter, 0.0884)
    assert_attn_close(out2, ref, "host plan over shorter device lengths")
    assert kv.ls_device_errors() == 0
    # Device lengths of 2500-3000 keys (in the tables) against host lengths of at
    # most 2000: the plan's one 2048-token split per session stops short.
    real = rng.integers(2500, 3001, size=256)
    pool2, tables2, q2, _, _ = _synthetic(rng, real, 16, 2, 128, False)
    dp2 = DevicePool(kv, pool2, 128)
    claimed = rng.integers(600, 2001, size=256)
    sc = _host_planned(kv, dp2, 256, 16, tables2.shape[1], claimed, False)
    assert sc["host_planned"] and sc["split_tokens"] == 2048 and not sc["merge"], sc
    ws2 = torch.zeros(kv.decode_workspace_bytes(dp2.pool, 256, 16, tables2.shape[1]), dtype=torch.uint8,
                      device="cuda")
    out3 = torch.empty((256, 16, 128), dtype=torch.bfloat16, device="cuda")
    kv.paged_attn_decode(dp2.pool, 0, bf16_dev(q2), i32_dev(tables2), i32_dev(real), 0.0884, out3, ws2,
                         context_lens_host=claimed)
    assert kv.ls_device_errors() & kv.LS_DEVERR_LENGTH


def test_thinker_decode_full_host_planned(kv, oracle_lib):
    """The full thinker batch with host lengths: 2048-token splits in the 16-bit
    item form, two chunks per full split, merge."""
    case = W.thinker_decode()
    dp = DevicePool(kv, case.pool.data, 128)
    sc = kv.ls_decode_schedule(dp.pool, case.num_sessions, case.num_q_heads, case.block_tables.shape[1],
                               context_lens_host=case.context_lens)
    assert sc["host_planned"] and sc["merge"], sc
    ws = torch.zeros(kv.decode_workspace_bytes(dp.pool, case.num_sessions, case.num_q_heads,
                                               case.block_tables.shape[1]), dtype=torch.uint8, device="cuda")
    out = torch.empty((case.num_sessions, case.num_q_heads, 128), dtype=torch.bfloat16, device="cuda")
    kv.paged_attn_decode(dp.pool, 0, bf16_dev(case.q[0]), i32_dev(case.block_tables), i32_dev(case.context_lens),
                         case.scale, out, ws, context_lens_host=case.context_lens)
    ref = oracle_lib.decode(case.pool.data, 16, 128, 0, case.q[0], case.block_tables, case.context_lens, case.scale)
    assert_attn_close(out, ref, "thinker decode, host-planned (split %d)" % sc["split_tokens"])
    assert kv.ls_device_errors() == 0


@pytest.mark.parametrize("d,hq,hkv", [(128, 16, 8), (64, 8, 8)])
def test_host_planned_wide_items(kv, oracle_lib, d, hq, hkv):
    """Eight KV heads: the host plan's items take the 32-bit form (the 16-bit form
    holds at most 4 heads).  A few sessions are long enough to be split, so the
    merge runs; the step's token is appended."""
    rng = np.random.default_rng(225)
    lens = np.concatenate([rng.integers(1, 3000, 20), [6000, 6001, 1, 2048]])
    pool, tables, q, kn, vn = _synthetic(rng, lens, hq, hkv, d, True)
    dp = DevicePool(kv, pool, d)
    sc = _host_planned(kv, dp, len(lens), hq, tables.shape[1], lens, True)
    log("schedule: %s" % sc)
    assert sc["host_planned"] and sc["merge"], sc
    ws = torch.zeros(kv.decode_workspace_bytes(dp.pool, len(lens), hq, tables.shape[1]), dtype=torch.uint8,
                     device="cuda")
    out = torch.empty((len(lens), hq, d), dtype=torch.bfloat16, device="cuda")
    kv.paged_attn_decode(dp.pool, 0, bf16_dev(q), i32_dev(tables), i32_dev(lens), 1 / math.sqrt(d), out, ws,
                         bf16_dev(kn), bf16_dev(vn), context_lens_host=lens)
    ref, ref_pool = oracle_lib.decode(pool, 16, d, 0, q, tables, lens, 1 / math.sqrt(d), k_new=kn, v_new=vn,
                                      pool_out=True)
    assert_attn_close(out, ref, "host-planned, 8 KV heads, D=%d" % d)
    assert np.array_equal(dp.host(), ref_pool)
    assert kv.ls_device_errors() == 0
