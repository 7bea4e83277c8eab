"""The talker's decode loop (each step appends its token, attends, merges its
splits) captured as one HIP graph and replayed: every replay gives bit for bit
the eager outputs and pool, with eager work between the replays, and the
replayed steps match the oracle."""
import numpy as np
import pytest
import torch

from paper_2606_22983_amd import workloads as W
from tests.gpu_util import DevicePool, assert_attn_close, bf16_dev, i32_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def kv():
    from paper_2606_22983_amd import kv as kv_mod
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return kv_mod


@pytest.mark.parametrize("host_lengths", [False, True])
def test_captured_talker_steps_replay_exactly(kv, oracle_lib, host_lengths):
    case = W.talker_decode(num_sessions=64, steps=8)
    dp = DevicePool(kv, case.pool.data, 128)
    tables = i32_dev(case.block_tables)
    S, hq = case.q.shape[1], case.q.shape[2]
    qs = [bf16_dev(case.q[t]) for t in range(case.steps)]
    kns = [bf16_dev(case.k_new[t]) for t in range(case.steps)]
    vns = [bf16_dev(case.v_new[t]) for t in range(case.steps)]
    lens = [i32_dev(case.lens_at(t)) for t in range(case.steps)]
    outs = [torch.empty((S, hq, 128), dtype=torch.bfloat16, device="cuda") for _ in range(case.steps)]
    ws = torch.zeros(kv.decode_workspace_bytes(dp.pool, S, hq, case.block_tables.shape[1]),
                     dtype=torch.uint8, device="cuda")

    lens_h = [case.lens_at(t) if host_lengths else None for t in range(case.steps)]

    def steps():
        for t in range(case.steps):
            kv.paged_attn_decode(dp.pool, 0, qs[t], tables, lens[t], case.scale, outs[t], ws, kns[t], vns[t],
                                 context_lens_host=lens_h[t])

    steps()
    torch.cuda.synchronize()
    eager = [o.clone() for o in outs]
    pool_after = dp.data.clone()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        steps()
    for r in range(3):
        for o in outs:
            o.zero_()                               # eager work between replays
        g.replay()
        torch.cuda.synchronize()
        for t in range(case.steps):
            assert torch.equal(outs[t].view(torch.int16), eager[t].view(torch.int16)), (r, t)
        assert torch.equal(dp.data.view(torch.int16), pool_after.view(torch.int16)), r
    assert kv.ls_device_errors() == 0
    # The replayed steps against the oracle (each step appends its token first).
    ref_pool = case.pool.data.copy()
    for t in range(case.steps):
        lens_t = case.lens_at(t)
        if t in (0, 1, 4, 7):
            ref, ref_pool = oracle_lib.decode(ref_pool, 16, 128, 0, case.q[t], case.block_tables, lens_t,
                                              case.scale, k_new=case.k_new[t], v_new=case.v_new[t],
                                              pool_out=True)
            assert_attn_close(outs[t], ref, "graph replay, step %d" % t)
        else:
            oracle_lib.append(ref_pool, 16, 128, 0, case.block_tables, np.arange(S), lens_t,
                              case.k_new[t], case.v_new[t])
    assert np.array_equal(dp.host(), ref_pool), "pool after the replays differs from the oracle's"
