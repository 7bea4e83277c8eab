"""The talker's 32-step decode loop (append + decode + split merge per step)
captured as one HIP graph and replayed: every replay gives bit for bit the
eager outputs and pool, with eager work between the replays."""
import numpy as np
import pytest
import torch

from paper_2606_22983_amd import workloads as W
from tests.gpu_util import DevicePool, bf16_dev, i32_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def kv():
    from paper_2606_22983_amd import kv as kv_mod
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return kv_mod


def test_captured_talker_steps_replay_exactly(kv):
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

    def steps():
        for t in range(case.steps):
            kv.paged_attn_decode(dp.pool, 0, qs[t], tables, lens[t], case.scale, outs[t], ws, kns[t], vns[t])

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
