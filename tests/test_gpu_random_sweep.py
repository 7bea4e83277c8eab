"""Seeded random sweep of the three entry points against the oracle.

Each case draws its own geometry (head_dim 64 or 128, 1-8 KV heads and groups
1-8, or 16-32 KV heads and groups 1-4; 1-3 layers with a random layer attended), batch shape (a length profile,
table widths wider than needed) and call mode (append or not, device or host
lengths, the static-scratch decode, prefill with or without the turn's K/V
and with or without the item counters), so that combinations the targeted
tests do not name still meet the oracle.  Sizes are bounded so the oracle
finishes each case in about a second.  Workspaces start filled with garbage.
"""
import math

import numpy as np
import pytest
import torch

from paper_2606_22983_amd import workloads as W
from tests.gpu_util import DevicePool, assert_attn_close, bf16_dev, host_bits, i32_dev, log

pytestmark = pytest.mark.gpu

POOL_ELEMS = 24 << 20          # bf16 elements of a case's pool, all layers
STATIC_SCRATCH = 32 << 20      # bytes of the library's static split scratch
DECODE_MACS = 6e8              # oracle multiply-adds per decode case (q.k and p.v)
PREFILL_MACS = 5e9


@pytest.fixture(scope="module")
def kv():
    from paper_2606_22983_amd import kv as kv_mod
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return kv_mod


def _geometry(rng, wide=False):
    """head_dim, KV heads, query heads, layers, attended layer.  ``wide``: 16 or
    32 KV heads (multi-head-like models), groups of 1, 2 or 4."""
    d = int(rng.choice([64, 128]))
    hkv = int(rng.choice([16, 32] if wide else [1, 2, 4, 8]))
    g = int(rng.choice([1, 2, 4] if wide else [1, 2, 4, 8]))
    nl = int(rng.integers(1, 4))
    return d, hkv, g * hkv, nl, int(rng.integers(0, nl))


def _paged(rng, valid, span, nl, hkv, d, extra_cols):
    """Pool and tables for sessions holding ``valid`` tokens now and ``span``
    tokens after the call (slots past ``valid`` are NaN until written)."""
    need = np.maximum((np.asarray(span) + 15) // 16, 1)
    nb = int(need.sum()) + int(rng.integers(0, 8))
    perm = rng.permutation(nb).astype(np.int32)
    tables = np.full((len(need), int(need.max()) + extra_cols), -1, np.int32)
    pos = 0
    for s, k in enumerate(need):
        tables[s, :k] = perm[pos:pos + k]
        pos += k
    pool = W.normal_bf16(rng, (nl, nb, 2, hkv, 16 * d))
    W._poison(pool, d, tables, np.asarray(valid), int(need.sum()))
    return pool, tables


def _decode_lengths(rng, append):
    lo = 0 if append else 1
    profile = str(rng.choice(["short", "mixed", "lognormal", "equal"]))
    if profile == "short":
        lens = rng.integers(lo, 65, size=int(rng.integers(1, 700)))
    elif profile == "mixed":
        lens = rng.integers(lo, 3001, size=int(rng.integers(1, 200)))
    elif profile == "lognormal":
        s = int(rng.integers(1, 65))
        lens = np.clip(np.round(np.exp(np.log(2000.0) + rng.standard_normal(s))), max(lo, 1), 20000)
    else:
        lens = np.full(int(rng.integers(1, 300)), int(rng.choice([16, 1023, 1024, 2048, 2049, 4100])))
    return profile, lens.astype(np.int64)


def decode_inputs(oracle_lib, seed, wide=False):
    """One seeded decode case and the oracle's result for it."""
    rng = np.random.default_rng((8600 if wide else 8100) + seed)
    d, hkv, hq, nl, layer = _geometry(rng, wide)
    append = bool(rng.random() < 0.5)
    host = bool(rng.random() < 0.5)
    static = bool(rng.random() < 0.25)
    profile, lens = _decode_lengths(rng, append)
    # Trim the batch to the oracle and pool budgets.
    while len(lens) > 1 and (lens.sum() * hq * d * 2 > DECODE_MACS or
                             (lens.sum() + 16 * len(lens)) * 2 * hkv * d * nl > POOL_ELEMS):
        lens = lens[: len(lens) // 2 + len(lens) // 4]
    if lens.sum() * 2 * hkv * d * nl > POOL_ELEMS:
        lens = np.minimum(lens, POOL_ELEMS // (4 * hkv * d * nl))
    S = len(lens)
    what = "decode seed %d: %s S=%d max %d D=%d Hq/Hkv=%d/%d layers %d (layer %d) append=%s host=%s static=%s" % (
        seed, profile, S, int(lens.max()), d, hq, hkv, nl, layer, append, host, static)
    log(what)
    span = lens + (1 if append else 0)
    pool, tables = _paged(rng, lens, span, nl, hkv, d, int(rng.integers(0, 3)))
    q = W.normal_bf16(rng, (S, hq, d))
    kn = W.normal_bf16(rng, (S, hkv, d)) if append else None
    vn = W.normal_bf16(rng, (S, hkv, d)) if append else None
    scale = float(rng.uniform(0.5, 1.5)) / math.sqrt(d)
    ref, ref_pool = oracle_lib.decode(pool, 16, d, layer, q, tables, lens, scale, k_new=kn, v_new=vn,
                                      pool_out=True)
    return dict(what=what, d=d, hq=hq, layer=layer, host=host, static=static, lens=lens, pool=pool,
                tables=tables, q=q, kn=kn, vn=vn, scale=scale, ref=ref, ref_pool=ref_pool)


@pytest.mark.parametrize("seed", range(64))
def test_decode_random(kv, oracle_lib, seed):
    _check_decode(kv, decode_inputs(oracle_lib, seed))


@pytest.mark.parametrize("seed", range(8))
def test_decode_random_many_kv_heads(kv, oracle_lib, seed):
    _check_decode(kv, decode_inputs(oracle_lib, seed, wide=True))


def _check_decode(kv, x):
    what, d, hq, layer, lens, tables, kn, vn, scale = (x[k] for k in ("what", "d", "hq", "layer", "lens",
                                                                      "tables", "kn", "vn", "scale"))
    S = len(lens)
    dp = DevicePool(kv, x["pool"], d)
    out = torch.empty((S, hq, d), dtype=torch.bfloat16, device="cuda")
    args = (dp.pool, layer, bf16_dev(x["q"]), i32_dev(tables), i32_dev(lens), scale, out)
    kw = dict(k_new=None if kn is None else bf16_dev(kn), v_new=None if vn is None else bf16_dev(vn),
              context_lens_host=lens.astype(np.int32) if x["host"] else None)
    nbytes = kv.decode_workspace_bytes(dp.pool, S, hq, tables.shape[1])
    if x["static"] and nbytes <= STATIC_SCRATCH:
        kv.paged_attn_decode_static(*args, **kw)
    else:
        ws = torch.full((max(nbytes, 1),), 0x5A, dtype=torch.uint8, device="cuda")
        kv.paged_attn_decode(*args, ws, **kw)
    assert_attn_close(out, x["ref"], what)
    assert np.array_equal(dp.host(), x["ref_pool"]), "%s: pool differs from the oracle's" % what
    assert kv.ls_device_errors() == 0


def _prefill_lengths(rng):
    S = int(rng.integers(1, 48))
    n = np.where(rng.random(S) < 0.5, rng.integers(1, 41, size=S), rng.integers(1, 701, size=S))
    n[rng.random(S) < 0.1] = 0
    if n.max() == 0:
        n[int(rng.integers(0, S))] = int(rng.integers(1, 300))
    c = rng.integers(0, 4001, size=S)
    c[rng.random(S) < 0.2] = 0
    on_block = rng.random(S) < 0.2
    c[on_block] = c[on_block] // 16 * 16
    return n.astype(np.int64), c.astype(np.int64)


def prefill_inputs(oracle_lib, seed, wide=False):
    """One seeded prefill case and the oracle's result for it."""
    rng = np.random.default_rng((9600 if wide else 9100) + seed)
    d, hkv, hq, nl, layer = _geometry(rng, wide)
    mode = str(rng.choice(["device-lengths", "host-lengths", "host-lengths-counters"]))
    with_kv = bool(rng.random() < 0.8)
    n, c = _prefill_lengths(rng)
    # Over the budgets, half of the cases drop sessions, the others shorten them.
    few = rng.random() < 0.5
    while few and len(n) > 1 and ((n * (c + n)).sum() * hq * d * 2 > PREFILL_MACS or
                                  ((c + n).sum() + 16 * len(n)) * 2 * hkv * d * nl > POOL_ELEMS):
        keep = len(n) // 2 + len(n) // 4
        n, c = n[:keep], c[:keep]
        if n.max() == 0:
            n[0] = 1
    while (n * (c + n)).sum() * hq * d * 2 > PREFILL_MACS or (c + n + 16).sum() * 2 * hkv * d * nl > POOL_ELEMS:
        c, n = c // 2, np.maximum(n // 2, np.minimum(n, 1))
    S = len(n)
    total = int(n.sum())
    max_new = int(n.max()) + (int(rng.integers(0, 40)) if rng.random() < 0.3 else 0)
    max_new = min(max_new, total)
    what = "prefill seed %d: S=%d n<=%d c<=%d D=%d Hq/Hkv=%d/%d layers %d (layer %d) %s k_new=%s" % (
        seed, S, int(n.max()), int(c.max()), d, hq, hkv, nl, layer, mode, with_kv)
    log(what)
    pool, tables = _paged(rng, c if with_kv else c + n, c + n, nl, hkv, d, int(rng.integers(0, 3)))
    q = W.normal_bf16(rng, (total, hq, d))
    kn = W.normal_bf16(rng, (total, hkv, d))
    vn = W.normal_bf16(rng, (total, hkv, d))
    cu = np.concatenate([[0], np.cumsum(n)]).astype(np.int32)
    scale = float(rng.uniform(0.5, 1.5)) / math.sqrt(d)
    if not with_kv:
        # The turn's K/V is already in the pool: write it there with the oracle first.
        tok_s = np.repeat(np.arange(S), n).astype(np.int32)
        tok_p = (c[tok_s] + np.arange(total) - cu[tok_s]).astype(np.int32)
        oracle_lib.append(pool, 16, d, layer, tables, tok_s, tok_p, kn, vn)
    ref, ref_pool = oracle_lib.prefill(pool, 16, d, layer, q, kn if with_kv else None, vn if with_kv else None,
                                       cu, c, tables, scale, pool_out=True)
    return dict(what=what, d=d, hq=hq, layer=layer, mode=mode, with_kv=with_kv, n=n, c=c, cu=cu,
                max_new=max_new, pool=pool, tables=tables, q=q, kn=kn, vn=vn, scale=scale, ref=ref,
                ref_pool=ref_pool)


@pytest.mark.parametrize("seed", range(48))
def test_prefill_random(kv, oracle_lib, seed):
    _check_prefill(kv, prefill_inputs(oracle_lib, seed))


@pytest.mark.parametrize("seed", range(8))
def test_prefill_random_many_kv_heads(kv, oracle_lib, seed):
    _check_prefill(kv, prefill_inputs(oracle_lib, seed, wide=True))


def _check_prefill(kv, x):
    what, d, hq, layer, mode, with_kv, n, c, cu, tables, kn, vn = (
        x[k] for k in ("what", "d", "hq", "layer", "mode", "with_kv", "n", "c", "cu", "tables", "kn", "vn"))
    total = int(n.sum())
    dp = DevicePool(kv, x["pool"], d)
    host = mode != "device-lengths"
    ws = torch.full((kv.PREFILL_WORKSPACE_BYTES,), 0xA5, dtype=torch.uint8, device="cuda") \
        if mode.endswith("counters") else None
    out = torch.full((total, hq, d), float("nan"), dtype=torch.bfloat16, device="cuda")
    kv.paged_attn_prefill(dp.pool, layer, bf16_dev(x["q"]), i32_dev(cu), i32_dev(c), x["max_new"],
                          i32_dev(tables), x["scale"], out, bf16_dev(kn) if with_kv else None,
                          bf16_dev(vn) if with_kv else None,
                          lens_host=np.stack([n, c], 1).astype(np.int32) if host else None, workspace=ws)
    assert_attn_close(out, x["ref"], what)
    assert np.array_equal(dp.host(), x["ref_pool"]), "%s: pool differs from the oracle's" % what
    assert kv.ls_device_errors() == 0


@pytest.mark.parametrize("seed", range(24))
def test_block_copy_random(kv, oracle_lib, seed):
    """Stash of random ids, then a restore into other random ids (whole, or by
    layer ranges), from device staging or pinned host staging through a ring
    of a random size; byte for byte against the oracle."""
    rng = np.random.default_rng(9900 + seed)
    d = int(rng.choice([64, 128]))
    hkv = int(rng.choice([1, 2, 4, 8]))
    nl = int(rng.integers(1, 7))
    nb = int(rng.integers(1, 300))
    n = int(rng.integers(0, nb + 1))
    on_host = bool(rng.random() < 0.5)
    by_layers = bool(rng.random() < 0.4)
    what = "copy seed %d: %d of %d blocks, layers %d, Hkv %d, D %d, host %s, by layers %s" % (
        seed, n, nb, nl, hkv, d, on_host, by_layers)
    log(what)
    pool = W.normal_bf16(rng, (nl, nb, 2, hkv, 16 * d))
    ids = rng.permutation(nb)[:n].astype(np.int32)
    ids2 = rng.permutation(nb)[:n].astype(np.int32)
    fresh = W.normal_bf16(rng, (n, nl, 2, hkv, 16 * d))
    layer_bytes = 2 * hkv * 16 * d * 2
    cuts = np.unique(np.concatenate([[0, nl], rng.integers(0, nl + 1, size=2)])) if by_layers else np.array([0, nl])
    ring = ring_back = None
    if on_host:
        # A stash moves whole blocks: its ring holds one to four of them.  A
        # restore by layer ranges needs room for the widest range of one block.
        block = layer_bytes * nl
        ring = torch.empty(block + int(rng.integers(0, 3 * block)), dtype=torch.uint8, device="cuda")
        least = layer_bytes * int(np.diff(cuts).max())
        ring_back = torch.empty(least + int(rng.integers(0, 3 * least)), dtype=torch.uint8, device="cuda")
    dp = DevicePool(kv, pool, d)
    shape = (n, nl, 2, hkv, 16 * d)
    if on_host:
        st = torch.empty(shape, dtype=torch.int16, pin_memory=True)
    else:
        st = torch.empty(shape, dtype=torch.int16, device="cuda")
    kv.kv_blocks_stash(dp.pool, i32_dev(ids), st, block_ids_host=ids, ring=ring)
    torch.cuda.synchronize()
    got = st.numpy().view(np.uint16) if on_host else host_bits(st)
    assert np.array_equal(got.reshape(shape), oracle_lib.stash(pool, 16, d, ids)), "%s: stash" % what
    st.copy_(torch.from_numpy(fresh.view(np.int16)))
    if by_layers:
        for lb, le in zip(cuts[:-1], cuts[1:]):
            kv.kv_blocks_restore_layers(dp.pool, int(lb), int(le - lb), i32_dev(ids2), st, block_ids_host=ids2,
                                        ring=ring_back)
    else:
        kv.kv_blocks_restore(dp.pool, i32_dev(ids2), st, block_ids_host=ids2, ring=ring_back)
    assert np.array_equal(dp.host(), oracle_lib.restore(pool.copy(), 16, d, ids2, fresh)), "%s: restore" % what
    assert kv.ls_device_errors() == 0
