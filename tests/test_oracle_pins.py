"""Pins for the CPU oracle (no GPU).

The oracle is checked against things other than itself: a library attention
routine (torch SDPA in float64) on dense logical K/V, hand-derived golden
cases, closed forms (one key, uniform keys, q = 0), invariants (physical
block permutation, affine V, GQA = MHA with repeated KV heads, chunked
prefill) and byte-level definitions of stash/restore.  Each is chosen so that
a plausible mistake (dropped scale, softmax over the wrong axis, K/V swapped,
wrong GQA head mapping, off-by-one causal edge, wrong block-table index,
transposed V tile) fails at least one of them.
"""
import json
import math
import os

import numpy as np
import pytest
import torch

from paper_2606_22983_amd import workloads as W

B = W.BLOCK
GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "hand_cases.json")


# ----------------------------------------------------------------------------
# test-side paged placement, written from the documented layout:
#   pool[layer][block][kv][head][tile]; K tile chunk-major [dim/8][token][8 dims],
#   V tile dim-major [dim][token]
# ----------------------------------------------------------------------------
def make_paged(rng, lens, hkv, d, spare=3, nl=1, layer=0, k=None, v=None):
    """Place logical K/V [S][L][Hkv][D] (bf16 bits) into a shuffled paged pool."""
    lens = list(lens)
    need = [(n + B - 1) // B for n in lens]
    nb = sum(need) + spare
    perm = rng.permutation(nb).astype(np.int32)
    tables = np.full((len(lens), max(need)), -1, dtype=np.int32)
    pool = np.full((nl, nb, 2, hkv, B * d), W.NAN_BF16, dtype=np.uint16)
    pos = 0
    ks, vs = [], []
    for s, n in enumerate(lens):
        tables[s, :need[s]] = perm[pos:pos + need[s]]
        pos += need[s]
        ks_ = W.normal_bf16(rng, (n, hkv, d)) if k is None else k[s]
        vs_ = W.normal_bf16(rng, (n, hkv, d)) if v is None else v[s]
        ks.append(ks_)
        vs.append(vs_)
        for t in range(n):
            b = tables[s, t // B]
            for g in range(hkv):
                w = min(8, d)   # K tile chunk-major [d/w][B][w]
                pool[layer, b, 0, g].reshape(d // w, B, w)[:, t % B, :] = ks_[t, g].reshape(d // w, w)
                pool[layer, b, 1, g].reshape(d, B)[:, t % B] = vs_[t, g]
    return pool, tables, ks, vs


def sdpa(q, k, v, scale, mask=None):
    """torch SDPA in float64: q [Hq][Lq][D], k/v [Hkv][Lk][D] (GQA by repetition)."""
    hq, hkv = q.shape[0], k.shape[0]
    kk = torch.from_numpy(k).double().repeat_interleave(hq // hkv, dim=0)
    vv = torch.from_numpy(v).double().repeat_interleave(hq // hkv, dim=0)
    qq = torch.from_numpy(q).double()
    m = None if mask is None else torch.from_numpy(mask)
    out = torch.nn.functional.scaled_dot_product_attention(qq[None], kk[None], vv[None],
                                                           attn_mask=m, scale=scale)
    return out[0].numpy()


def f32(b):
    return W.from_bf16(b).astype(np.float64)


# ----------------------------------------------------------------------------
# reduction to a library routine
# ----------------------------------------------------------------------------
@pytest.mark.parametrize("L", [1, 2, 15, 16, 17, 31, 32, 33, 255, 511, 512])
@pytest.mark.parametrize("d,hq,hkv", [(64, 8, 2), (128, 8, 1), (128, 8, 8), (128, 32, 4)])
def test_decode_equals_sdpa(oracle_lib, L, d, hq, hkv):
    rng = np.random.default_rng(1000 + L + d + hq)
    lens = [L, max(1, L // 2), L + 3]
    pool, tables, ks, vs = make_paged(rng, lens, hkv, d)
    q = W.normal_bf16(rng, (len(lens), hq, d))
    scale = 1.0 / math.sqrt(d)
    out = oracle_lib.decode(pool, B, d, 0, q, tables, np.array(lens), scale)
    for s, n in enumerate(lens):
        ref = sdpa(f32(q[s])[:, None, :], f32(ks[s]).transpose(1, 0, 2),
                   f32(vs[s]).transpose(1, 0, 2), scale)[:, 0, :]
        np.testing.assert_allclose(out[s], ref, rtol=1e-10, atol=1e-12)


@pytest.mark.parametrize("c,n", [(0, 1), (0, 17), (0, 40), (5, 1), (16, 16), (37, 29), (200, 3)])
def test_prefill_equals_masked_sdpa(oracle_lib, c, n):
    """c = 0 is textbook causal self-attention; c > 0 uses the bottom-right mask
    (row j sees keys 0..c+j) built explicitly for the library routine."""
    rng = np.random.default_rng(77 + c * 100 + n)
    hq, hkv, d = 8, 2, 64
    ctx_k = W.normal_bf16(rng, (c, hkv, d))
    ctx_v = W.normal_bf16(rng, (c, hkv, d))
    pool, tables, _, _ = make_paged(rng, [c + n], hkv, d, k=[np.concatenate(
        [ctx_k, np.full((n, hkv, d), W.NAN_BF16, np.uint16)])], v=[np.concatenate(
            [ctx_v, np.full((n, hkv, d), W.NAN_BF16, np.uint16)])])
    q = W.normal_bf16(rng, (n, hq, d))
    kn = W.normal_bf16(rng, (n, hkv, d))
    vn = W.normal_bf16(rng, (n, hkv, d))
    scale = 1.0 / math.sqrt(d)
    out = oracle_lib.prefill(pool, B, d, 0, q, kn, vn, [0, n], [c], tables, scale)
    k_all = f32(np.concatenate([ctx_k, kn])).transpose(1, 0, 2)
    v_all = f32(np.concatenate([ctx_v, vn])).transpose(1, 0, 2)
    if c == 0:
        qq = torch.from_numpy(f32(q).transpose(1, 0, 2)).double()
        kk = torch.from_numpy(k_all).double().repeat_interleave(hq // hkv, 0)
        vv = torch.from_numpy(v_all).double().repeat_interleave(hq // hkv, 0)
        ref = torch.nn.functional.scaled_dot_product_attention(
            qq[None], kk[None], vv[None], is_causal=True, scale=scale)[0].numpy()
    else:
        mask = np.arange(c + n)[None, :] <= (c + np.arange(n))[:, None]
        ref = sdpa(f32(q).transpose(1, 0, 2), k_all, v_all, scale, mask)
    np.testing.assert_allclose(out, ref.transpose(1, 0, 2), rtol=1e-10, atol=1e-12)


# ----------------------------------------------------------------------------
# hand-derived golden cases
# ----------------------------------------------------------------------------
def _scale(text):
    return {"ln3/2": math.log(3) / 2, "ln2/4": math.log(2) / 4, "ln2/2": math.log(2) / 2}.get(
        text, None) or float(text)


@pytest.mark.parametrize("case", json.load(open(GOLDEN))["cases"], ids=lambda c: c["name"])
def test_golden_hand_cases(oracle_lib, case):
    d = case["head_dim"]
    k = W.to_bf16(np.array(case["k"], np.float32))[:, None, :]
    v = W.to_bf16(np.array(case["v"], np.float32))[:, None, :]
    q = W.to_bf16(np.array(case["q"], np.float32))[:, None, :]
    assert np.array_equal(W.from_bf16(k)[:, 0], np.array(case["k"], np.float32)), "not bf16-exact"
    rng = np.random.default_rng(5)
    scale = _scale(case["scale"])
    if case["kind"] == "decode":
        L = k.shape[0]
        pool, tables, _, _ = make_paged(rng, [L], 1, d, spare=4, k=[k], v=[v])
        out = oracle_lib.decode(pool, B, d, 0, q, tables, [L], scale)[:, 0, :]
    else:
        c = case["context"]
        n = q.shape[0]
        pad = np.full((n, 1, d), W.NAN_BF16, np.uint16)
        pool, tables, _, _ = make_paged(rng, [c + n], 1, d, spare=4,
                                        k=[np.concatenate([k[:c], pad])],
                                        v=[np.concatenate([v[:c], pad])])
        out = oracle_lib.prefill(pool, B, d, 0, q, k[c:], v[c:], [0, n], [c], tables,
                                 scale)[:, 0, :]
    np.testing.assert_allclose(out, np.array(case["expected"]), rtol=0, atol=1e-12)


# ----------------------------------------------------------------------------
# closed forms
# ----------------------------------------------------------------------------
def test_one_key_returns_v_exactly(oracle_lib):
    rng = np.random.default_rng(11)
    pool, tables, ks, vs = make_paged(rng, [1, 1, 1], 2, 128)
    q = W.normal_bf16(rng, (3, 8, 128))
    out = oracle_lib.decode(pool, B, 128, 0, q, tables, [1, 1, 1], 0.0883883)
    for s in range(3):
        for h in range(8):
            assert np.array_equal(out[s, h], f32(vs[s][0, h // 4]))


@pytest.mark.parametrize("mode", ["equal_keys", "zero_keys", "zero_q"])
def test_uniform_scores_give_mean_of_v(oracle_lib, mode):
    rng = np.random.default_rng(12)
    L, hkv, d = 53, 2, 64
    k = W.normal_bf16(rng, (L, hkv, d))
    if mode == "equal_keys":
        k[:] = k[0]
    elif mode == "zero_keys":
        k[:] = 0
    v = W.normal_bf16(rng, (L, hkv, d))
    pool, tables, _, _ = make_paged(rng, [L], hkv, d, k=[k], v=[v])
    q = W.normal_bf16(rng, (1, 8, d))
    if mode == "zero_q":
        q[:] = 0
    out = oracle_lib.decode(pool, B, d, 0, q, tables, [L], 0.125)
    mean_v = f32(v).mean(axis=0)
    for h in range(8):
        np.testing.assert_allclose(out[0, h], mean_v[h // 4], rtol=1e-12, atol=1e-14)


def test_needle_selects_its_value_at_every_block_position(oracle_lib):
    """A key aligned with q and scaled large dominates the softmax: out -> V at the
    needle.  Sweeping the needle over every slot of every block pins block-table
    indexing and slot order."""
    rng = np.random.default_rng(13)
    L, hkv, d = 5 * B + 3, 1, 64
    q = W.normal_bf16(rng, (1, 1, d))
    needle = W.to_bf16(40.0 * W.from_bf16(q[0, 0]) / np.linalg.norm(W.from_bf16(q[0, 0])))
    for p in list(range(L)):
        k = W.to_bf16(0.05 * W.from_bf16(W.normal_bf16(rng, (L, hkv, d))))
        k[p, 0] = needle
        v = W.normal_bf16(rng, (L, hkv, d))
        pool, tables, _, _ = make_paged(rng, [L], hkv, d, k=[k], v=[v])
        out = oracle_lib.decode(pool, B, d, 0, q, tables, [L], 1.0 / 8.0)
        np.testing.assert_allclose(out[0, 0], f32(v[p, 0]), atol=1e-6)


# ----------------------------------------------------------------------------
# invariants
# ----------------------------------------------------------------------------
def test_block_permutation_invariance(oracle_lib):
    case = W.tiny_decode()
    pool = case.pool.data
    out = oracle_lib.decode(pool, B, 64, 0, case.q[0], case.block_tables, case.context_lens,
                            case.scale)
    rng = np.random.default_rng(14)
    nb = pool.shape[1]
    sigma = rng.permutation(nb)            # block b moves to slot sigma[b]
    moved = np.empty_like(pool)
    moved[:, sigma] = pool
    tables = np.where(case.block_tables >= 0, sigma[np.maximum(case.block_tables, 0)], -1)
    out2 = oracle_lib.decode(moved, B, 64, 0, case.q[0], tables.astype(np.int32),
                             case.context_lens, case.scale)
    assert np.array_equal(out, out2)


def test_affine_values(oracle_lib):
    """V -> 2 V + 1 maps out -> 2 out + 1 (values on a 1/4 grid keep bf16 exact)."""
    rng = np.random.default_rng(15)
    L, hkv, d = 70, 2, 64
    vq = rng.integers(-8, 8, size=(L, hkv, d)).astype(np.float32) / 4
    k = W.normal_bf16(rng, (L, hkv, d))
    p1, t1, _, _ = make_paged(np.random.default_rng(1), [L], hkv, d, k=[k], v=[W.to_bf16(vq)])
    p2, t2, _, _ = make_paged(np.random.default_rng(1), [L], hkv, d, k=[k],
                              v=[W.to_bf16(2 * vq + 1)])
    q = W.normal_bf16(rng, (1, 8, d))
    o1 = oracle_lib.decode(p1, B, d, 0, q, t1, [L], 0.125)
    o2 = oracle_lib.decode(p2, B, d, 0, q, t2, [L], 0.125)
    np.testing.assert_allclose(o2, 2 * o1 + 1, rtol=1e-12, atol=1e-12)


def test_gqa_equals_mha_with_repeated_kv_heads(oracle_lib):
    rng = np.random.default_rng(16)
    L, hkv, g, d = 45, 2, 4, 64
    k = W.normal_bf16(rng, (L, hkv, d))
    v = W.normal_bf16(rng, (L, hkv, d))
    q = W.normal_bf16(rng, (1, hkv * g, d))
    pg, tg, _, _ = make_paged(np.random.default_rng(2), [L], hkv, d, k=[k], v=[v])
    pm, tm, _, _ = make_paged(np.random.default_rng(2), [L], hkv * g, d,
                              k=[np.repeat(k, g, axis=1)], v=[np.repeat(v, g, axis=1)])
    og = oracle_lib.decode(pg, B, d, 0, q, tg, [L], 0.125)
    om = oracle_lib.decode(pm, B, d, 0, q, tm, [L], 0.125)
    assert np.array_equal(og, om)


def test_prefill_chunking_and_decode_equivalence(oracle_lib):
    """prefill(n) == prefill(n1) then prefill(n - n1) with c += n1; prefill with
    n = 1 == decode with append."""
    rng = np.random.default_rng(17)
    c, n, n1, hq, hkv, d = 37, 29, 11, 8, 2, 64
    ctx_k = W.normal_bf16(rng, (c, hkv, d))
    ctx_v = W.normal_bf16(rng, (c, hkv, d))
    pad = np.full((n, hkv, d), W.NAN_BF16, np.uint16)
    pool, tables, _, _ = make_paged(rng, [c + n], hkv, d, k=[np.concatenate([ctx_k, pad])],
                                    v=[np.concatenate([ctx_v, pad])])
    q = W.normal_bf16(rng, (n, hq, d))
    kn = W.normal_bf16(rng, (n, hkv, d))
    vn = W.normal_bf16(rng, (n, hkv, d))
    full = oracle_lib.prefill(pool, B, d, 0, q, kn, vn, [0, n], [c], tables, 0.125)
    a, pool_a = oracle_lib.prefill(pool, B, d, 0, q[:n1], kn[:n1], vn[:n1], [0, n1], [c], tables,
                                   0.125, pool_out=True)
    b = oracle_lib.prefill(pool_a, B, d, 0, q[n1:], kn[n1:], vn[n1:], [0, n - n1], [c + n1],
                           tables, 0.125)
    assert np.array_equal(full, np.concatenate([a, b]))
    one = oracle_lib.prefill(pool, B, d, 0, q[:1], kn[:1], vn[:1], [0, 1], [c], tables, 0.125)
    dec = oracle_lib.decode(pool, B, d, 0, q[:1], tables, [c], 0.125, k_new=kn[:1], v_new=vn[:1])
    assert np.array_equal(one, dec)


def test_masked_slots_never_read(oracle_lib):
    """The generator fills every unreferenced slot with NaN; a finite result shows
    the oracle reads only slots 0..L-1 of each table."""
    case = W.tiny_decode()
    out = oracle_lib.decode(case.pool.data, B, 64, 0, case.q[0], case.block_tables,
                            case.context_lens, case.scale)
    assert np.isfinite(out).all()
    nan_slots = (case.pool.data == W.NAN_BF16).sum()
    assert nan_slots > 0


# ----------------------------------------------------------------------------
# stash / restore: byte definitions (§5 offload, §5.2 preload)
# ----------------------------------------------------------------------------
def _random_pool(rng, nl, nb, hkv, d):
    return rng.integers(0, 1 << 16, size=(nl, nb, 2, hkv, B * d), dtype=np.uint16)


def test_stash_is_block_gather(oracle_lib):
    rng = np.random.default_rng(18)
    pool = _random_pool(rng, 3, 40, 2, 64)
    ids = rng.permutation(40)[:9].astype(np.int32)
    st = oracle_lib.stash(pool, B, 64, ids)
    assert np.array_equal(st, np.take(pool, ids, axis=1).transpose(1, 0, 2, 3, 4))


def test_restore_then_stash_is_identity_and_canaries_hold(oracle_lib):
    rng = np.random.default_rng(19)
    pool = _random_pool(rng, 3, 40, 2, 64)
    ids = rng.permutation(40)[:9].astype(np.int32)
    staging = _random_pool(rng, 9, 3, 2, 64).reshape(9, 3, 2, 2, B * 64)
    before = pool.copy()
    oracle_lib.restore(pool, B, 64, ids, staging)
    assert np.array_equal(oracle_lib.stash(pool, B, 64, ids), staging)
    others = np.setdiff1d(np.arange(40), ids)
    assert np.array_equal(pool[:, others], before[:, others])
    # and stash followed by restore into the same slots leaves the pool unchanged
    st = oracle_lib.stash(pool, B, 64, ids)
    again = pool.copy()
    oracle_lib.restore(again, B, 64, ids, st)
    assert np.array_equal(again, pool)


def test_cancelled_restore_then_synchronous_fallback(oracle_lib):
    """An incomplete preload followed by a synchronous load of the rest leaves the
    pool identical to one full restore (§5.2: preloading affects latency, not
    correctness)."""
    rng = np.random.default_rng(20)
    pool = _random_pool(rng, 2, 50, 2, 64)
    ids = rng.permutation(50)[:20].astype(np.int32)
    staging = _random_pool(rng, 20, 2, 2, 64).reshape(20, 2, 2, 2, B * 64)
    full = pool.copy()
    oracle_lib.restore(full, B, 64, ids, staging)
    part = pool.copy()
    oracle_lib.restore(part, B, 64, ids[:7], staging[:7])
    oracle_lib.restore(part, B, 64, ids[7:], staging[7:])
    assert np.array_equal(part, full)


def test_oracle_rejects_out_of_range(oracle_lib):
    rng = np.random.default_rng(21)
    pool = _random_pool(rng, 1, 10, 1, 64)
    with pytest.raises(ValueError):
        oracle_lib.stash(pool, B, 64, np.array([3, 10], np.int32))
    pool2, tables, _, _ = make_paged(rng, [20], 1, 64)
    q = W.normal_bf16(rng, (1, 1, 64))
    with pytest.raises(ValueError):
        oracle_lib.decode(pool2, B, 64, 0, q, tables, [0], 0.125)
