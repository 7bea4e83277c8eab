"""Seeded synthetic multi-turn speech sessions for the paged-KV hot path.

Inputs only: this module draws random numbers, lengths and block-id
permutations and lays them out in the documented pool layout.  It computes no
attention, no softmax and no copy — both the GPU library and the CPU oracle are
fed from here, and neither shares anything else.

The paper measures on ShareGPT conversations, interactive multi-turn traces,
StreamingBench and BurstGPT arrivals (§7.1); none of those is available, so the
five workloads below stand in for them with the shapes of its multi-turn speech
sessions (thinker/talker decode, next-turn prefill over reused history,
block restore during user speech).

Pool layout: ``pool[layer][block][kv][head][tile]`` (bf16 bit patterns, uint16),
K tile chunk-major ``[D/W][B][W]`` with ``W = min(8, D)`` (element (t, d) at
``((d//W)*B + t)*W + d%W``), V tile dim-major ``[D][B]``.  Every slot that no
session references (unused blocks, the tail of a session's last block, slots
reserved for tokens not yet appended) holds the bf16 quiet NaN 0x7FC0, so a
kernel that lets a masked slot leak into a result produces NaN.

Draw order per workload (one ``numpy.random.Generator(PCG64(seed))``):
lengths -> block-id permutation -> q -> pool (K and V of every slot) -> new K/V.
Values are N(0, 1) drawn in float32 and rounded to bf16 (round to nearest even).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional

import numpy as np

BLOCK = 16
NAN_BF16 = np.uint16(0x7FC0)
SEEDS = {"tiny": 26061, "thinker": 26062, "prefill": 26063, "talker": 26064, "restore": 26065}


def to_bf16(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns, round to nearest even (finite inputs)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    return ((u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)).astype(
        np.uint16)


def from_bf16(b: np.ndarray) -> np.ndarray:
    """bf16 bit patterns -> float32 (exact)."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def normal_bf16(rng: np.random.Generator, shape, chunk: int = 1 << 24) -> np.ndarray:
    """N(0,1) float32 draws rounded to bf16, generated in fixed-size chunks."""
    n = int(np.prod(shape))
    out = np.empty(n, dtype=np.uint16)
    for lo in range(0, n, chunk):
        hi = min(n, lo + chunk)
        out[lo:hi] = to_bf16(rng.standard_normal(hi - lo, dtype=np.float32))
    return out.reshape(shape)


@dataclass
class Pool:
    """Host image of the paged KV pool (bf16 bits) plus its geometry."""
    data: np.ndarray            # uint16 [layers][blocks][2][kv_heads][B*D]
    num_kv_heads: int
    head_dim: int
    block_size: int = BLOCK

    @property
    def num_layers(self) -> int:
        return self.data.shape[0]

    @property
    def num_blocks(self) -> int:
        return self.data.shape[1]

    @property
    def nbytes(self) -> int:
        return self.data.nbytes


@dataclass
class DecodeCase:
    name: str
    seed: int
    pool: Pool
    num_q_heads: int
    block_tables: np.ndarray     # int32 [S][max_blocks]
    context_lens: np.ndarray     # int32 [S] (steps > 1: lens at step 0)
    q: np.ndarray                # uint16 [steps][S][Hq][D]
    k_new: Optional[np.ndarray]  # uint16 [steps][S][Hkv][D] or None (no append)
    v_new: Optional[np.ndarray]
    scale: float
    steps: int = 1
    notes: dict = field(default_factory=dict)

    @property
    def num_sessions(self) -> int:
        return self.block_tables.shape[0]

    def lens_at(self, step: int) -> np.ndarray:
        """Tokens already in the pool before decode step ``step``."""
        return (self.context_lens + step).astype(np.int32)


@dataclass
class PrefillCase:
    name: str
    seed: int
    pool: Pool
    num_q_heads: int
    block_tables: np.ndarray     # int32 [S][max_blocks]
    new_lens: np.ndarray         # int32 [S]  n_s (tokens of the new turn)
    reused_lens: np.ndarray      # int32 [S]  c_s (reused multi-turn context)
    q: np.ndarray                # uint16 [sum n][Hq][D]
    k_new: np.ndarray            # uint16 [sum n][Hkv][D]
    v_new: np.ndarray
    scale: float

    @property
    def num_sessions(self) -> int:
        return self.block_tables.shape[0]

    @property
    def cu_new_lens(self) -> np.ndarray:
        return np.concatenate([[0], np.cumsum(self.new_lens)]).astype(np.int32)


@dataclass
class RestoreCase:
    name: str
    seed: int
    num_layers: int
    num_kv_heads: int
    head_dim: int
    num_blocks: int
    stash_ids: np.ndarray        # int32 [n]  slot set A (stashed)
    restore_ids: np.ndarray      # int32 [n]  slot permutation B (restored into)
    block_size: int = BLOCK

    @property
    def slab_bytes(self) -> int:
        """Bytes of one (layer, block) slab: K and V of every KV head."""
        return 2 * self.num_kv_heads * self.block_size * self.head_dim * 2

    @property
    def payload_bytes(self) -> int:
        return len(self.stash_ids) * self.num_layers * self.slab_bytes


def _blocks_for(tokens: np.ndarray) -> np.ndarray:
    return (tokens + BLOCK - 1) // BLOCK


def _poison(pool: np.ndarray, head_dim: int, tables: np.ndarray, valid_tokens: np.ndarray,
            referenced_blocks: int):
    """NaN every slot that holds no valid token: unreferenced blocks entirely, and
    slots at or past ``valid_tokens[s]`` inside session s's table."""
    nl, nb, _, hkv, tile = pool.shape
    used = np.zeros(nb, dtype=bool)
    for s in range(tables.shape[0]):
        nblk = int((tables[s] >= 0).sum())
        used[tables[s, :nblk]] = True
    unused = np.nonzero(~used)[0]
    pool[:, unused] = NAN_BF16
    w = min(8, head_dim)
    k_view = pool[:, :, 0].reshape(nl, nb, hkv, head_dim // w, BLOCK, w)
    v_view = pool[:, :, 1].reshape(nl, nb, hkv, head_dim, BLOCK)
    for s in range(tables.shape[0]):
        nblk = int((tables[s] >= 0).sum())
        v = int(valid_tokens[s])
        for j in range(v // BLOCK, nblk):
            b = tables[s, j]
            first = max(0, v - j * BLOCK)
            k_view[:, b, :, :, first:, :] = NAN_BF16
            v_view[:, b, :, :, first:] = NAN_BF16
    assert referenced_blocks == int(used.sum())


def _tables(perm: np.ndarray, blocks_per_session: np.ndarray, width: int) -> np.ndarray:
    tables = np.full((len(blocks_per_session), width), -1, dtype=np.int32)
    pos = 0
    for s, nblk in enumerate(blocks_per_session):
        tables[s, :nblk] = perm[pos:pos + nblk]
        pos += nblk
    return tables


def _decode_case(name, seed, rng, lens, hq, hkv, d, num_blocks, steps, append,
                 pool_factor=None):
    s = len(lens)
    final_tokens = lens + (steps if append else 0)
    need_final = _blocks_for(final_tokens)
    need_now = _blocks_for(lens)
    if num_blocks is None:
        num_blocks = int(np.ceil(pool_factor * need_final.sum()))
    perm = rng.permutation(num_blocks).astype(np.int32)
    width = int(need_final.max())
    tables = _tables(perm, need_now, width)
    # Blocks for tokens appended later come off a shuffled free list, in the order
    # the steps need them (a fresh block whenever a token starts a new block).
    free = list(perm[int(need_now.sum()):][::-1])
    for t in range(steps if append else 0):
        for si in range(s):
            pos = int(lens[si]) + t
            if pos % BLOCK == 0:
                tables[si, pos // BLOCK] = free.pop()
    q = normal_bf16(rng, (steps, s, hq, d))
    pool = normal_bf16(rng, (1, num_blocks, 2, hkv, BLOCK * d))
    k_new = normal_bf16(rng, (steps, s, hkv, d)) if append else None
    v_new = normal_bf16(rng, (steps, s, hkv, d)) if append else None
    _poison(pool, d, tables, lens, int(need_final.sum()))
    return DecodeCase(name=name, seed=seed, pool=Pool(pool, hkv, d), num_q_heads=hq,
                      block_tables=tables, context_lens=lens.astype(np.int32), q=q, k_new=k_new,
                      v_new=v_new, scale=1.0 / np.sqrt(d), steps=steps)


def tiny_decode(seed: int = SEEDS["tiny"], append: bool = False) -> DecodeCase:
    """4 sessions, L ~ U[64, 512], 8/2 heads (GQA), D = 64, 256-block pool with
    randomly permuted block ids, one decode token per session."""
    rng = np.random.Generator(np.random.PCG64(seed))
    lens = rng.integers(64, 512, size=4, endpoint=True).astype(np.int64)
    return _decode_case("tiny_decode", seed, rng, lens, 8, 2, 64, 256, 1, append)


def _thinker_lengths(rng: np.random.Generator, num_sessions: int, sigma: float) -> np.ndarray:
    z = rng.standard_normal(num_sessions)
    return np.clip(np.round(np.exp(np.log(4096.0) + sigma * z)), 512, 16384).astype(np.int64)


def _talker_lengths(rng: np.random.Generator, num_sessions: int) -> np.ndarray:
    return rng.integers(512, 4096, size=num_sessions, endpoint=True).astype(np.int64)


def thinker_lengths(seed: int = SEEDS["thinker"], num_sessions: int = 64, sigma: float = 1.0) -> np.ndarray:
    """The context lengths of :func:`thinker_decode` alone (its first draws)."""
    return _thinker_lengths(np.random.Generator(np.random.PCG64(seed)), num_sessions, sigma)


def talker_lengths(seed: int = SEEDS["talker"], num_sessions: int = 256) -> np.ndarray:
    """The starting context lengths of :func:`talker_decode` alone (its first draws)."""
    return _talker_lengths(np.random.Generator(np.random.PCG64(seed)), num_sessions)


def thinker_decode(seed: int = SEEDS["thinker"], num_sessions: int = 64, sigma: float = 1.0,
                   append: bool = False) -> DecodeCase:
    """64 sessions, L = clip(round(exp(ln 4096 + sigma * N(0,1))), 512, 16384),
    32/4 heads, D = 128, pool 1.25x the blocks in use, one query token each."""
    rng = np.random.Generator(np.random.PCG64(seed))
    lens = _thinker_lengths(rng, num_sessions, sigma)
    case = _decode_case("thinker_decode", seed, rng, lens, 32, 4, 128, None, 1, append,
                        pool_factor=1.25)
    case.notes["sigma"] = sigma
    return case


def talker_decode(seed: int = SEEDS["talker"], num_sessions: int = 256, steps: int = 32
                  ) -> DecodeCase:
    """256 sessions, L0 ~ U[512, 4096], 16/2 heads, D = 128, ``steps`` consecutive
    decode steps each appending one fresh token per session."""
    rng = np.random.Generator(np.random.PCG64(seed))
    lens = _talker_lengths(rng, num_sessions)
    return _decode_case("talker_decode", seed, rng, lens, 16, 2, 128, None, steps, True,
                        pool_factor=1.25)


def next_turn_prefill(seed: int = SEEDS["prefill"], num_sessions: int = 32,
                      new_range=(256, 2048), ctx_range=(2048, 32768), hq: int = 32,
                      hkv: int = 4, d: int = 128) -> PrefillCase:
    """32 sessions, a new user turn of n ~ U[256, 2048] tokens attending causally to
    c ~ U[2048, 32768] reused context tokens in paged blocks, 32/4 heads, D = 128."""
    rng = np.random.Generator(np.random.PCG64(seed))
    n = rng.integers(new_range[0], new_range[1], size=num_sessions, endpoint=True).astype(np.int64)
    c = rng.integers(ctx_range[0], ctx_range[1], size=num_sessions, endpoint=True).astype(np.int64)
    need = _blocks_for(c + n)
    num_blocks = int(np.ceil(1.25 * need.sum()))
    perm = rng.permutation(num_blocks).astype(np.int32)
    tables = _tables(perm, need, int(need.max()))
    total = int(n.sum())
    q = normal_bf16(rng, (total, hq, d))
    pool = normal_bf16(rng, (1, num_blocks, 2, hkv, BLOCK * d))
    k_new = normal_bf16(rng, (total, hkv, d))
    v_new = normal_bf16(rng, (total, hkv, d))
    _poison(pool, d, tables, c, int(need.sum()))
    return PrefillCase(name="next_turn_prefill", seed=seed, pool=Pool(pool, hkv, d),
                       num_q_heads=hq, block_tables=tables, new_lens=n.astype(np.int32),
                       reused_lens=c.astype(np.int32), q=q, k_new=k_new, v_new=v_new,
                       scale=1.0 / np.sqrt(d))


def restore_case(seed: int = SEEDS["restore"], num_sessions: int = 128, tokens: int = 8192,
                 num_layers: int = 48, hkv: int = 4, d: int = 128, spare_factor: float = 1.0
                 ) -> RestoreCase:
    """Stash then restore ``num_layers`` x ``hkv`` x ``d`` bf16 KV for ``num_sessions``
    sessions of ``tokens`` tokens: slot set A is a seeded random subset of the pool,
    B a fresh seeded permutation (the slots the preload lands in)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    n = num_sessions * ((tokens + BLOCK - 1) // BLOCK)
    num_blocks = int(np.ceil(spare_factor * n))
    a = rng.permutation(num_blocks)[:n].astype(np.int32)
    b = rng.permutation(num_blocks)[:n].astype(np.int32)
    return RestoreCase(name="kv_restore", seed=seed, num_layers=num_layers, num_kv_heads=hkv,
                       head_dim=d, num_blocks=num_blocks, stash_ids=a, restore_ids=b)


@dataclass
class ManagerTrace:
    """Seeded event sequence for the KV manager (the policy of §5.1, §5.2).

    ``context_blocks[s]``: blocks of session s's reused multi-turn context at the
    start.  ``events``: tuples
      ("play", s, t_play)       monitor update: seconds of audio still to play
      ("pressure", n)           running requests need n more device blocks
      ("turn", s, t_avail, new_blocks, reply_s, t_play)
                                speech start with t_avail seconds before the LLM
                                stage runs, then the turn appends new_blocks; the
                                observed reply interval and the new reply's horizon.
    """
    name: str
    seed: int
    num_device_blocks: int
    num_host_slots: int
    context_blocks: np.ndarray
    events: list
    bytes_per_block: float
    bandwidth: float


def manager_trace(seed: int = 26066, num_sessions: int = 4096, num_events: int = 20000,
                  device_fraction: float = 0.5) -> ManagerTrace:
    """Multi-turn speech sessions against a pool that holds about half of their
    KV: contexts lognormal (median 64 blocks = 1024 tokens, sigma 1, clipped to
    [4, 1024] blocks), playback horizons U[0, 30] s, reply intervals U[0.5, 8] s,
    speech-to-LLM-stage windows U[0.1, 2] s, turns of U[1, 16] new blocks.
    Blocks are the thinker's all-layer slab (48 layers x 4 KV heads x 128 dims x
    16 tokens x K,V in bf16 = 1.5 MiB); host link 50 GB/s."""
    rng = np.random.default_rng(seed)
    ctx = np.clip(np.round(np.exp(np.log(64) + rng.standard_normal(num_sessions))), 4, 1024).astype(np.int64)
    total = int(ctx.sum())
    kinds = rng.choice(3, size=num_events, p=[0.6, 0.2, 0.2])
    events = []
    for k in kinds:
        if k == 0:
            events.append(("play", int(rng.integers(num_sessions)), float(rng.uniform(0, 30))))
        elif k == 1:
            events.append(("pressure", int(rng.integers(8, 65))))
        else:
            events.append(("turn", int(rng.integers(num_sessions)), float(rng.uniform(0.1, 2.0)),
                           int(rng.integers(1, 17)), float(rng.uniform(0.5, 8.0)), float(rng.uniform(0, 30))))
    return ManagerTrace("kv manager trace", seed, int(total * device_fraction), 2 * total, ctx, events,
                        48 * 4 * 128 * 16 * 2 * 2.0, 50e9)


@dataclass
class PipelineTurn:
    """Next-turn prefill whose reused context was offloaded (every layer)."""
    name: str
    seed: int
    num_layers: int
    num_kv_heads: int
    num_q_heads: int
    head_dim: int
    num_blocks: int
    new_lens: np.ndarray
    reused_lens: np.ndarray
    block_tables: np.ndarray
    context_block_ids: np.ndarray   # blocks holding reused context, session after session


def pipeline_turn(seed: int = 26067, num_sessions: int = 4, num_layers: int = 48) -> PipelineTurn:
    """Sessions of the thinker's geometry (48 layers, 32/4 heads, D = 128) come
    back for a new turn of n ~ U[256, 1024] tokens over c ~ U[8192, 16384]
    reused tokens that sit in host DRAM (the reload before prefill of §5.2 and
    §7); block ids are a permutation of a pool 1.1x the blocks needed."""
    rng = np.random.default_rng(seed)
    n = rng.integers(256, 1025, size=num_sessions).astype(np.int32)
    c = rng.integers(8192, 16385, size=num_sessions).astype(np.int32)
    need = _blocks_for(c.astype(np.int64) + n)
    nb = int(need.sum() * 1.1) + 1
    perm = rng.permutation(nb).astype(np.int32)
    tables = _tables(perm, need, int(need.max()))
    ctx = np.concatenate([tables[s, :(int(c[s]) + BLOCK - 1) // BLOCK] for s in range(num_sessions)])
    return PipelineTurn("layer-pipelined reload + next-turn prefill", seed, num_layers, 4, 32, 128, nb, n, c,
                        tables, ctx.astype(np.int32))
