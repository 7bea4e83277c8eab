"""Brute-force reference of the KV manager policy (LiveServe §5.1, §5.2, §6).

TEST INFRASTRUCTURE ONLY.  Only ``tests/`` and the benchmark's baseline leg
may import this module.  It shares no code with the library's C++ manager:
every decision is recomputed from scratch with plain Python containers — the
eviction order is a sort of all eligible sessions on every call (the
"tail scanning" the paper's indexed heap replaces, §6 and the eviction-index
overhead table of §7), and the allocators take ``min`` of a set.

Rules, in the paper's terms:

* next-use estimate (§5.1): T_next = T_play + T_reply.  T_play is the remaining
  playback horizon, or unfinished tokens x seconds per token when the monitor
  gives none (the progress-counter fallback); T_reply is a per-session moving
  average of observed reply intervals (weight ``alpha`` on the newest), or the
  workload prior before the first observation;
* eviction (§5.1): only idle sessions with resident blocks are candidates
  (running ones are pinned; speech/barge-in sessions and warm sessions after a
  preload are protected).  Candidates are taken by decreasing T_next (ties:
  smaller id), and each gives up resident blocks from its last position down
  (suffix first) until enough blocks are free;
* preload (§5.2): speech start protects the session.  Its offloaded blocks are
  preloaded only if blocks x bytes / bandwidth <= the time available and the
  missing device blocks can be freed from candidates; restores go prefix
  first; completion makes the KV warm (protected) for ``warm_ttl`` seconds,
  releasing the oldest warm protections while the warm total exceeds the cap;
  a cancel returns loading blocks to the host copy.
"""
from __future__ import annotations

RESIDENT, OFFLOADED, LOADING = 0, 1, 2
RUNNING, IMMEDIATE, WARM, EVICTABLE = 0x1, 0x2, 0x4, 0x8


class RefKVManager:
    def __init__(self, num_device_blocks, num_host_slots, max_sessions, reply_prior_s=3.0,
                 reply_ema_alpha=0.5, seconds_per_token=0.04, warm_ttl_s=5.0, warm_cap_blocks=1 << 40):
        self.free_dev = set(range(num_device_blocks))
        self.free_host = set(range(num_host_slots))
        self.max_sessions = max_sessions
        self.prior = reply_prior_s
        self.alpha = reply_ema_alpha
        self.spt = seconds_per_token
        self.ttl = warm_ttl_s
        self.cap = warm_cap_blocks
        self.sessions = {}
        self.warm_seq = 0

    # ---- helpers
    def t_next(self, i):
        s = self.sessions[i]
        play = s["t_play"] if s["t_play"] >= 0 else s["tokens"] * self.spt
        reply = s["reply"] if s["reply"] is not None else self.prior
        return play + reply

    def _resident(self, i):
        return sum(1 for e in self.sessions[i]["table"] if e[2] == RESIDENT)

    def _eligible(self, i):
        s = self.sessions[i]
        return not (s["running"] or s["immediate"] or s["warm"]) and self._resident(i) > 0

    def _evictable(self):
        return sum(self._resident(i) for i in self.sessions if self._eligible(i))

    def _warm_blocks(self):
        return sum(len(s["table"]) for s in self.sessions.values() if s["warm"])

    def _take(self, pool):
        v = min(pool)
        pool.remove(v)
        return v

    # ---- calls
    def add_session(self, i):
        if not 0 <= i < self.max_sessions or i in self.sessions:
            raise ValueError("bad session")
        self.sessions[i] = dict(table=[], running=False, immediate=False, warm=False, warm_since=0.0,
                                warm_order=0, t_play=-1.0, tokens=0, reply=None)

    def remove_session(self, i):
        for dev, host, _ in self.sessions.pop(i)["table"]:
            if dev >= 0:
                self.free_dev.add(dev)
            if host >= 0:
                self.free_host.add(host)

    def append_blocks(self, i, n):
        if len(self.free_dev) < n:
            raise MemoryError("not enough free blocks")
        ids = [self._take(self.free_dev) for _ in range(n)]
        self.sessions[i]["table"] += [[b, -1, RESIDENT] for b in ids]
        return ids

    def set_running(self, i, running):
        s = self.sessions[i]
        s["running"] = bool(running)
        if running:
            s["immediate"] = False
            s["warm"] = False

    def set_playback(self, i, t_play, tokens=0):
        s = self.sessions[i]
        s["t_play"] = t_play if t_play >= 0 else -1.0
        s["tokens"] = tokens

    def observe_reply(self, i, interval):
        s = self.sessions[i]
        s["reply"] = interval if s["reply"] is None else self.alpha * interval + (1 - self.alpha) * s["reply"]

    def speech_start(self, i):
        self.sessions[i]["immediate"] = True

    def evict(self, need):
        moves = []
        while len(moves) < need and self.free_host:
            cands = [i for i in self.sessions if self._eligible(i)]
            if not cands:
                break
            i = min(cands, key=lambda j: (-self.t_next(j), j))
            table = self.sessions[i]["table"]
            for pos in range(len(table) - 1, -1, -1):
                if len(moves) == need or not self.free_host:
                    break
                dev, _, state = table[pos]
                if state != RESIDENT:
                    continue
                host = self._take(self.free_host)
                moves.append((i, pos, dev, host))
                self.free_dev.add(dev)
                table[pos] = [-1, host, OFFLOADED]
        return moves

    def preload(self, i, time_available, bytes_per_block, bandwidth):
        """(admitted, restores, evictions)."""
        s = self.sessions[i]
        if any(e[2] == LOADING for e in s["table"]):
            raise ValueError("preload in flight")
        s["immediate"] = True
        off = [pos for pos, e in enumerate(s["table"]) if e[2] == OFFLOADED]
        if not off:
            return True, [], []
        if len(off) * bytes_per_block / bandwidth > time_available:
            return False, [], []
        short = max(0, len(off) - len(self.free_dev))
        if short > self._evictable() or short > len(self.free_host):
            return False, [], []
        evictions = self.evict(short) if short else []
        restores = []
        for pos in off:                              # prefix first
            host = s["table"][pos][1]
            dev = self._take(self.free_dev)
            s["table"][pos] = [dev, host, LOADING]
            restores.append((i, pos, dev, host))
        return True, restores, evictions

    def load_sync(self, i):
        ok, r, e = self.preload(i, float("inf"), 0.0, 1.0)
        if not ok:
            raise MemoryError("not enough HBM")
        return r, e

    def preload_done(self, i, now):
        s = self.sessions[i]
        for e in s["table"]:
            if e[2] == LOADING:
                self.free_host.add(e[1])
                e[1] = -1
                e[2] = RESIDENT
        if not s["running"]:
            s["immediate"] = False
            s["warm"] = True
            s["warm_since"] = now
            self.warm_seq += 1
            s["warm_order"] = self.warm_seq
        while self._warm_blocks() > self.cap:
            older = [j for j, t in self.sessions.items() if t["warm"] and j != i]
            if not older:
                break
            self.sessions[min(older, key=lambda j: self.sessions[j]["warm_order"])]["warm"] = False

    def preload_cancel(self, i):
        for e in self.sessions[i]["table"]:
            if e[2] == LOADING:
                self.free_dev.add(e[0])
                e[0] = -1
                e[2] = OFFLOADED

    def tick(self, now):
        for s in self.sessions.values():
            if s["warm"] and now - s["warm_since"] >= self.ttl:
                s["warm"] = False

    def session_info(self, i):
        s = self.sessions[i]
        flags = ((RUNNING if s["running"] else 0) | (IMMEDIATE if s["immediate"] else 0) |
                 (WARM if s["warm"] else 0) | (EVICTABLE if self._eligible(i) else 0))
        return self.t_next(i), flags, len(s["table"])

    def table(self, i):
        t = self.sessions[i]["table"]
        return [e[0] for e in t], [e[1] for e in t], [e[2] for e in t]

    def counts(self):
        return dict(free_device_blocks=len(self.free_dev), free_host_slots=len(self.free_host),
                    evictable_blocks=self._evictable(), warm_blocks=self._warm_blocks())
