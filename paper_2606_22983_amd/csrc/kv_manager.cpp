// Host-side KV manager: where each session's multi-turn KV blocks live (HBM
// pool or host DRAM) and which blocks the stash/restore copies move.
//
// It implements the policy side of the paper's hierarchical KV manager:
//   - next-use estimate T_next = T_play + T_reply per session (§5.1, Eq. for
//     the next-use estimate): T_play is the audio still to be played, or,
//     when the monitor gives none, unfinished response tokens times a playback
//     rate (the progress-counter fallback of §5.1); T_reply is a per-session
//     exponential moving average of observed reply intervals, or a workload
//     prior before the first observation;
//   - eviction (§5.1): only idle resident multi-turn KV is eligible (running
//     sessions are pinned; sessions in speech or barge-in, and warmed sessions
//     after a preload, are protected).  Eligible sessions are taken in
//     decreasing T_next, and each gives up its suffix blocks first, until
//     enough blocks are free;
//   - the indexed candidate heap of §6: a binary max-heap over the eligible
//     sessions with each session's heap position kept in its record, so that
//     a change of T_next or of eligibility costs O(log n) and an eviction
//     costs O(log n) per session visited, instead of a scan over all sessions;
//   - speech-triggered preload (§5.2): a preload is admitted only when its
//     transfer time (offloaded bytes / bandwidth) fits in the time left before
//     the LLM stage runs and enough HBM can be freed from later-use idle KV;
//     restores go prefix first, so a cancelled preload leaves a usable prefix;
//     a finished preload keeps its KV protected for a bounded time, with the
//     total protected amount capped (oldest protection released first); a
//     cancelled or skipped preload falls back to a synchronous load.
//
// Device block ids and host slots are handed out lowest first, so the blocks
// of one eviction or preload tend to form runs that one stash/restore call
// each can move.  Everything here is host code and single-threaded per
// manager; the library's kernels are not called from here.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <functional>
#include <limits>
#include <new>
#include <queue>
#include <vector>

#include "liveserve_kv.h"

namespace ls {
void set_last_error(const char *fmt, ...);
}

namespace {

enum EntryState : int8_t { kResident = LS_KV_RESIDENT, kOffloaded = LS_KV_OFFLOADED, kLoading = LS_KV_LOADING };

struct Entry {
    int32_t dev;       // device block id, or -1
    int32_t host;      // host slot, or -1
    EntryState state;
};

struct Session {
    bool present = false;
    bool running = false;        // pinned by a running request
    bool immediate = false;      // speech start / barge-in: protected
    bool warm = false;           // protected after a completed preload
    double warm_since = 0.0;
    uint32_t warm_epoch = 0;     // identifies the current protection in the FIFO
    double t_play = -1.0;        // audio still to be played (s), < 0: unknown
    int64_t unfinished_tokens = 0;
    bool has_reply = false;
    double reply_avg = 0.0;
    std::vector<Entry> table;    // by block position
    int32_t resident = 0;        // entries in state kResident
    int32_t loading = 0;         // entries in state kLoading
    int32_t heap_pos = -1;       // position in the candidate heap, -1 if absent
};

// Lowest-first id allocator over [0, n).
class IdPool {
public:
    explicit IdPool(int64_t n) : n_(n) {
        for (int64_t i = 0; i < n; ++i) heap_.push((int32_t)i);
    }
    int64_t free_count() const { return (int64_t)heap_.size(); }
    int32_t take() {
        const int32_t v = heap_.top();
        heap_.pop();
        return v;
    }
    void give(int32_t v) { heap_.push(v); }
    int64_t size() const { return n_; }

private:
    int64_t n_;
    std::priority_queue<int32_t, std::vector<int32_t>, std::greater<int32_t>> heap_;
};

}  // namespace

struct ls_kv_manager {
    ls_kv_manager_desc d;
    std::vector<Session> sessions;
    IdPool dev;
    IdPool host;
    std::vector<int32_t> heap;          // eligible sessions, max-heap on (T_next, -id)
    int64_t evictable_blocks = 0;       // resident blocks of the sessions in the heap
    struct WarmRef {
        int32_t id;
        uint32_t epoch;
    };
    std::vector<WarmRef> warm_fifo;     // protections by start time (stale entries are skipped)
    int64_t warm_blocks = 0;

    explicit ls_kv_manager(const ls_kv_manager_desc &desc)
        : d(desc), sessions((size_t)desc.max_sessions), dev(desc.num_device_blocks),
          host(desc.num_host_slots) {}

    double t_next(const Session &s) const {
        const double play = s.t_play >= 0.0 ? s.t_play : (double)s.unfinished_tokens * d.seconds_per_token;
        const double reply = s.has_reply ? s.reply_avg : d.reply_prior_s;
        return play + reply;
    }
    bool eligible(const Session &s) const {
        return s.present && !s.running && !s.immediate && !s.warm && s.resident > 0;
    }
    // a ranks before b: larger T_next, then smaller id.
    bool before(int32_t a, int32_t b) const {
        const double ta = t_next(sessions[(size_t)a]), tb = t_next(sessions[(size_t)b]);
        return ta > tb || (ta == tb && a < b);
    }
    void place(size_t i, int32_t id) {
        heap[i] = id;
        sessions[(size_t)id].heap_pos = (int32_t)i;
    }
    void sift_up(size_t i) {
        const int32_t id = heap[i];
        while (i > 0) {
            const size_t p = (i - 1) / 2;
            if (!before(id, heap[p])) break;
            place(i, heap[p]);
            i = p;
        }
        place(i, id);
    }
    void sift_down(size_t i) {
        const int32_t id = heap[i];
        const size_t n = heap.size();
        for (;;) {
            size_t c = 2 * i + 1;
            if (c >= n) break;
            if (c + 1 < n && before(heap[c + 1], heap[c])) ++c;
            if (!before(heap[c], id)) break;
            place(i, heap[c]);
            i = c;
        }
        place(i, id);
    }
    void heap_remove(int32_t id) {
        Session &s = sessions[(size_t)id];
        const size_t i = (size_t)s.heap_pos;
        evictable_blocks -= s.resident;
        s.heap_pos = -1;
        const int32_t last = heap.back();
        heap.pop_back();
        if (i < heap.size()) {
            place(i, last);
            sift_down(i);
            sift_up((size_t)sessions[(size_t)last].heap_pos);
        }
    }
    // Bring session id's heap membership and position up to date after a
    // change of its state, T_next or resident count (old_resident: the count
    // the heap accounted for).
    void refresh(int32_t id, int32_t old_resident) {
        Session &s = sessions[(size_t)id];
        const bool in = s.heap_pos >= 0;
        const bool want = eligible(s);
        if (in) {
            evictable_blocks += s.resident - old_resident;
            if (!want) {
                // heap_remove subtracts the current count, which is what is accounted now
                heap_remove(id);
                return;
            }
            sift_up((size_t)s.heap_pos);
            sift_down((size_t)s.heap_pos);
        } else if (want) {
            heap.push_back(id);
            s.heap_pos = (int32_t)heap.size() - 1;
            evictable_blocks += s.resident;
            sift_up((size_t)s.heap_pos);
        }
    }
    bool warm_valid(const WarmRef &w) const {
        const Session &s = sessions[(size_t)w.id];
        return s.present && s.warm && s.warm_epoch == w.epoch;
    }
    void unwarm(int32_t id) {
        Session &s = sessions[(size_t)id];
        if (!s.warm) return;
        const int32_t r = s.resident;
        s.warm = false;
        warm_blocks -= (int64_t)s.table.size();
        refresh(id, r);
    }
    // Evict up to `need` blocks, appending the moves to out[*n .. cap).  Returns
    // the number of blocks freed.
    int64_t evict(int64_t need, ls_kv_move *out, int32_t cap, int32_t *n) {
        int64_t freed = 0;
        while (freed < need && !heap.empty() && *n < cap && host.free_count() > 0) {
            const int32_t id = heap[0];
            Session &s = sessions[(size_t)id];
            const int32_t r0 = s.resident;
            for (int32_t pos = (int32_t)s.table.size() - 1;
                 pos >= 0 && freed < need && *n < cap && host.free_count() > 0; --pos) {
                Entry &e = s.table[(size_t)pos];
                if (e.state != kResident) continue;
                e.host = host.take();
                out[*n] = ls_kv_move{id, pos, e.dev, e.host};
                ++*n;
                dev.give(e.dev);
                e.dev = -1;
                e.state = kOffloaded;
                --s.resident;
                ++freed;
            }
            refresh(id, r0);
        }
        return freed;
    }
};

namespace {

ls_status fail(ls_status st, const char *fmt, ...) {
    char buf[400];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    ls::set_last_error("%s", buf);
    return st;
}

Session *get(ls_kv_manager *m, int32_t session, const char *what) {
    if (!m) {
        fail(LS_EINVAL, "%s: null manager", what);
        return nullptr;
    }
    if (session < 0 || session >= m->d.max_sessions || !m->sessions[(size_t)session].present) {
        fail(LS_EINVAL, "%s: session %d is not registered", what, session);
        return nullptr;
    }
    return &m->sessions[(size_t)session];
}

}  // namespace

extern "C" {

ls_status kv_manager_create(const ls_kv_manager_desc *desc, ls_kv_manager **out) {
    if (!desc || !out) return fail(LS_EINVAL, "kv_manager_create: null argument");
    *out = nullptr;
    const ls_kv_manager_desc &d = *desc;
    if (d.num_device_blocks < 0 || d.num_device_blocks > INT32_MAX || d.num_host_slots < 0 ||
        d.num_host_slots > INT32_MAX || d.max_sessions <= 0)
        return fail(LS_EINVAL, "kv_manager_create: block, slot or session count out of range");
    if (!(d.reply_ema_alpha > 0.0 && d.reply_ema_alpha <= 1.0))
        return fail(LS_EINVAL, "kv_manager_create: reply_ema_alpha must be in (0, 1]");
    if (!(d.reply_prior_s >= 0.0) || !(d.seconds_per_token >= 0.0) || !(d.warm_ttl_s >= 0.0) ||
        d.warm_cap_blocks < 0)
        return fail(LS_EINVAL, "kv_manager_create: negative or NaN time, rate or cap");
    try {
        *out = new ls_kv_manager(d);
    } catch (const std::bad_alloc &) {
        return fail(LS_ENOMEM, "kv_manager_create: out of host memory");
    }
    return LS_OK;
}

ls_status kv_manager_destroy(ls_kv_manager *m) {
    delete m;
    return LS_OK;
}

ls_status kv_manager_add_session(ls_kv_manager *m, int32_t session) {
    if (!m) return fail(LS_EINVAL, "kv_manager_add_session: null manager");
    if (session < 0 || session >= m->d.max_sessions)
        return fail(LS_EINVAL, "kv_manager_add_session: session %d outside [0, %d)", session,
                    m->d.max_sessions);
    Session &s = m->sessions[(size_t)session];
    if (s.present) return fail(LS_EINVAL, "kv_manager_add_session: session %d exists", session);
    s = Session();
    s.present = true;
    return LS_OK;
}

ls_status kv_manager_remove_session(ls_kv_manager *m, int32_t session) {
    Session *s = get(m, session, "kv_manager_remove_session");
    if (!s) return LS_EINVAL;
    if (s->heap_pos >= 0) m->heap_remove(session);
    if (s->warm) m->warm_blocks -= (int64_t)s->table.size();
    for (const Entry &e : s->table) {
        if (e.dev >= 0) m->dev.give(e.dev);
        if (e.host >= 0) m->host.give(e.host);
    }
    *s = Session();
    return LS_OK;
}

ls_status kv_manager_append_blocks(ls_kv_manager *m, int32_t session, int32_t n, int32_t *block_ids) {
    Session *s = get(m, session, "kv_manager_append_blocks");
    if (!s) return LS_EINVAL;
    if (n < 0 || (n > 0 && !block_ids)) return fail(LS_EINVAL, "kv_manager_append_blocks: bad n or null output");
    if (m->dev.free_count() < n)
        return fail(LS_ENOMEM, "kv_manager_append_blocks: %d blocks asked, %lld free (evict first)", n,
                    (long long)m->dev.free_count());
    const int32_t r = s->resident;
    for (int32_t i = 0; i < n; ++i) {
        const int32_t b = m->dev.take();
        s->table.push_back(Entry{b, -1, kResident});
        block_ids[i] = b;
    }
    s->resident += n;
    if (s->warm) m->warm_blocks += n;
    m->refresh(session, r);
    return LS_OK;
}

ls_status kv_manager_set_running(ls_kv_manager *m, int32_t session, int32_t running) {
    Session *s = get(m, session, "kv_manager_set_running");
    if (!s) return LS_EINVAL;
    const int32_t r = s->resident;
    s->running = running != 0;
    if (s->running) {
        // The turn the protections were waiting for has started.
        s->immediate = false;
        if (s->warm) {
            s->warm = false;
            m->warm_blocks -= (int64_t)s->table.size();
        }
    }
    m->refresh(session, r);
    return LS_OK;
}

ls_status kv_manager_set_playback(ls_kv_manager *m, int32_t session, double t_play_s,
                                  int64_t unfinished_tokens) {
    Session *s = get(m, session, "kv_manager_set_playback");
    if (!s) return LS_EINVAL;
    if (std::isnan(t_play_s) || unfinished_tokens < 0)
        return fail(LS_EINVAL, "kv_manager_set_playback: NaN horizon or negative token count");
    const int32_t r = s->resident;
    s->t_play = t_play_s < 0.0 ? -1.0 : t_play_s;
    s->unfinished_tokens = unfinished_tokens;
    m->refresh(session, r);
    return LS_OK;
}

ls_status kv_manager_observe_reply(ls_kv_manager *m, int32_t session, double interval_s) {
    Session *s = get(m, session, "kv_manager_observe_reply");
    if (!s) return LS_EINVAL;
    if (!(interval_s >= 0.0)) return fail(LS_EINVAL, "kv_manager_observe_reply: interval must be >= 0");
    const int32_t r = s->resident;
    const double a = m->d.reply_ema_alpha;
    s->reply_avg = s->has_reply ? a * interval_s + (1.0 - a) * s->reply_avg : interval_s;
    s->has_reply = true;
    m->refresh(session, r);
    return LS_OK;
}

ls_status kv_manager_speech_start(ls_kv_manager *m, int32_t session) {
    Session *s = get(m, session, "kv_manager_speech_start");
    if (!s) return LS_EINVAL;
    const int32_t r = s->resident;
    s->immediate = true;
    m->refresh(session, r);
    return LS_OK;
}

ls_status kv_manager_evict(ls_kv_manager *m, int64_t blocks_needed, ls_kv_move *moves,
                           int32_t max_moves, int32_t *num_moves) {
    if (!m || !num_moves || (max_moves > 0 && !moves) || max_moves < 0 || blocks_needed < 0)
        return fail(LS_EINVAL, "kv_manager_evict: bad argument");
    *num_moves = 0;
    if (blocks_needed > max_moves)
        return fail(LS_ENOMEM, "kv_manager_evict: room for %d moves, %lld blocks asked", max_moves,
                    (long long)blocks_needed);
    m->evict(blocks_needed, moves, max_moves, num_moves);
    return LS_OK;
}

ls_status kv_manager_preload(ls_kv_manager *m, int32_t session, double time_available_s,
                             double bytes_per_block, double bandwidth_bytes_per_s,
                             ls_kv_move *restores, int32_t max_restores, int32_t *num_restores,
                             ls_kv_move *evictions, int32_t max_evictions, int32_t *num_evictions,
                             int32_t *admitted) {
    Session *s = get(m, session, "kv_manager_preload");
    if (!s) return LS_EINVAL;
    if (!num_restores || !num_evictions || !admitted || max_restores < 0 || max_evictions < 0 ||
        (max_restores > 0 && !restores) || (max_evictions > 0 && !evictions) || std::isnan(time_available_s) ||
        !(bytes_per_block >= 0.0) || !(bandwidth_bytes_per_s > 0.0))
        return fail(LS_EINVAL, "kv_manager_preload: bad argument");
    *num_restores = 0;
    *num_evictions = 0;
    *admitted = 0;
    if (s->loading > 0) return fail(LS_EINVAL, "kv_manager_preload: a preload of session %d is in flight", session);
    // Speech start protects the session's resident KV whatever the admission says.
    {
        const int32_t r = s->resident;
        s->immediate = true;
        m->refresh(session, r);
    }
    int64_t off = 0;
    for (const Entry &e : s->table) off += e.state == kOffloaded;
    if (off == 0) {
        *admitted = 1;
        return LS_OK;
    }
    if (off > max_restores)
        return fail(LS_ENOMEM, "kv_manager_preload: room for %d restores, %lld needed", max_restores,
                    (long long)off);
    const double transfer_s = (double)off * bytes_per_block / bandwidth_bytes_per_s;
    if (transfer_s > time_available_s) return LS_OK;                 // not admitted: load on demand
    const int64_t short_by = std::max<int64_t>(0, off - m->dev.free_count());
    if (short_by > m->evictable_blocks || short_by > max_evictions ||
        (short_by > 0 && m->host.free_count() < short_by))
        return LS_OK;                                                // not enough HBM can be freed
    if (short_by > 0) m->evict(short_by, evictions, max_evictions, num_evictions);
    // Prefix first: a cancelled preload leaves the leading positions usable.
    for (int32_t pos = 0; pos < (int32_t)s->table.size(); ++pos) {
        Entry &e = s->table[(size_t)pos];
        if (e.state != kOffloaded) continue;
        e.dev = m->dev.take();
        e.state = kLoading;
        restores[*num_restores] = ls_kv_move{session, pos, e.dev, e.host};
        ++*num_restores;
        ++s->loading;
    }
    *admitted = 1;
    return LS_OK;
}

ls_status kv_manager_load_sync(ls_kv_manager *m, int32_t session, ls_kv_move *restores, int32_t max_restores,
                               int32_t *num_restores, ls_kv_move *evictions, int32_t max_evictions,
                               int32_t *num_evictions) {
    int32_t admitted = 0;
    const ls_status st = kv_manager_preload(m, session, std::numeric_limits<double>::infinity(), 0.0, 1.0,
                                            restores, max_restores, num_restores, evictions, max_evictions,
                                            num_evictions, &admitted);
    if (st != LS_OK) return st;
    if (!admitted)
        return fail(LS_ENOMEM, "kv_manager_load_sync: not enough HBM can be freed for session %d", session);
    return LS_OK;
}

ls_status kv_manager_preload_done(ls_kv_manager *m, int32_t session, double now_s) {
    Session *s = get(m, session, "kv_manager_preload_done");
    if (!s) return LS_EINVAL;
    if (std::isnan(now_s)) return fail(LS_EINVAL, "kv_manager_preload_done: NaN time");
    const int32_t r = s->resident;
    for (Entry &e : s->table) {
        if (e.state != kLoading) continue;
        m->host.give(e.host);
        e.host = -1;
        e.state = kResident;
        ++s->resident;
    }
    s->loading = 0;
    if (!s->running) {
        // Warm protection replaces the speech-start protection, bounded in time
        // and in total size (oldest protections are released first).
        s->immediate = false;
        if (!s->warm) {
            s->warm = true;
            m->warm_blocks += (int64_t)s->table.size();
        }
        s->warm_since = now_s;
        ++s->warm_epoch;
        m->warm_fifo.push_back(ls_kv_manager::WarmRef{session, s->warm_epoch});
    }
    m->refresh(session, r);
    size_t keep = 0;
    for (size_t i = 0; i < m->warm_fifo.size(); ++i) {
        const ls_kv_manager::WarmRef w = m->warm_fifo[i];
        if (!m->warm_valid(w)) continue;
        if (m->warm_blocks > m->d.warm_cap_blocks && w.id != session) {
            m->unwarm(w.id);
            continue;
        }
        m->warm_fifo[keep++] = w;
    }
    m->warm_fifo.resize(keep);
    return LS_OK;
}

ls_status kv_manager_preload_cancel(ls_kv_manager *m, int32_t session) {
    Session *s = get(m, session, "kv_manager_preload_cancel");
    if (!s) return LS_EINVAL;
    for (Entry &e : s->table) {
        if (e.state != kLoading) continue;
        m->dev.give(e.dev);
        e.dev = -1;
        e.state = kOffloaded;
    }
    s->loading = 0;
    return LS_OK;
}

ls_status kv_manager_tick(ls_kv_manager *m, double now_s) {
    if (!m || std::isnan(now_s)) return fail(LS_EINVAL, "kv_manager_tick: bad argument");
    size_t keep = 0;
    for (size_t i = 0; i < m->warm_fifo.size(); ++i) {
        const ls_kv_manager::WarmRef w = m->warm_fifo[i];
        if (!m->warm_valid(w)) continue;
        if (now_s - m->sessions[(size_t)w.id].warm_since >= m->d.warm_ttl_s) m->unwarm(w.id);
        else m->warm_fifo[keep++] = w;
    }
    m->warm_fifo.resize(keep);
    return LS_OK;
}

ls_status kv_manager_session_info(ls_kv_manager *m, int32_t session, double *t_next, int32_t *flags,
                                  int32_t *num_blocks) {
    Session *s = get(m, session, "kv_manager_session_info");
    if (!s) return LS_EINVAL;
    if (t_next) *t_next = m->t_next(*s);
    if (flags)
        *flags = (s->running ? LS_KV_RUNNING : 0) | (s->immediate ? LS_KV_IMMEDIATE : 0) |
                 (s->warm ? LS_KV_WARM : 0) | (s->heap_pos >= 0 ? LS_KV_EVICTABLE : 0);
    if (num_blocks) *num_blocks = (int32_t)s->table.size();
    return LS_OK;
}

ls_status kv_manager_table(ls_kv_manager *m, int32_t session, int32_t max_blocks, int32_t *device_ids,
                           int32_t *host_slots, int32_t *states) {
    Session *s = get(m, session, "kv_manager_table");
    if (!s) return LS_EINVAL;
    if (max_blocks < (int32_t)s->table.size())
        return fail(LS_ENOMEM, "kv_manager_table: room for %d entries, %zu needed", max_blocks, s->table.size());
    for (size_t i = 0; i < s->table.size(); ++i) {
        if (device_ids) device_ids[i] = s->table[i].dev;
        if (host_slots) host_slots[i] = s->table[i].host;
        if (states) states[i] = s->table[i].state;
    }
    return LS_OK;
}

ls_status kv_manager_counts(ls_kv_manager *m, int64_t *free_device_blocks, int64_t *free_host_slots,
                            int64_t *evictable_blocks, int64_t *warm_blocks) {
    if (!m) return fail(LS_EINVAL, "kv_manager_counts: null manager");
    if (free_device_blocks) *free_device_blocks = m->dev.free_count();
    if (free_host_slots) *free_host_slots = m->host.free_count();
    if (evictable_blocks) *evictable_blocks = m->evictable_blocks;
    if (warm_blocks) *warm_blocks = m->warm_blocks;
    return LS_OK;
}

}  // extern "C"
