/*
 * liveserve_kv.h — C ABI of the MI355X (gfx950) paged-KV hot path under
 * LiveServe's interaction-aware serving (arXiv 2606.22983).
 *
 * The paper keeps the serving engine's paged KV block pool and its
 * block-level allocation (§5.1, §6 "Hierarchical KV cache manager"), reuses a
 * session's multi-turn KV so the next turn does not re-prefill history (§5),
 * offloads idle multi-turn KV from HBM to host DRAM (§5, §5.1) and preloads it
 * back during user speech through the HBM-DRAM offload connector's
 * asynchronous transfer path (§5.2, §6).  This library is the data-parallel
 * part of that: attention of the thinker/talker decoders (§2.1) over the
 * per-session paged cache — batched single-token decode and next-turn chunked
 * prefill over reused context — and the block stash/restore copies.
 *
 * Conventions for every entry point
 *   - Ownership: the caller owns every buffer (device memory, pinned host
 *     memory).  The library never allocates device memory; a pool handle owns
 *     only host-side metadata.
 *   - Asynchrony: work is enqueued on the given HIP stream (NULL = the default
 *     stream) and the call returns without waiting for it.
 *   - Errors: arguments are validated on the host before anything is
 *     enqueued; any status other than LS_OK means nothing was enqueued.
 *     ls_last_error() returns a message for the calling thread's last failure.
 *     No C++ exception crosses this boundary.
 *   - Device-side index arrays (block tables, lengths, block ids) are read by
 *     the kernels, which bounds-check every block id they dereference: an id
 *     outside [0, num_blocks) is skipped (its keys are treated as absent, its
 *     copy is not made) and a bit is set in a device error word that
 *     ls_device_errors() returns.  A result computed with such an id is not
 *     meaningful.
 *   - Concurrency: calls on different streams may run concurrently only on
 *     disjoint sets of blocks and with their own scratch buffers (a decode or
 *     prefill workspace, a copy's staging ring); ordering between streams is the
 *     caller's (events).  Blocks being restored must not be read by attention
 *     until the restore's stream has been waited on — the same rule the
 *     paper's KV manager follows before reusing preloaded KV (§5.2).
 *   - Data types: K, V, Q and outputs are bfloat16 (bf16); arithmetic inside
 *     attention accumulates in fp32.
 *
 * Pool layout (device memory, bf16, num_layers x num_blocks x 2 x Hkv tiles):
 *   pool[layer][block][kv][head][tile]         kv = 0: K, kv = 1: V
 *   K tile = [head_dim / 8][block_size tokens][8 dims]
 *            (chunk-major: element (token t, dim d) at ((d / 8) * block_size
 *            + t) * 8 + d % 8, i.e. 16-byte chunks of 8 dims, all tokens of
 *            dims 0..7 first; every supported head_dim is a multiple of 8)
 *   V tile = [head_dim][block_size tokens]     (dim-major)
 * Logical token t of session s lives in slot t % block_size of block
 * block_tables[s * max_blocks_per_session + t / block_size].
 *
 * Staging layout of stash/restore (device or pinned host memory):
 *   staging[i][layer][kv][head][tile]   for block ids[i], i = 0..n-1
 * i.e. every layer's (K, V) slab of one block is contiguous, block after block.
 */
#ifndef LIVESERVE_KV_H
#define LIVESERVE_KV_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    LS_OK = 0,
    LS_EINVAL = -22,        /* invalid argument; nothing enqueued */
    LS_ENOMEM = -12,        /* a caller-provided buffer is too small */
    LS_EHIP = -5,           /* a HIP runtime call failed */
    LS_EUNSUPPORTED = -95   /* valid but unsupported geometry (head_dim, group size) */
} ls_status;

/* Bits of the device error word (ls_device_errors). */
#define LS_DEVERR_BLOCK_ID 0x1u     /* a block id outside [0, num_blocks) was skipped */
#define LS_DEVERR_LENGTH   0x2u     /* a length outside what the call can attend (an empty
                                       decode context, a context past its block table, a
                                       turn longer than max_new_len); see each call */
#define LS_DEVERR_INTERNAL 0x4u     /* an internal bounded wait expired (a library bug) */

typedef struct ls_kv_pool ls_kv_pool;

typedef struct {
    int32_t num_layers;        /* >= 1 */
    int32_t num_kv_heads;      /* Hkv >= 1 */
    int32_t head_dim;          /* D: 64 or 128 */
    int32_t block_size;        /* tokens per block: 16 */
    int64_t num_blocks;        /* blocks per layer */
    void *kv_base;             /* device, >= ls_kv_pool_bytes(...) bytes, 256-byte aligned */
    size_t kv_bytes;
} ls_kv_pool_desc;

/* Bytes of pool memory for the given geometry (0 on overflow or bad geometry). */
size_t ls_kv_pool_bytes(int32_t num_layers, int64_t num_blocks, int32_t num_kv_heads,
                        int32_t head_dim, int32_t block_size);

/*
 * kv_pool_create — wrap caller-owned device memory as a paged KV block pool
 * (the paged KV block pool of §6, block-level allocation of §5.1).  Validates
 * the geometry (block_size 16, head_dim 64 or 128, kv_bytes large enough,
 * 256-byte alignment), records the layout and the current HIP device, and
 * writes an opaque handle to *out.  Launches nothing and touches no device
 * memory.  LS_EINVAL on bad arguments, LS_EUNSUPPORTED on an unsupported
 * head_dim or block_size.
 */
ls_status kv_pool_create(const ls_kv_pool_desc *desc, ls_kv_pool **out);

/* Free the handle's host metadata (never the caller's memory).  NULL is OK. */
ls_status kv_pool_destroy(ls_kv_pool *pool);

/*
 * Workspace bytes paged_attn_decode needs for this shape: the split-K partial
 * results (running max, running sum and unnormalised output per split, fp32).
 * No initialisation is needed; calls on one stream may reuse the same
 * workspace, concurrent calls need their own.  Returns 0 for invalid arguments.
 */
size_t ls_decode_workspace_bytes(const ls_kv_pool *pool, int32_t num_sessions,
                                 int32_t num_q_heads, int32_t max_blocks_per_session);

/*
 * paged_attn_decode — one batched decode step of the thinker/talker
 * autoregressive decoders (§2.1; the engines' continuous-batching decode loop,
 * §4 and §6) over the per-session paged KV cache.
 *
 *   q              device bf16 [num_sessions][num_q_heads][head_dim]: the step's query
 *   k_new, v_new   device bf16 [num_sessions][num_kv_heads][head_dim], or both NULL.
 *                  When given, the step's own K/V row is appended: the query attends
 *                  to context_lens[s] + 1 keys, the last being this row, and the row
 *                  is written at logical position context_lens[s] (its block must
 *                  already be in the table) by the same launch.
 *   block_tables   device int32 [num_sessions][max_blocks_per_session]
 *   context_lens   device int32 [num_sessions]: tokens already in the pool, >= 1
 *                  (>= 0 with append).  An empty context (no key to attend) gives a
 *                  zero output row and is flagged (LS_DEVERR_LENGTH); so is a length
 *                  whose keys do not fit the table, which is clipped to it.
 *   context_lens_host  optional host copy of context_lens (NULL: the kernel plans the
 *                  split-K schedule from the device lengths).  When given it must hold
 *                  the same values; the host then rejects empty or over-long contexts
 *                  (LS_EINVAL) and plans the splits itself: sessions are split only as
 *                  far as the batch needs to fill the GPU, and the split merge is
 *                  launched only when some session was split.  A device length that
 *                  differs from its host copy so that the plan no longer covers it is
 *                  flagged (LS_DEVERR_LENGTH).
 *   scale          softmax scale applied to q.k (normally 1/sqrt(head_dim))
 *   out            device bf16 [num_sessions][num_q_heads][head_dim]:
 *                  out = softmax(scale * q K^T) V over the session's keys, per query
 *                  head h using KV head h / (num_q_heads / num_kv_heads)
 *   workspace      device, >= ls_decode_workspace_bytes(...) bytes
 *
 * Supported: num_q_heads / num_kv_heads in {1, 2, 4, 8}; at most 2048 sessions
 * and 16384 blocks (262,144 tokens) per session.  Errors: LS_EINVAL
 * (NULL pointer, layer out of range, num_q_heads not a multiple of num_kv_heads,
 * only one of k_new / v_new, a bad host length), LS_ENOMEM (workspace too
 * small), LS_EUNSUPPORTED (group size, batch limits), LS_EHIP (launch failure).
 */
ls_status paged_attn_decode(ls_kv_pool *pool, int32_t layer, int32_t num_sessions,
                            int32_t num_q_heads, const void *q, const void *k_new,
                            const void *v_new, const int32_t *block_tables,
                            int32_t max_blocks_per_session, const int32_t *context_lens,
                            const int32_t *context_lens_host, float scale, void *out,
                            void *workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * ls_decode_schedule — how paged_attn_decode will run a batch of this shape
 * on `stream`: *split_tokens tokens per split, *host_planned 1 when the
 * schedule is planned on the host from context_lens_host (0: in the kernel,
 * also when the host plan is estimated to be no faster or has more items than
 * the kernel arguments carry: 7680 for batches of at most 1024 sessions, 4 KV
 * heads and 8 splits per session, else 3840), *merge 1 when the split merge
 * kernel runs.  appended: 1
 * when k_new / v_new will be given.  Pure host computation; LS_EINVAL as for
 * paged_attn_decode.
 */
ls_status ls_decode_schedule(const ls_kv_pool *pool, int32_t num_sessions, int32_t num_q_heads,
                             int32_t max_blocks_per_session, const int32_t *context_lens_host,
                             int32_t appended, hipStream_t stream, int32_t *split_tokens,
                             int32_t *host_planned, int32_t *merge);

/* Bytes of the static split scratch behind paged_attn_decode_static. */
#define LS_DECODE_STATIC_SCRATCH_BYTES ((size_t)32 << 20)

/*
 * paged_attn_decode_static — paged_attn_decode without a workspace argument,
 * for callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation).  The split
 * partials go to a static buffer of LS_DECODE_STATIC_SCRATCH_BYTES inside the
 * library: one per GPU, resolved on the first call on that GPU and held until
 * the process ends.  The call allocates nothing and calls no allocating
 * routine.  LS_ENOMEM when the shape needs more scratch than that
 * (ls_decode_workspace_bytes of the same shape).  Every call on a GPU shares
 * its buffer, so calls that may overlap on one GPU (different streams) race:
 * serialise them.  Other arguments, results and errors as paged_attn_decode.
 */
ls_status paged_attn_decode_static(ls_kv_pool *pool, int32_t layer, int32_t num_sessions,
                                   int32_t num_q_heads, const void *q, const void *k_new,
                                   const void *v_new, const int32_t *block_tables,
                                   int32_t max_blocks_per_session, const int32_t *context_lens,
                                   const int32_t *context_lens_host, float scale, void *out,
                                   hipStream_t stream);

/*
 * paged_attn_prefill — next-turn (chunked) prefill over reused multi-turn
 * context (§5: reusing LLM-stage KV avoids re-prefilling conversation history;
 * §3: the prefetch endpoint's current-turn prefill).  Session s brings n_s new
 * tokens; they are appended at logical positions c_s .. c_s + n_s - 1 and new
 * row j attends causally to keys 0 .. c_s + j (bottom-right alignment).  A
 * chunked prefill is repeated calls with c_s advanced by the previous chunk.
 *
 *   q              device bf16 [total_new_tokens][num_q_heads][head_dim], sessions
 *                  back to back in cu_new_lens order
 *   k_new, v_new   device bf16 [total_new_tokens][num_kv_heads][head_dim], or both
 *                  NULL when the turn's K/V is already in the pool
 *   cu_new_lens    device int32 [num_sessions + 1]: prefix sums of n_s (cu[0] = 0)
 *   reused_lens    device int32 [num_sessions]: c_s >= 0
 *   lens_host      optional host int32 [num_sessions][2] = (n_s, c_s), the same values
 *                  as the device arrays (NULL: nothing is checked on the host).  When
 *                  given, the host checks every turn against max_new_len, the table
 *                  and total_new_tokens (LS_EINVAL) before anything is enqueued, and
 *                  deals the query tiles to the XCDs itself (up to 256 sessions and
 *                  256 session/KV-head pairs; beyond that the kernel deals them).  A
 *                  device turn longer than its planned tiles is flagged
 *                  (LS_DEVERR_LENGTH); its rows past them are not written.
 *   total_new_tokens, max_new_len   host ints: cu[S] and max_s n_s (grid sizing).
 *                  A turn longer than max_new_len (device lengths only) is flagged
 *                  (LS_DEVERR_LENGTH) and its rows past max_new_len are not written.
 *   block_tables   device int32 [num_sessions][max_blocks_per_session], covering
 *                  c_s + n_s tokens
 *   out            device bf16 [total_new_tokens][num_q_heads][head_dim]
 *   workspace      optional device memory (16-byte aligned) of workspace_bytes >=
 *                  LS_PREFILL_WORKSPACE_BYTES, or NULL (LS_ENOMEM if too small,
 *                  LS_EINVAL if misaligned).  With host lengths the workgroups then stay
 *                  resident, one per CU, and take query tiles in order through a
 *                  counter per XCD kept here; an XCD whose tiles run out takes the next
 *                  tiles of the XCD with the most left, so XCDs of different speeds
 *                  finish together.  The call clears it first (its contents on entry do
 *                  not matter).  Calls that may run at the same time need different
 *                  workspaces.  Unused without host lengths.
 *
 * Supported: head_dim 128 or 64, num_q_heads / num_kv_heads in {1, 2, 4, 8}.
 * Errors as for paged_attn_decode.
 */
#define LS_PREFILL_WORKSPACE_BYTES ((size_t)256)
ls_status paged_attn_prefill(ls_kv_pool *pool, int32_t layer, int32_t num_sessions,
                             int32_t num_q_heads, const void *q, const void *k_new,
                             const void *v_new, const int32_t *cu_new_lens,
                             const int32_t *reused_lens, const int32_t *lens_host,
                             int32_t total_new_tokens, int32_t max_new_len,
                             const int32_t *block_tables, int32_t max_blocks_per_session,
                             float scale, void *out, void *workspace, size_t workspace_bytes,
                             hipStream_t stream);

/*
 * Arguments shared by the three block-copy calls below.
 *
 *   block_ids       device int32 [n]: distinct ids in [0, num_blocks)
 *   block_ids_host  optional host copy of the same ids; when given, range and
 *                   distinctness are checked on the host (LS_EINVAL)
 *   staging         device memory, or pinned host memory when staging_on_host != 0,
 *                   of staging_bytes >= n x (one block's all-layer slab) bytes
 *                   (LS_ENOMEM otherwise), layout above
 *   ring            with host staging: caller-owned device memory (16-byte aligned)
 *                   that the copy moves through in whole-block chunks: a DMA engine
 *                   transfer and a copy kernel per chunk, on the caller's stream.  It
 *                   must hold the copied layer range of at least one block (LS_ENOMEM
 *                   otherwise).  Two copies that may run at the same time (different
 *                   streams) need different rings.  Ignored (may be NULL) with device
 *                   staging.
 *   max_gbps        0: full rate (a persistent grid of four (restore) or six (stash)
 *                   256-thread workgroups per CU the stream may use).  r > 0: a
 *                   rate-bounded copy of at most r GB/s
 *                   (10^9 bytes per second) of payload, for background work beside live
 *                   decode (§5.2: preloads must not interfere with live requests; the
 *                   KV manager's admission divides bytes by such a rate).  It runs one
 *                   workgroup per CU, small enough to share the CU with a decode
 *                   workgroup, each copying a burst of up to 32 slabs per window of
 *                   the GPU's constant-frequency clock (at the window's start, then
 *                   it sleeps; windows of about a millisecond, longer at rates too
 *                   low for one slab per workgroup in a millisecond).  A rate above what that grid moves gives its maximum.
 *                   LS_EINVAL for a negative or NaN rate.
 * Bit-exact byte copies.  n == 0 is a no-op.
 */

/*
 * kv_blocks_stash — offload: copy every layer's K/V slab of blocks ids[0..n-1]
 * into staging (layout above), the HBM-to-DRAM eviction of idle multi-turn KV
 * (§5, §5.1; eviction stays block-level, suffix blocks first — the order is
 * the caller's).  The pool is left unchanged; freeing the ids is the caller's
 * decision once the stream has passed this call.  With host staging and a
 * ring, each chunk is a gather kernel into the ring, then a device-to-host DMA.
 */
ls_status kv_blocks_stash(ls_kv_pool *pool, int32_t n, const int32_t *block_ids,
                          const int32_t *block_ids_host, void *staging, size_t staging_bytes,
                          int32_t staging_on_host, void *ring, size_t ring_bytes,
                          double max_gbps, hipStream_t stream);

/*
 * kv_blocks_restore — reload / speech-triggered preload: copy staging (layout
 * above) back into pool blocks ids[0..n-1] (§5.2; the offload connector's
 * asynchronous transfer path, §6).  Blocks are written in id order, so a
 * restore cut short by the caller (a cancelled preload) leaves a complete
 * prefix, and restoring the remaining ids afterwards (the synchronous
 * fallback of §5.2) gives the same pool as one full restore.  With host
 * staging and a ring, each chunk is a host-to-device DMA into the ring, then
 * the scatter kernel.
 */
ls_status kv_blocks_restore(ls_kv_pool *pool, int32_t n, const int32_t *block_ids,
                            const int32_t *block_ids_host, const void *staging,
                            size_t staging_bytes, int32_t staging_on_host, void *ring,
                            size_t ring_bytes, double max_gbps, hipStream_t stream);

/*
 * kv_blocks_restore_layers — kv_blocks_restore of the layers
 * [layer_begin, layer_begin + layer_count) only, from the same all-layer
 * staging layout.  A next-turn prefill can then start on layer l as soon as
 * layer l is back, while later layers are still being restored (the reload
 * leaves the critical path, §5.2 and §7): the caller restores layer by layer
 * on a copy stream and makes the compute stream wait on an event per layer.
 * With host staging and a ring, each chunk is one strided host-to-device
 * copy (the range of every block) into the ring, then the scatter kernel; the
 * ring must hold the range of one block.  LS_EINVAL for a range outside [0, num_layers);
 * otherwise as kv_blocks_restore.  Restoring every layer range of a set of
 * blocks gives the same pool as one kv_blocks_restore.
 */
ls_status kv_blocks_restore_layers(ls_kv_pool *pool, int32_t layer_begin, int32_t layer_count, int32_t n,
                                   const int32_t *block_ids, const int32_t *block_ids_host,
                                   const void *staging, size_t staging_bytes, int32_t staging_on_host,
                                   void *ring, size_t ring_bytes, double max_gbps,
                                   hipStream_t stream);

/* ------------------------------------------------------------------------
 * KV manager (host only): the policy that decides which blocks the
 * stash/restore calls above move — next-use-aware eviction (§5.1) with the
 * indexed candidate heap (§6) and speech-triggered preload with admission,
 * cancellation and synchronous fallback (§5.2).  It tracks, per session, the
 * block table (by block position: device block, host slot, state) and the
 * side-table metadata of §6 (running, speech/barge-in protection, warm
 * protection after a preload, playback horizon, reply-interval average).
 * It launches nothing: a call that frees or assigns blocks returns moves, and
 * the caller issues the copies (kv_blocks_stash for evictions,
 * kv_blocks_restore for restores) on a stream before any kernel writes the
 * freed blocks or reads the restored ones.  Host slots index the caller's
 * host store of whole blocks (staging layout above).  Device block ids and
 * host slots are handed out lowest first.  One manager must not be used from
 * two threads at once.  Status and ls_last_error() as for the rest of the ABI.
 * ---------------------------------------------------------------------- */

typedef struct ls_kv_manager ls_kv_manager;

typedef struct {
    int64_t num_device_blocks;  /* pool block ids the manager owns: [0, n) */
    int64_t num_host_slots;     /* host store capacity in blocks: slots [0, n) */
    int32_t max_sessions;       /* session ids are [0, max_sessions) */
    double reply_prior_s;       /* T_reply before a session's first observed reply interval */
    double reply_ema_alpha;     /* weight of the newest interval in the moving average, (0, 1] */
    double seconds_per_token;   /* playback per unfinished response token, when the horizon is unknown */
    double warm_ttl_s;          /* how long a completed preload stays protected */
    int64_t warm_cap_blocks;    /* cap on blocks under that protection (oldest released first) */
} ls_kv_manager_desc;

/* Block states in kv_manager_table. */
#define LS_KV_RESIDENT  0       /* in the pool at the listed device block */
#define LS_KV_OFFLOADED 1       /* in the host store at the listed host slot */
#define LS_KV_LOADING   2       /* restore issued: host slot -> device block, not yet done */

/* Session flags in kv_manager_session_info. */
#define LS_KV_RUNNING   0x1     /* pinned by a running request */
#define LS_KV_IMMEDIATE 0x2     /* speech start / barge-in: protected from eviction */
#define LS_KV_WARM      0x4     /* protected after a completed preload */
#define LS_KV_EVICTABLE 0x8     /* an eviction candidate (idle, resident blocks, unprotected) */

/* One block move: position `position` of `session` between device block
 * `device_block` and host slot `host_slot` (direction given by the call). */
typedef struct {
    int32_t session;
    int32_t position;
    int32_t device_block;
    int32_t host_slot;
} ls_kv_move;

/* Create / destroy (destroy frees host metadata only; NULL is OK). */
ls_status kv_manager_create(const ls_kv_manager_desc *desc, ls_kv_manager **out);
ls_status kv_manager_destroy(ls_kv_manager *m);

/* Register / forget a session (forgetting returns its blocks and slots). */
ls_status kv_manager_add_session(ls_kv_manager *m, int32_t session);
ls_status kv_manager_remove_session(ls_kv_manager *m, int32_t session);

/* Allocate n device blocks at the tail of the session's table (new tokens);
 * block_ids[n] receives them.  LS_ENOMEM when fewer than n are free: evict
 * first (kv_manager_evict). */
ls_status kv_manager_append_blocks(ls_kv_manager *m, int32_t session, int32_t n, int32_t *block_ids);

/* A request of the session starts (running != 0: its KV is pinned, and the
 * speech and warm protections end) or finishes (running == 0: idle). */
ls_status kv_manager_set_running(ls_kv_manager *m, int32_t session, int32_t running);

/* Monitor inputs to T_next = T_play + T_reply (§5.1, the next-use estimate).
 * t_play_s: seconds of the session's audio still to be played, or < 0 when
 * unknown (then unfinished_tokens x seconds_per_token stands in).
 * observe_reply: one measured gap between the end of the session's playback
 * and the user's next finished utterance (averaged over the session). */
ls_status kv_manager_set_playback(ls_kv_manager *m, int32_t session, double t_play_s,
                                  int64_t unfinished_tokens);
ls_status kv_manager_observe_reply(ls_kv_manager *m, int32_t session, double interval_s);

/* Speech start or barge-in: the session's resident KV becomes immediate
 * reuse, excluded from eviction until its request runs. */
ls_status kv_manager_speech_start(ls_kv_manager *m, int32_t session);

/*
 * Free at least blocks_needed device blocks (fewer only when every eligible
 * block is gone or the host store is full): eligible sessions in decreasing
 * T_next (ties: smaller id first), each from its last resident position
 * downwards (suffix first, §5.1).  Writes the moves (device block -> host
 * slot) to moves[0 .. *num_moves); the blocks are free once the call returns,
 * so the caller stashes them before anything else writes them.
 * LS_ENOMEM if max_moves < blocks_needed.
 */
ls_status kv_manager_evict(ls_kv_manager *m, int64_t blocks_needed, ls_kv_move *moves,
                           int32_t max_moves, int32_t *num_moves);

/*
 * Speech-triggered preload (§5.2).  Marks the session immediate (as
 * kv_manager_speech_start).  When it has offloaded blocks, the preload is
 * admitted (*admitted = 1) only if offloaded blocks x bytes_per_block /
 * bandwidth_bytes_per_s <= time_available_s (the time left before its LLM
 * stage runs, under the current transfer pressure the caller measures) and
 * enough device blocks are free or can be freed from eligible sessions.  Then
 * restores[0 .. *num_restores) lists, prefix first, every offloaded position
 * with its host slot and newly assigned device block (state LOADING), and
 * evictions[0 .. *num_evictions) the blocks evicted to make room: stash those
 * before restoring into them.  Not admitted: *admitted = 0, nothing moves;
 * the caller may retry later or load on demand (kv_manager_load_sync).
 * LS_ENOMEM if max_restores is below the offloaded count; LS_EINVAL if a
 * preload of the session is still in flight.
 */
ls_status kv_manager_preload(ls_kv_manager *m, int32_t session, double time_available_s,
                             double bytes_per_block, double bandwidth_bytes_per_s,
                             ls_kv_move *restores, int32_t max_restores, int32_t *num_restores,
                             ls_kv_move *evictions, int32_t max_evictions, int32_t *num_evictions,
                             int32_t *admitted);

/* The synchronous fallback: kv_manager_preload without the time test;
 * LS_ENOMEM when not enough device blocks can be freed. */
ls_status kv_manager_load_sync(ls_kv_manager *m, int32_t session, ls_kv_move *restores,
                               int32_t max_restores, int32_t *num_restores, ls_kv_move *evictions,
                               int32_t max_evictions, int32_t *num_evictions);

/* The restores of the session's preload have completed (the caller has
 * waited on their stream): LOADING blocks become resident, their host slots
 * free, and unless the session is running its KV is protected for warm_ttl_s
 * (releasing the oldest protections beyond warm_cap_blocks). */
ls_status kv_manager_preload_done(ls_kv_manager *m, int32_t session, double now_s);

/* Abandon the session's preload: LOADING blocks return to OFFLOADED and their
 * device blocks are freed (the caller must not let the abandoned restores
 * land after those blocks are reused: same stream, or wait first). */
ls_status kv_manager_preload_cancel(ls_kv_manager *m, int32_t session);

/* Release warm protections older than warm_ttl_s at time now_s. */
ls_status kv_manager_tick(ls_kv_manager *m, double now_s);

/* Queries: T_next, LS_KV_* flags and table length; the table itself
 * (device block or -1, host slot or -1, LS_KV_* state per position; NULL
 * arrays are skipped; LS_ENOMEM if max_blocks is below the length); counts. */
ls_status kv_manager_session_info(ls_kv_manager *m, int32_t session, double *t_next, int32_t *flags,
                                  int32_t *num_blocks);
ls_status kv_manager_table(ls_kv_manager *m, int32_t session, int32_t max_blocks, int32_t *device_ids,
                           int32_t *host_slots, int32_t *states);
ls_status kv_manager_counts(ls_kv_manager *m, int64_t *free_device_blocks, int64_t *free_host_slots,
                            int64_t *evictable_blocks, int64_t *warm_blocks);

/* ------------------------------------------------------------------------
 * Interaction-aware batch selection (host only; §4, the scheduling procedure
 * and its algorithm): one stage, one scheduling round.  It orders the ready
 * requests by urgency class and admits them into the next batch under the
 * round's token and KV-block budgets; the batch is what paged_attn_decode /
 * paged_attn_prefill then run.
 * ---------------------------------------------------------------------- */

typedef struct {
    double playback_buffer_s;   /* stage-aware playback buffer P (s); NaN: unknown */
    double ready_age_s;         /* time since the request became ready (A) */
    int32_t first_audio_done;   /* 1 once it produced its first playable audio */
    int32_t reserved;
    int64_t kv_blocks_held;     /* GPU KV it occupies (K); < 0: unknown */
    int64_t tokens_needed;      /* token budget it uses if admitted */
    int64_t kv_blocks_needed;   /* KV blocks it allocates if admitted */
} ls_sched_request;

typedef struct {
    double p_safe_s;            /* minimum safe buffer P_safe (> 0) */
    double alpha;               /* weight of the barge-in exposure cost */
    double beta;                /* weight of the KV-pressure benefit */
    double kv_occupancy;        /* occupied / allocatable GPU KV of the stage (R_occ); NaN: unknown */
    int64_t token_budget;       /* round budgets M */
    int64_t kv_block_budget;
} ls_sched_stage;

/*
 * Classes: 0 (U0) first audio done and P <= P_safe, ordered by P ascending;
 * 1 (U1) no first audio yet, ordered by ready age descending; 2 (U2) the
 * rest, ordered by U = beta * K * R_occ - alpha * max(0, P - P_safe) / P_safe
 * descending.  order[0..n) receives the request indices in priority order
 * (U0, then U1, then U2; ties to the smaller index); the scan admits them in
 * that order and stops at the first one that does not fit the remaining
 * budgets: order[0 .. *num_admitted) is the batch.  classes[i] and
 * utility[i] (per request index; either may be NULL) give the class and, for
 * U2, the utility.  Fail-closed: if any P is NaN, every request is class 1
 * (ready-age order); if R_occ is NaN or a U2 request's K is negative, U2 is
 * ordered by ready age.  LS_EINVAL for p_safe <= 0, NaN weights or ages,
 * negative budgets or demands.
 */
ls_status ls_schedule_round(const ls_sched_stage *stage, int32_t n, const ls_sched_request *requests,
                            int32_t *order, int32_t *classes, double *utility, int32_t *num_admitted);

/*
 * Wait for all work on the current device (every stream), then return and
 * clear its device error word in *bits: the LS_DEVERR_* bits raised by every
 * call enqueued on the device before this one (0 when none met a bad index or
 * length).  The word is shared by all pools on the device.
 */
ls_status ls_device_errors(uint32_t *bits);

/* Message of the calling thread's most recent non-OK status ("" if none). */
const char *ls_last_error(void);

/* Library version string. */
const char *ls_version(void);

#ifdef __cplusplus
}
#endif

#endif /* LIVESERVE_KV_H */
