// C-ABI entry points: argument validation, pool bookkeeping and kernel
// launches.  Every check happens before anything is enqueued, so a non-OK
// status means the stream is untouched.
#include <cstdarg>
#include <cstdio>
#include <algorithm>
#include <cstring>
#include <mutex>
#include <new>
#include <vector>

#include "common.h"

struct ls_kv_pool {
    ls::PoolGeom geom;
};

namespace ls {

namespace {
// One error word per device, in the library's own code object, and the slot
// that ls_device_errors exchanges it into.
__device__ unsigned int g_device_errors = 0;
__device__ unsigned int g_device_errors_taken = 0;

// Read and clear the error word in one atomic step, so that a bit raised by a
// kernel running at the same time is either returned now or kept for the next
// query, never lost.
__global__ void take_errors_kernel(unsigned int *word, unsigned int *taken) {
    *taken = atomicExch(word, 0u);
}

struct ErrorWords {
    unsigned int *word = nullptr;
    unsigned int *taken = nullptr;
};

ErrorWords error_words() {
    static std::mutex mu;
    static ErrorWords addr[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return {};
    std::lock_guard<std::mutex> lock(mu);
    if (!addr[dev].word) {
        void *w = nullptr, *t = nullptr;
        if (hipGetSymbolAddress(&w, HIP_SYMBOL(g_device_errors)) == hipSuccess &&
            hipGetSymbolAddress(&t, HIP_SYMBOL(g_device_errors_taken)) == hipSuccess) {
            addr[dev].word = static_cast<unsigned int *>(w);
            addr[dev].taken = static_cast<unsigned int *>(t);
        }
    }
    return addr[dev];
}
}  // namespace

unsigned int *device_error_word() { return error_words().word; }

namespace {
// Split-K scratch of paged_attn_decode_static: a fixed buffer in the
// library's code object, one per GPU, so that the call allocates nothing.  In
// host code `scratch` only names the symbol; its device address (different on
// every GPU) comes from hipGetSymbolAddress with that GPU current.
constexpr size_t kDecodeScratchBytes = LS_DECODE_STATIC_SCRATCH_BYTES;
__device__ __align__(256) uint8_t scratch[kDecodeScratchBytes];

// Device address of this GPU's scratch (resolved once per device), or null.
void *decode_scratch() {
    static std::mutex mu;
    static void *addr[64] = {};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return nullptr;
    std::lock_guard<std::mutex> lock(mu);
    if (!addr[dev]) {
        void *ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess) {
            (void)hipGetLastError();
            return nullptr;
        }
        addr[dev] = ptr;
    }
    return addr[dev];
}
}  // namespace

int stream_cus(const PoolGeom &p, hipStream_t stream) {
    const int dev_cus = p.num_cus > 0 ? p.num_cus : 256;
    if (!stream) return dev_cus;
    uint32_t mask[32] = {};                    // up to 1024 CUs
    if (hipExtStreamGetCUMask(stream, 32, mask) != hipSuccess) {
        (void)hipGetLastError();               // leave no sticky error behind
        return dev_cus;
    }
    int n = 0;
    for (uint32_t w : mask) n += __builtin_popcount(w);
    return n > 0 && n < dev_cus ? n : dev_cus;
}

namespace {

thread_local char t_last_error[512] = "";

ls_status fail(ls_status st, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(t_last_error, sizeof t_last_error, fmt, ap);
    va_end(ap);
    return st;
}

ls_status hip_fail(hipError_t e, const char *what) {
    return fail(LS_EHIP, "%s: %s", what, hipGetErrorString(e));
}

bool supported_head_dim(int32_t d) { return d == 64 || d == 128; }
bool supported_group(int32_t g) { return g == 1 || g == 2 || g == 4 || g == 8; }

ls_status check_pool(const ls_kv_pool *pool) {
    if (!pool) return fail(LS_EINVAL, "pool handle is NULL");
    return LS_OK;
}

ls_status check_heads(const PoolGeom &p, int32_t num_q_heads) {
    if (num_q_heads <= 0 || num_q_heads % p.num_kv_heads != 0)
        return fail(LS_EINVAL, "num_q_heads (%d) must be a positive multiple of num_kv_heads (%d)",
                    num_q_heads, p.num_kv_heads);
    if (!supported_group(num_q_heads / p.num_kv_heads))
        return fail(LS_EUNSUPPORTED, "query heads per KV head must be 1, 2, 4 or 8 (got %d)",
                    num_q_heads / p.num_kv_heads);
    return LS_OK;
}

// Host check of a restore/stash id list: range and distinctness.
ls_status check_ids_host(const PoolGeom &p, int32_t n, const int32_t *ids) {
    std::vector<unsigned char> seen((size_t)p.num_blocks, 0);
    for (int32_t i = 0; i < n; ++i) {
        const int32_t b = ids[i];
        if (b < 0 || b >= p.num_blocks)
            return fail(LS_EINVAL, "block id %d at position %d is outside [0, %lld)", b, i,
                        (long long)p.num_blocks);
        if (seen[(size_t)b]) return fail(LS_EINVAL, "block id %d appears twice", b);
        seen[(size_t)b] = 1;
    }
    return LS_OK;
}

// Copy the slabs of layers [lb, lb + lc) of n blocks between the pool and a
// block-major all-layer staging array (device, or pinned host through the
// caller's ring).
ls_status copy_blocks(ls_kv_pool *pool, int32_t lb, int32_t lc, int32_t n, const int32_t *block_ids,
                      const int32_t *block_ids_host, void *staging, size_t staging_bytes,
                      int32_t staging_on_host, void *ring_ptr, size_t ring_bytes,
                      double max_gbps, bool to_pool, hipStream_t stream) {
    if (ls_status st = check_pool(pool)) return st;
    const PoolGeom &p = pool->geom;
    if (lb < 0 || lc < 1 || lb > p.num_layers - lc)
        return fail(LS_EINVAL, "layer range [%d, %d + %d) outside [0, %d)", lb, lb, lc, p.num_layers);
    if (n < 0) return fail(LS_EINVAL, "n must be >= 0");
    if (!(max_gbps >= 0.0) || max_gbps > 1e9)
        return fail(LS_EINVAL, "max_gbps must be a number >= 0 (got %g)", max_gbps);
    if (n == 0) return LS_OK;
    if (!block_ids || !staging) return fail(LS_EINVAL, "block_ids and staging must not be NULL");
    if (n > p.num_blocks) return fail(LS_EINVAL, "n (%d) exceeds num_blocks", n);
    const size_t per_block = p.slab_bytes() * (size_t)p.num_layers;   // staging stride of a block
    const size_t range = p.slab_bytes() * (size_t)lc;                   // bytes of the layer range
    if (staging_bytes / per_block < (size_t)n)
        return fail(LS_ENOMEM, "staging_bytes (%zu) < %d blocks x %zu bytes", staging_bytes, n, per_block);
    uint8_t *ring = static_cast<uint8_t *>(ring_ptr);
    if (staging_on_host) {
        if (!ring || ring_bytes < range)
            return fail(LS_ENOMEM, "host staging needs a device ring of at least %zu bytes", range);
        if (reinterpret_cast<uintptr_t>(ring) % 16 != 0)
            return fail(LS_EINVAL, "the ring must be 16-byte aligned");
    }
    if (block_ids_host)
        if (ls_status st = check_ids_host(p, n, block_ids_host)) return st;
    unsigned int *err = device_error_word();
    if (!err) return fail(LS_EHIP, "cannot resolve the device error word");
    if (!staging_on_host) {
        hipError_t e = launch_block_copy(p, n, block_ids, static_cast<uint8_t *>(staging), lb, lc,
                                         p.num_layers, lb, to_pool, max_gbps, err, stream);
        return e == hipSuccess ? LS_OK : hip_fail(e, "block copy launch");
    }
    // Whole blocks per chunk, in id order, all on the caller's stream.  The
    // ring holds the layer range of each block compactly; a range narrower
    // than all layers moves as a strided (2D) copy of one row per block.
    const int32_t chunk = (int32_t)std::min<size_t>(ring_bytes / range, (size_t)n);
    uint8_t *host = static_cast<uint8_t *>(staging) + p.slab_bytes() * (size_t)lb;
    for (int32_t i0 = 0; i0 < n; i0 += chunk) {
        const int32_t cnt = (n - i0) < chunk ? (n - i0) : chunk;
        uint8_t *h = host + per_block * (size_t)i0;
        hipError_t e;
        if (to_pool) {
            e = range == per_block
                    ? hipMemcpyAsync(ring, h, range * (size_t)cnt, hipMemcpyHostToDevice, stream)
                    : hipMemcpy2DAsync(ring, range, h, per_block, range, cnt, hipMemcpyHostToDevice, stream);
            if (e != hipSuccess) return hip_fail(e, "restore host-to-device copy");
            e = launch_block_copy(p, cnt, block_ids + i0, ring, lb, lc, lc, 0, true, max_gbps, err,
                                  stream);
            if (e != hipSuccess) return hip_fail(e, "restore scatter launch");
        } else {
            e = launch_block_copy(p, cnt, block_ids + i0, ring, lb, lc, lc, 0, false, max_gbps, err,
                                  stream);
            if (e != hipSuccess) return hip_fail(e, "stash gather launch");
            e = range == per_block
                    ? hipMemcpyAsync(h, ring, range * (size_t)cnt, hipMemcpyDeviceToHost, stream)
                    : hipMemcpy2DAsync(h, per_block, ring, range, range, cnt, hipMemcpyDeviceToHost, stream);
            if (e != hipSuccess) return hip_fail(e, "stash device-to-host copy");
        }
    }
    return LS_OK;
}

// Host check of decode lengths: every session attends to at least one key,
// and its keys (the appended one included) fit its block table.
ls_status check_decode_lens_host(int32_t S, const int32_t *lens, int32_t appended, int32_t max_blocks) {
    const int64_t cap = (int64_t)max_blocks * kBlock;
    for (int32_t s = 0; s < S; ++s) {
        const int64_t L = (int64_t)lens[s] + appended;
        if (lens[s] < 0 || L < 1)
            return fail(LS_EINVAL, "session %d: context length %d leaves no key to attend", s, lens[s]);
        if (L > cap)
            return fail(LS_EINVAL, "session %d: %lld keys do not fit its %d-block table", s, (long long)L,
                        max_blocks);
    }
    return LS_OK;
}

// Host check of prefill lengths (n_s, c_s): turns within max_new_len and the
// table, adding up to total_new_tokens.
ls_status check_prefill_lens_host(int32_t S, const int32_t *lens, int32_t total, int32_t max_new_len,
                                  int32_t max_blocks) {
    const int64_t cap = (int64_t)max_blocks * kBlock;
    int64_t sum = 0;
    for (int32_t s = 0; s < S; ++s) {
        const int32_t n = lens[2 * s], c = lens[2 * s + 1];
        if (n < 0 || c < 0) return fail(LS_EINVAL, "session %d: negative length (n %d, c %d)", s, n, c);
        if (n > max_new_len)
            return fail(LS_EINVAL, "session %d: turn of %d tokens exceeds max_new_len (%d)", s, n, max_new_len);
        if ((int64_t)n + c > cap)
            return fail(LS_EINVAL, "session %d: %lld keys do not fit its %d-block table", s,
                        (long long)n + c, max_blocks);
        sum += n;
    }
    if (sum != total)
        return fail(LS_EINVAL, "turn lengths add up to %lld, not total_new_tokens (%d)", (long long)sum, total);
    return LS_OK;
}

}  // namespace

// Message for ls_last_error() from code outside this file (the KV manager).
void set_last_error(const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(t_last_error, sizeof t_last_error, fmt, ap);
    va_end(ap);
}

}  // namespace ls

using namespace ls;

extern "C" {

size_t ls_kv_pool_bytes(int32_t num_layers, int64_t num_blocks, int32_t num_kv_heads,
                        int32_t head_dim, int32_t block_size) {
    if (num_layers <= 0 || num_blocks <= 0 || num_kv_heads <= 0 || head_dim <= 0 || block_size <= 0)
        return 0;
    const unsigned __int128 bytes = (unsigned __int128)num_layers * (unsigned __int128)num_blocks *
                                    2u * (unsigned)num_kv_heads * (unsigned)block_size *
                                    (unsigned)head_dim * 2u;
    if (bytes > (unsigned __int128)SIZE_MAX) return 0;
    return (size_t)bytes;
}

ls_status kv_pool_create(const ls_kv_pool_desc *desc, ls_kv_pool **out) {
    if (!desc || !out) return fail(LS_EINVAL, "desc and out must not be NULL");
    *out = nullptr;
    if (desc->num_layers <= 0 || desc->num_kv_heads <= 0 || desc->num_blocks <= 0)
        return fail(LS_EINVAL, "num_layers, num_kv_heads and num_blocks must be positive");
    if (desc->block_size != kBlock)
        return fail(LS_EUNSUPPORTED, "block_size must be %d (got %d)", kBlock, desc->block_size);
    if (!supported_head_dim(desc->head_dim))
        return fail(LS_EUNSUPPORTED, "head_dim must be 64 or 128 (got %d)", desc->head_dim);
    if (desc->num_blocks > INT32_MAX)
        return fail(LS_EINVAL, "num_blocks must fit in int32 (block ids are int32)");
    if (!desc->kv_base) return fail(LS_EINVAL, "kv_base must not be NULL");
    if (reinterpret_cast<uintptr_t>(desc->kv_base) % 256 != 0)
        return fail(LS_EINVAL, "kv_base must be 256-byte aligned");
    const size_t need = ls_kv_pool_bytes(desc->num_layers, desc->num_blocks, desc->num_kv_heads,
                                         desc->head_dim, desc->block_size);
    if (need == 0) return fail(LS_EINVAL, "pool size overflows");
    if (desc->kv_bytes < need)
        return fail(LS_ENOMEM, "kv_bytes (%zu) is smaller than the layout needs (%zu)",
                    desc->kv_bytes, need);
    int dev = 0, cus = 0, wall_khz = 0;
    if (hipGetDevice(&dev) != hipSuccess) dev = -1;
    if (dev >= 0 && hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
        cus = 0;
    if (dev >= 0 && hipDeviceGetAttribute(&wall_khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess)
        wall_khz = 0;
    (void)hipGetLastError();
    ls_kv_pool *pool = new (std::nothrow) ls_kv_pool;
    if (!pool) return fail(LS_ENOMEM, "out of host memory");
    pool->geom.num_layers = desc->num_layers;
    pool->geom.num_kv_heads = desc->num_kv_heads;
    pool->geom.head_dim = desc->head_dim;
    pool->geom.num_blocks = desc->num_blocks;
    pool->geom.base = static_cast<uint16_t *>(desc->kv_base);
    pool->geom.device = dev;
    pool->geom.num_cus = cus;
    pool->geom.wall_khz = wall_khz;
    *out = pool;
    return LS_OK;
}

ls_status kv_pool_destroy(ls_kv_pool *pool) {
    delete pool;
    return LS_OK;
}

size_t ls_decode_workspace_bytes(const ls_kv_pool *pool, int32_t num_sessions,
                                 int32_t num_q_heads, int32_t max_blocks_per_session) {
    if (!pool || num_sessions <= 0 || max_blocks_per_session <= 0 || num_q_heads <= 0) return 0;
    return plan_decode(pool->geom, num_sessions, num_q_heads, max_blocks_per_session).total();
}

ls_status paged_attn_decode(ls_kv_pool *pool, int32_t layer, int32_t num_sessions,
                            int32_t num_q_heads, const void *q, const void *k_new,
                            const void *v_new, const int32_t *block_tables,
                            int32_t max_blocks_per_session, const int32_t *context_lens,
                            const int32_t *context_lens_host, float scale, void *out,
                            void *workspace, size_t workspace_bytes, hipStream_t stream) {
    if (ls_status st = check_pool(pool)) return st;
    const PoolGeom &p = pool->geom;
    if (layer < 0 || layer >= p.num_layers)
        return fail(LS_EINVAL, "layer %d outside [0, %d)", layer, p.num_layers);
    if (num_sessions < 0) return fail(LS_EINVAL, "num_sessions must be >= 0");
    if (ls_status st = check_heads(p, num_q_heads)) return st;
    if (num_sessions == 0) return LS_OK;
    if (!q || !block_tables || !context_lens || !out || !workspace)
        return fail(LS_EINVAL, "q, block_tables, context_lens, out and workspace must not be NULL");
    if ((k_new == nullptr) != (v_new == nullptr))
        return fail(LS_EINVAL, "k_new and v_new must both be given or both be NULL");
    if (max_blocks_per_session <= 0) return fail(LS_EINVAL, "max_blocks_per_session must be > 0");
    if (!(scale > 0.f) || scale != scale) return fail(LS_EINVAL, "scale must be a positive number");
    if (context_lens_host)
        if (ls_status st = check_decode_lens_host(num_sessions, context_lens_host, k_new ? 1 : 0,
                                                  max_blocks_per_session))
            return st;
    const DecodePlan plan = plan_decode(p, num_sessions, num_q_heads, max_blocks_per_session);
    if (!plan.supported)
        return fail(LS_EUNSUPPORTED, "batch of %d sessions with %d blocks each exceeds the decode "
                    "limits (2048 sessions, 16384 blocks per session)", num_sessions, max_blocks_per_session);
    if (workspace_bytes < plan.total())
        return fail(LS_ENOMEM, "workspace_bytes (%zu) < required (%zu)", workspace_bytes, plan.total());
    unsigned int *err = device_error_word();
    if (!err) return fail(LS_EHIP, "cannot resolve the device error word");
    // The step's own K/V row is written by the decode kernel (no separate append launch).
    hipError_t e = launch_decode(p, layer, num_sessions, num_q_heads, static_cast<const uint16_t *>(q),
                                 static_cast<const uint16_t *>(k_new), static_cast<const uint16_t *>(v_new),
                                 block_tables, max_blocks_per_session, context_lens, context_lens_host,
                                 scale, static_cast<uint16_t *>(out), workspace, plan, err, stream);
    return e == hipSuccess ? LS_OK : hip_fail(e, "decode launch");
}

ls_status ls_decode_schedule(const ls_kv_pool *pool, int32_t num_sessions, int32_t num_q_heads,
                             int32_t max_blocks_per_session, const int32_t *context_lens_host, int32_t appended,
                             hipStream_t stream, int32_t *split_tokens, int32_t *host_planned, int32_t *merge) {
    if (ls_status st = check_pool(pool)) return st;
    const PoolGeom &p = pool->geom;
    if (num_sessions <= 0 || max_blocks_per_session <= 0 || (appended != 0 && appended != 1))
        return fail(LS_EINVAL, "num_sessions and max_blocks_per_session must be > 0, appended 0 or 1");
    if (!split_tokens || !host_planned || !merge) return fail(LS_EINVAL, "output pointers must not be NULL");
    if (ls_status st = check_heads(p, num_q_heads)) return st;
    const DecodePlan plan = plan_decode(p, num_sessions, num_q_heads, max_blocks_per_session);
    if (!plan.supported) return fail(LS_EUNSUPPORTED, "batch exceeds the decode limits");
    if (context_lens_host)
        if (ls_status st = check_decode_lens_host(num_sessions, context_lens_host, appended, max_blocks_per_session))
            return st;
    const DecodeSchedule sc = decode_schedule(p, num_sessions, context_lens_host, appended, plan, stream);
    *split_tokens = sc.split_tokens;
    *host_planned = sc.host_planned ? 1 : 0;
    *merge = sc.merge ? 1 : 0;
    return LS_OK;
}

ls_status paged_attn_decode_static(ls_kv_pool *pool, int32_t layer, int32_t num_sessions,
                                   int32_t num_q_heads, const void *q, const void *k_new,
                                   const void *v_new, const int32_t *block_tables,
                                   int32_t max_blocks_per_session, const int32_t *context_lens,
                                   const int32_t *context_lens_host, float scale, void *out,
                                   hipStream_t stream) {
    if (ls_status st = check_pool(pool)) return st;
    if (num_sessions > 0 && max_blocks_per_session > 0 && num_q_heads > 0) {
        const size_t need = ls_decode_workspace_bytes(pool, num_sessions, num_q_heads, max_blocks_per_session);
        if (need > kDecodeScratchBytes)
            return fail(LS_ENOMEM, "this batch needs %zu bytes of split scratch; the static buffer holds %zu",
                        need, kDecodeScratchBytes);
    }
    void *ws = decode_scratch();
    if (!ws) return fail(LS_EHIP, "cannot resolve the static decode scratch on this device");
    return paged_attn_decode(pool, layer, num_sessions, num_q_heads, q, k_new, v_new, block_tables,
                             max_blocks_per_session, context_lens, context_lens_host, scale, out, ws,
                             kDecodeScratchBytes, stream);
}

ls_status paged_attn_prefill(ls_kv_pool *pool, int32_t layer, int32_t num_sessions,
                             int32_t num_q_heads, const void *q, const void *k_new,
                             const void *v_new, const int32_t *cu_new_lens,
                             const int32_t *reused_lens, const int32_t *lens_host,
                             int32_t total_new_tokens, int32_t max_new_len,
                             const int32_t *block_tables, int32_t max_blocks_per_session,
                             float scale, void *out, void *workspace, size_t workspace_bytes,
                             hipStream_t stream) {
    if (ls_status st = check_pool(pool)) return st;
    const PoolGeom &p = pool->geom;
    if (layer < 0 || layer >= p.num_layers)
        return fail(LS_EINVAL, "layer %d outside [0, %d)", layer, p.num_layers);
    if (num_sessions < 0 || total_new_tokens < 0 || max_new_len < 0)
        return fail(LS_EINVAL, "num_sessions, total_new_tokens and max_new_len must be >= 0");
    if (ls_status st = check_heads(p, num_q_heads)) return st;
    if (num_sessions == 0 || total_new_tokens == 0) return LS_OK;
    if (!q || !cu_new_lens || !reused_lens || !block_tables || !out)
        return fail(LS_EINVAL, "q, cu_new_lens, reused_lens, block_tables and out must not be NULL");
    if ((k_new == nullptr) != (v_new == nullptr))
        return fail(LS_EINVAL, "k_new and v_new must both be given or both be NULL");
    if (max_blocks_per_session <= 0) return fail(LS_EINVAL, "max_blocks_per_session must be > 0");
    if (max_new_len > total_new_tokens)
        return fail(LS_EINVAL, "max_new_len (%d) exceeds total_new_tokens (%d)", max_new_len,
                    total_new_tokens);
    if (!(scale > 0.f) || scale != scale) return fail(LS_EINVAL, "scale must be a positive number");
    if (workspace && workspace_bytes < LS_PREFILL_WORKSPACE_BYTES)
        return fail(LS_ENOMEM, "prefill workspace of %zu bytes, %zu needed", workspace_bytes,
                    LS_PREFILL_WORKSPACE_BYTES);
    if (reinterpret_cast<uintptr_t>(workspace) % 16)
        return fail(LS_EINVAL, "prefill workspace must be 16-byte aligned");
    if (lens_host)
        if (ls_status st = check_prefill_lens_host(num_sessions, lens_host, total_new_tokens, max_new_len,
                                                   max_blocks_per_session))
            return st;
    unsigned int *err = device_error_word();
    if (!err) return fail(LS_EHIP, "cannot resolve the device error word");
    if (k_new) {
        hipError_t e = launch_append_prefill(p, layer, num_sessions, total_new_tokens, max_new_len,
                                             static_cast<const uint16_t *>(k_new),
                                             static_cast<const uint16_t *>(v_new), cu_new_lens,
                                             reused_lens, block_tables, max_blocks_per_session, err,
                                             stream);
        if (e != hipSuccess) return hip_fail(e, "append launch");
    }
    hipError_t e = launch_prefill(p, layer, num_sessions, num_q_heads, static_cast<const uint16_t *>(q),
                                  cu_new_lens, reused_lens, lens_host, total_new_tokens, max_new_len, block_tables,
                                  max_blocks_per_session, scale, static_cast<uint16_t *>(out),
                                  static_cast<uint32_t *>(workspace), err, stream);
    return e == hipSuccess ? LS_OK : hip_fail(e, "prefill launch");
}

ls_status kv_blocks_stash(ls_kv_pool *pool, int32_t n, const int32_t *block_ids,
                          const int32_t *block_ids_host, void *staging, size_t staging_bytes,
                          int32_t staging_on_host, void *ring, size_t ring_bytes,
                          double max_gbps, hipStream_t stream) {
    return copy_blocks(pool, 0, pool ? pool->geom.num_layers : 1, n, block_ids, block_ids_host, staging,
                       staging_bytes, staging_on_host, ring, ring_bytes, max_gbps, false, stream);
}

ls_status kv_blocks_restore(ls_kv_pool *pool, int32_t n, const int32_t *block_ids,
                            const int32_t *block_ids_host, const void *staging,
                            size_t staging_bytes, int32_t staging_on_host, void *ring,
                            size_t ring_bytes, double max_gbps, hipStream_t stream) {
    return copy_blocks(pool, 0, pool ? pool->geom.num_layers : 1, n, block_ids, block_ids_host,
                       const_cast<void *>(staging), staging_bytes, staging_on_host, ring, ring_bytes,
                       max_gbps, true, stream);
}

ls_status kv_blocks_restore_layers(ls_kv_pool *pool, int32_t layer_begin, int32_t layer_count, int32_t n,
                                   const int32_t *block_ids, const int32_t *block_ids_host,
                                   const void *staging, size_t staging_bytes, int32_t staging_on_host,
                                   void *ring, size_t ring_bytes, double max_gbps,
                                   hipStream_t stream) {
    return copy_blocks(pool, layer_begin, layer_count, n, block_ids, block_ids_host,
                       const_cast<void *>(staging), staging_bytes, staging_on_host, ring, ring_bytes,
                       max_gbps, true, stream);
}

ls_status ls_device_errors(uint32_t *bits) {
    if (!bits) return fail(LS_EINVAL, "bits must not be NULL");
    const ErrorWords w = error_words();
    if (!w.word) return fail(LS_EHIP, "cannot resolve the device error word");
    hipError_t e = hipDeviceSynchronize();
    if (e != hipSuccess) return hip_fail(e, "device synchronize");
    hipLaunchKernelGGL(take_errors_kernel, dim3(1), dim3(1), 0, nullptr, w.word, w.taken);
    e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, "error word exchange launch");
    unsigned int v = 0;
    e = hipMemcpy(&v, w.taken, sizeof v, hipMemcpyDeviceToHost);
    if (e != hipSuccess) return hip_fail(e, "read device error word");
    *bits = v;
    return LS_OK;
}

const char *ls_last_error(void) { return t_last_error; }

const char *ls_version(void) { return "liveserve_kv 0.1.0 (gfx950)"; }

}  // extern "C"
