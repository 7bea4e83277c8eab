// KV append of a next turn's tokens (prefill over reused context, §5): write
// their K and V rows into their pool slots before attention reads them.  Slot
// of logical token t of session s: block block_tables[s][t / 16], offset
// t % 16; K tiles are chunk-major ([D/8][16 tokens][8 dims]), V tiles
// dim-major ([D][16 tokens]).  (The decode step's own token is written by the
// decode kernel.)
#include "common.h"

namespace ls {

namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kAppendThreads = 256;

// Workgroup (session s, j, KV head g) appends the turn's tokens of the pool
// blocks j, j + bps, ... that the turn touches (bps workgroups per session:
// normally one block each; a turn longer than max_new_len still gets every
// block).  Per block it writes 16-byte chunks.  A K chunk is 8 dims of one
// token, i.e. 16 contiguous bytes of that token's k_new row.  A V chunk is 8
// tokens of one dim, gathered from 8 rows through LDS.  The turn's first and
// last blocks may be shared with other tokens (the reused context before it,
// nothing after it): K chunks of other tokens are left alone, and a V chunk
// that mixes the turn's tokens with others is read, merged and written back
// (no other workgroup writes this tile in the launch).
template <int D>
__global__ __launch_bounds__(kAppendThreads) void append_kernel(
    uint16_t *__restrict__ layer_pool, int64_t num_blocks, int32_t num_kv_heads,
    const uint16_t *__restrict__ k_new, const uint16_t *__restrict__ v_new,
    const int32_t *__restrict__ block_tables, int32_t max_blocks, const int32_t *__restrict__ cu,
    const int32_t *__restrict__ ctx, int32_t total_tokens, int32_t blocks_per_session, unsigned int *err) {
    __shared__ __attribute__((aligned(16))) uint16_t sv[kBlock][D];
    const int s = blockIdx.x / blocks_per_session;
    const int j = blockIdx.x % blocks_per_session;
    const int g = blockIdx.y;
    const int tid = threadIdx.x;
    const int c = ctx[s];
    const int n = cu[s + 1] - cu[s];
    // Nothing to append, or lengths that do not fit the token arrays (flagged by prefill).
    if (n <= 0 || c < 0 || cu[s] < 0 || cu[s + 1] > total_tokens) return;
    const int first = c / kBlock, last = (c + n - 1) / kBlock;
    constexpr int kChunks = D / 8 * kBlock;                     // 16-byte chunks per tile
    const int64_t tile = (int64_t)kBlock * D;
    for (int jb = first + j; jb <= last; jb += blocks_per_session) {
        if (jb >= max_blocks) {
            if (tid == 0) flag_error(err, LS_DEVERR_LENGTH);
            return;
        }
        const int32_t blk = block_tables[(int64_t)s * max_blocks + jb];
        if (blk < 0 || blk >= num_blocks) {
            if (tid == 0) flag_error(err, LS_DEVERR_BLOCK_ID);
            continue;
        }
        const int t_lo = max(c, jb * kBlock) - jb * kBlock;        // the turn's slots of this block: [t_lo, t_hi)
        const int t_hi = min(c + n, (jb + 1) * kBlock) - jb * kBlock;
        const int64_t row0 = (int64_t)cu[s] + (jb * kBlock - c);   // new-token index of slot 0 (may be negative)
        uint16_t *ktile = layer_pool + ((int64_t)blk * 2 * num_kv_heads + g) * tile;
        uint16_t *vtile = ktile + (int64_t)num_kv_heads * tile;

        // K: chunk ci = (dim chunk ci / 16, token ci % 16), contiguous across threads.
        for (int ci = tid; ci < kChunks; ci += kAppendThreads) {
            const int t = ci % kBlock;
            if (t < t_lo || t >= t_hi) continue;
            const u32x4 v =
                *reinterpret_cast<const u32x4 *>(k_new + ((row0 + t) * num_kv_heads + g) * D + (ci / kBlock) * 8);
            *reinterpret_cast<u32x4 *>(ktile + ci * 8) = v;
        }
        // V: the block's rows into LDS, then chunk ci = (dim ci / 2, tokens 8 * (ci % 2) ..).
        __syncthreads();                                        // the previous block's LDS reads are done
        for (int ci = tid; ci < kChunks; ci += kAppendThreads) {
            const int t = ci / (D / 8), d8 = ci % (D / 8);
            if (t < t_lo || t >= t_hi) continue;
            *reinterpret_cast<u32x4 *>(&sv[t][d8 * 8]) =
                *reinterpret_cast<const u32x4 *>(v_new + ((row0 + t) * num_kv_heads + g) * D + d8 * 8);
        }
        __syncthreads();
        for (int ci = tid; ci < 2 * D; ci += kAppendThreads) {
            const int d = ci / 2, t0 = (ci % 2) * 8;
            const int lo = max(t_lo, t0), hi = min(t_hi, t0 + 8);
            if (lo >= hi) continue;
            u32x4 *dst = reinterpret_cast<u32x4 *>(vtile + (int64_t)d * kBlock + t0);
            u32x4 w = (lo == t0 && hi == t0 + 8) ? u32x4{0u, 0u, 0u, 0u} : *dst;
            for (int t = lo; t < hi; ++t) {
                const uint32_t half = sv[t][d];
                const int k = (t - t0) >> 1, sh = ((t - t0) & 1) * 16;
                w[k] = (w[k] & ~(0xFFFFu << sh)) | (half << sh);
            }
            *dst = w;
        }
    }
}

}  // namespace

hipError_t launch_append_prefill(const PoolGeom &p, int layer, int32_t num_sessions, int32_t total_tokens,
                                 int32_t max_new_len, const uint16_t *k_new, const uint16_t *v_new,
                                 const int32_t *cu_new_lens, const int32_t *reused_lens,
                                 const int32_t *block_tables, int32_t max_blocks, unsigned int *err,
                                 hipStream_t stream) {
    if (num_sessions <= 0 || max_new_len <= 0) return hipSuccess;
    // A turn of n tokens touches at most (n + 15) / 16 + 1 blocks (one more
    // when it starts inside a block).
    const int32_t bps = (max_new_len + kBlock - 1) / kBlock + 1;
    const int64_t grid = (int64_t)num_sessions * bps;
    if (grid > 0x7FFFFFFFLL) return hipErrorInvalidConfiguration;
    const dim3 g((unsigned)grid, (unsigned)p.num_kv_heads);
    if (p.head_dim == 128)
        hipLaunchKernelGGL(append_kernel<128>, g, dim3(kAppendThreads), 0, stream, p.layer_base(layer),
                           p.num_blocks, p.num_kv_heads, k_new, v_new, block_tables, max_blocks, cu_new_lens,
                           reused_lens, total_tokens, bps, err);
    else
        hipLaunchKernelGGL(append_kernel<64>, g, dim3(kAppendThreads), 0, stream, p.layer_base(layer),
                           p.num_blocks, p.num_kv_heads, k_new, v_new, block_tables, max_blocks, cu_new_lens,
                           reused_lens, total_tokens, bps, err);
    return hipGetLastError();
}

}  // namespace ls
