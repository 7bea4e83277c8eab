// KV append of a next turn's tokens (prefill over reused context, §5): write
// their K and V rows into their pool slots before attention reads them.  Slot
// of logical token t of session s: block block_tables[s][t / 16], offset
// t % 16; K tiles are chunk-major ([D/8][16 tokens][8 dims]), V tiles
// dim-major.  (The decode step's own token is written by the decode kernel.)
#include "common.h"

namespace ls {

namespace {

// One workgroup per (token, KV head); one thread per head dimension.
__global__ void append_kernel(uint16_t *__restrict__ layer_pool, int64_t num_blocks,
                              int32_t num_kv_heads, int32_t head_dim, int32_t num_sessions,
                              const uint16_t *__restrict__ k_new,
                              const uint16_t *__restrict__ v_new,
                              const int32_t *__restrict__ block_tables, int32_t max_blocks,
                              const int32_t *__restrict__ cu_new_lens,    // cu[S+1]
                              const int32_t *__restrict__ reused_lens,
                              unsigned int *err) {
    const int32_t tok = blockIdx.x;
    const int32_t g = blockIdx.y;
    // session of this token: largest s with cu[s] <= tok
    int lo = 0, hi = num_sessions - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (cu_new_lens[mid] <= tok) lo = mid; else hi = mid - 1;
    }
    const int32_t s = lo;
    const int32_t pos = reused_lens[s] + (tok - cu_new_lens[s]);
    const int32_t jb = pos / kBlock;
    if (pos < 0 || jb >= max_blocks) {
        if (threadIdx.x == 0) flag_error(err, LS_DEVERR_LENGTH);
        return;
    }
    const int32_t blk = block_tables[(int64_t)s * max_blocks + jb];
    if (blk < 0 || blk >= num_blocks) {
        if (threadIdx.x == 0) flag_error(err, LS_DEVERR_BLOCK_ID);
        return;
    }
    const int32_t o = pos % kBlock;
    const int64_t tile = (int64_t)kBlock * head_dim;
    uint16_t *ktile = layer_pool + (((int64_t)blk * 2 + 0) * num_kv_heads + g) * tile;
    uint16_t *vtile = layer_pool + (((int64_t)blk * 2 + 1) * num_kv_heads + g) * tile;
    const int64_t src = ((int64_t)tok * num_kv_heads + g) * head_dim;
    for (int d = threadIdx.x; d < head_dim; d += blockDim.x) {
        ktile[((d >> 3) * kBlock + o) * 8 + (d & 7)] = k_new[src + d];
        vtile[d * kBlock + o] = v_new[src + d];
    }
}

}  // namespace

hipError_t launch_append_prefill(const PoolGeom &p, int layer, int32_t num_sessions,
                                 int32_t total_tokens, const uint16_t *k_new,
                                 const uint16_t *v_new, const int32_t *cu_new_lens,
                                 const int32_t *reused_lens, const int32_t *block_tables,
                                 int32_t max_blocks, unsigned int *err, hipStream_t stream) {
    if (total_tokens <= 0) return hipSuccess;
    hipLaunchKernelGGL(append_kernel, dim3(total_tokens, p.num_kv_heads), dim3(p.head_dim), 0,
                       stream, p.layer_base(layer), p.num_blocks, p.num_kv_heads, p.head_dim,
                       num_sessions, k_new, v_new, block_tables, max_blocks, cu_new_lens,
                       reused_lens, err);
    return hipGetLastError();
}

}  // namespace ls
