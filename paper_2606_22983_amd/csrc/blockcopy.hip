// Block stash (gather) and restore (scatter) kernels: the device leg of the
// HBM<->DRAM offload connector the KV manager drives (LiveServe §5 eviction to
// host DRAM, §5.2 speech-triggered preload back into HBM).  Pure byte copies
// at block granularity: one (layer, block) slab — the K and V tiles of every
// KV head — is contiguous both in the pool and in the staging array.
#include <algorithm>

#include "common.h"

namespace ls {

namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kCopyThreads = 256;
constexpr int kCopyUnroll = 8;      // 16-byte chunks in flight per thread
constexpr int kCopyWorkgroupsPerCu = 4;   // persistent grid: resident workgroups per CU

// Persistent copy: workgroup w copies the (block i, layer) slabs
// unit = w, w + grid, ... (unit = i * num_layers + layer), so a copy of any
// size is one short dispatch.  The grid is bounded (a few workgroups per CU)
// and every workgroup is resident at once, so a restore on a side stream
// leaves CU slots and dispatch to the decode stream instead of queueing
// millions of workgroups ahead of it.
// to_pool: staging -> pool (restore); otherwise pool -> staging (stash).
__global__ __launch_bounds__(kCopyThreads) void block_copy_kernel(
    uint8_t *__restrict__ pool, const int32_t *__restrict__ ids, uint8_t *__restrict__ staging,
    int64_t num_blocks, int32_t num_layers, int64_t slab_bytes, int64_t units, int32_t to_pool,
    unsigned int *err) {
    const int64_t chunks = slab_bytes / 16;
    for (int64_t unit = blockIdx.x; unit < units; unit += gridDim.x) {
        const int64_t i = unit / num_layers;
        const int32_t layer = (int32_t)(unit - i * num_layers);
        const int32_t id = ids[i];
        if (id < 0 || id >= num_blocks) {
            if (threadIdx.x == 0) flag_error(err, LS_DEVERR_BLOCK_ID);
            continue;
        }
        u32x4 *pool_slab = reinterpret_cast<u32x4 *>(pool + ((int64_t)layer * num_blocks + id) * slab_bytes);
        u32x4 *stage_slab = reinterpret_cast<u32x4 *>(staging + unit * slab_bytes);
        const u32x4 *src = to_pool ? stage_slab : pool_slab;
        u32x4 *dst = to_pool ? pool_slab : stage_slab;
        for (int64_t base = threadIdx.x; base < chunks; base += (int64_t)kCopyThreads * kCopyUnroll) {
            u32x4 v[kCopyUnroll];
#pragma unroll
            for (int u = 0; u < kCopyUnroll; ++u) {
                const int64_t c = base + (int64_t)u * kCopyThreads;
                if (c < chunks) v[u] = __builtin_nontemporal_load(src + c);
            }
#pragma unroll
            for (int u = 0; u < kCopyUnroll; ++u) {
                const int64_t c = base + (int64_t)u * kCopyThreads;
                if (c < chunks) __builtin_nontemporal_store(v[u], dst + c);
            }
        }
    }
}

}  // namespace

hipError_t launch_block_copy(const PoolGeom &p, int32_t n, const int32_t *ids, uint8_t *staging,
                             bool to_pool, unsigned int *err, hipStream_t stream) {
    if (n <= 0) return hipSuccess;
    const int64_t units = (int64_t)n * p.num_layers;
    const int64_t grid = std::min<int64_t>(units, (int64_t)kCopyWorkgroupsPerCu * stream_cus(p, stream));
    hipLaunchKernelGGL(block_copy_kernel, dim3((unsigned)grid), dim3(kCopyThreads), 0, stream,
                       reinterpret_cast<uint8_t *>(p.base), ids, staging, p.num_blocks,
                       p.num_layers, (int64_t)p.slab_bytes(), units, to_pool ? 1 : 0, err);
    return hipGetLastError();
}

}  // namespace ls
