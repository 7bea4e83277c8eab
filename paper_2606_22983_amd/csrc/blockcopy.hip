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
// unit = w, w + grid, ... (unit = i * layer_count + (layer - layer_begin)) of
// the layers [layer_begin, layer_begin + layer_count), so a copy of any size is
// one short dispatch.  The grid is bounded (a few workgroups per CU) and every
// workgroup is resident at once, so a restore on a side stream leaves CU slots
// and dispatch to the decode stream instead of queueing millions of
// workgroups ahead of it.  In the staging array block i holds
// stage_block_slabs slabs and the slab of layer_begin is its stage_layer0-th
// (a full all-layer staging: num_layers and layer_begin; a compact copy of the
// layer range: layer_count and 0).
// to_pool: staging -> pool (restore); otherwise pool -> staging (stash).
__global__ __launch_bounds__(kCopyThreads) void block_copy_kernel(
    uint8_t *__restrict__ pool, const int32_t *__restrict__ ids, uint8_t *__restrict__ staging,
    int64_t num_blocks, int32_t layer_begin, int32_t layer_count, int32_t stage_block_slabs,
    int32_t stage_layer0, int64_t slab_bytes, int64_t units, int32_t to_pool, unsigned int *err) {
    const int64_t chunks = slab_bytes / 16;
    for (int64_t unit = blockIdx.x; unit < units; unit += gridDim.x) {
        const int64_t i = unit / layer_count;
        const int32_t lr = (int32_t)(unit - i * layer_count);
        const int32_t layer = layer_begin + lr;
        const int32_t id = ids[i];
        if (id < 0 || id >= num_blocks) {
            if (threadIdx.x == 0) flag_error(err, LS_DEVERR_BLOCK_ID);
            continue;
        }
        u32x4 *pool_slab = reinterpret_cast<u32x4 *>(pool + ((int64_t)layer * num_blocks + id) * slab_bytes);
        u32x4 *stage_slab = reinterpret_cast<u32x4 *>(
            staging + (i * stage_block_slabs + stage_layer0 + lr) * slab_bytes);
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
                             int32_t layer_begin, int32_t layer_count, int32_t stage_block_slabs,
                             int32_t stage_layer0, bool to_pool, int32_t max_workgroups,
                             unsigned int *err, hipStream_t stream) {
    if (n <= 0 || layer_count <= 0) return hipSuccess;
    const int64_t units = (int64_t)n * layer_count;
    int64_t grid = std::min<int64_t>(units, (int64_t)kCopyWorkgroupsPerCu * stream_cus(p, stream));
    if (max_workgroups > 0) grid = std::min<int64_t>(grid, max_workgroups);
    hipLaunchKernelGGL(block_copy_kernel, dim3((unsigned)grid), dim3(kCopyThreads), 0, stream,
                       reinterpret_cast<uint8_t *>(p.base), ids, staging, p.num_blocks, layer_begin,
                       layer_count, stage_block_slabs, stage_layer0, (int64_t)p.slab_bytes(), units,
                       to_pool ? 1 : 0, err);
    return hipGetLastError();
}

}  // namespace ls
