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
// Persistent grid, resident workgroups per CU.  The scatter (restore) is
// fastest with four; the gather (stash), whose reads are the scattered side,
// gains ~2% from six (all still resident: six waves of 80 registers per SIMD).
constexpr int kCopyWorkgroupsPerCu = 4;
constexpr int kGatherWorkgroupsPerCu = 6;
// A rate-bounded copy (a background preload beside live decode) runs one
// workgroup per CU: with four waves (one per SIMD, 80 registers each) it fits
// beside a decode workgroup (two waves per SIMD of 208 registers), whereas the
// full-rate grid holds four or six workgroups per CU and keeps decode off the
// CU until it ends.  Each workgroup copies a burst of slabs at the start of
// each window of the GPU's constant-frequency wall clock (the same boundaries
// for all), then sleeps until the next window.  Beside the thinker decode,
// copying at 0.5-0.6 TB/s (read + write): a steady trickle from single waves,
// or bursts staggered over the window, slowed the decode by ~28%; bursts of
// 4, 8, 16 and 32 slabs by 9-11%, 9-10%, 9-9.5% and 7-9%.  Longer, rarer
// bursts disturb fewer decode steps: a burst is up to 32 slabs, as many as
// keep the window within about a millisecond (so that a small copy at a low
// rate does not wait long for its first window), and at least one.
constexpr int kPacedWorkgroupsPerCu = 1;
constexpr int kPacedMaxBurst = 32;
constexpr double kPacedWindowSeconds = 1e-3;

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
// ticks_per_unit > 0 (paced copies): a workgroup starts its slabs at the
// boundaries of the global clock windows of ticks_per_unit ticks, at most
// `burst` slabs per window (a workgroup that falls behind waits for the
// next boundary instead of catching up).  The first burst waits at least one whole window,
// so that a copy of any size stays within its rate.  Every wait ends: the
// clock only moves forward.
template <int kThreads>
__global__ __launch_bounds__(kThreads) void block_copy_kernel(
    uint8_t *__restrict__ pool, const int32_t *__restrict__ ids, uint8_t *__restrict__ staging,
    int64_t num_blocks, int32_t layer_begin, int32_t layer_count, int32_t stage_block_slabs,
    int32_t stage_layer0, int64_t slab_bytes, int64_t units, int32_t to_pool, unsigned int *err,
    uint64_t ticks_per_unit, int32_t burst_slabs) {
    const int64_t chunks = slab_bytes / 16;
    uint64_t next = 0;
    int burst = 0;
    if (ticks_per_unit) {
        const uint64_t now = __builtin_amdgcn_s_memrealtime();
        next = (now / ticks_per_unit + 2) * ticks_per_unit;
    }
    for (int64_t unit = blockIdx.x; unit < units; unit += gridDim.x) {
        if (ticks_per_unit) {
            // Long sleeps while the boundary is far (s_sleep 127 is ~8k cycles,
            // a few microseconds; the clock ticks every ~10 ns), short ones near it.
            uint64_t now = __builtin_amdgcn_s_memrealtime();
            while ((int64_t)(now - next) < 0) {
                if (next - now > 512) __builtin_amdgcn_s_sleep(127);
                else __builtin_amdgcn_s_sleep(2);
                now = __builtin_amdgcn_s_memrealtime();
            }
            if (++burst == burst_slabs) {
                burst = 0;
                next += ticks_per_unit;
                if ((int64_t)(now - next) >= 0) next = (now / ticks_per_unit + 1) * ticks_per_unit;
            }
        }
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
        for (int64_t base = threadIdx.x; base < chunks; base += (int64_t)kThreads * kCopyUnroll) {
            u32x4 v[kCopyUnroll];
#pragma unroll
            for (int u = 0; u < kCopyUnroll; ++u) {
                const int64_t c = base + (int64_t)u * kThreads;
                if (c < chunks) v[u] = __builtin_nontemporal_load(src + c);
            }
#pragma unroll
            for (int u = 0; u < kCopyUnroll; ++u) {
                const int64_t c = base + (int64_t)u * kThreads;
                if (c < chunks) __builtin_nontemporal_store(v[u], dst + c);
            }
        }
    }
}

}  // namespace

hipError_t launch_block_copy(const PoolGeom &p, int32_t n, const int32_t *ids, uint8_t *staging,
                             int32_t layer_begin, int32_t layer_count, int32_t stage_block_slabs,
                             int32_t stage_layer0, bool to_pool, double max_gbps,
                             unsigned int *err, hipStream_t stream) {
    if (n <= 0 || layer_count <= 0) return hipSuccess;
    const int64_t units = (int64_t)n * layer_count;
    const int64_t slab = (int64_t)p.slab_bytes();
    const int64_t per_cu =
        max_gbps > 0.0 ? kPacedWorkgroupsPerCu : (to_pool ? kCopyWorkgroupsPerCu : kGatherWorkgroupsPerCu);
    const int64_t grid = std::min<int64_t>(units, per_cu * stream_cus(p, stream));
    uint64_t ticks = 0;
    int32_t burst = 1;
    if (max_gbps > 0.0) {
        // burst * grid slabs per window: the window lasts slab * burst * grid /
        // rate (the wall clock ticks wall_khz thousand times a second).
        const double per_burst = (double)slab * (double)grid;
        burst = (int32_t)std::min<double>(kPacedMaxBurst,
                                          std::max(1.0, std::floor(max_gbps * 1e9 * kPacedWindowSeconds / per_burst)));
        const double khz = p.wall_khz > 0 ? (double)p.wall_khz : 100000.0;
        const double secs = per_burst * burst / (max_gbps * 1e9);
        ticks = std::max<uint64_t>(1, (uint64_t)(secs * khz * 1e3));
    }
    hipLaunchKernelGGL(block_copy_kernel<kCopyThreads>, dim3((unsigned)grid), dim3(kCopyThreads), 0, stream,
                       reinterpret_cast<uint8_t *>(p.base), ids, staging, p.num_blocks, layer_begin,
                       layer_count, stage_block_slabs, stage_layer0, slab, units, to_pool ? 1 : 0, err, ticks,
                       burst);
    return hipGetLastError();
}

}  // namespace ls
