// Internal declarations shared by the library's translation units (host API,
// kernels).  Nothing here is visible through the C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

#include "liveserve_kv.h"

namespace ls {

constexpr int kBlock = 16;          // tokens per KV block (every supported geometry)
constexpr int kWave = 64;           // CDNA wavefront width

// Host-side description of a pool: what kv_pool_create recorded.
struct PoolGeom {
    int32_t num_layers;
    int32_t num_kv_heads;
    int32_t head_dim;
    int64_t num_blocks;
    uint16_t *base;                 // bf16 bit patterns
    int device;
    int num_cus;                    // compute units of that device (0 if unknown)
    int wall_khz;                   // frequency of its constant wall clock (0 if unknown)

    // Elements of one (kv, head) tile and of one (layer, block) slab.
    int64_t tile_elems() const { return (int64_t)kBlock * head_dim; }
    int64_t slab_elems() const { return 2 * (int64_t)num_kv_heads * tile_elems(); }
    size_t slab_bytes() const { return (size_t)slab_elems() * sizeof(uint16_t); }
    uint16_t *layer_base(int layer) const {
        return base + (int64_t)layer * num_blocks * slab_elems();
    }
};

// Compute units a kernel launched on `stream` may use: the popcount of the
// stream's CU mask when it is narrower than the device (a stream created with
// hipExtStreamCreateWithCUMask), else the device's CU count.  Persistent grids
// are sized from it, so a kernel confined to part of the GPU does not queue
// workgroups that cannot become resident.
int stream_cus(const PoolGeom &p, hipStream_t stream);

// Device address of this device's error word (LS_DEVERR_* bits), or null if
// the runtime could not resolve it.  Kernels receive it as an argument.
unsigned int *device_error_word();

// Split-K planning shared by paged_attn_decode and its workspace query.
struct DecodePlan {
    int split_tokens;               // tokens per split (multiple of 64)
    int max_splits;                 // splits of the longest possible session
    bool supported;                 // false when a session could need too many splits
    size_t ml_bytes;                // fp32 [S][Hkv][max_splits][G][2]
    size_t acc_bytes;               // fp32 [S][Hkv][max_splits][G][D]
    size_t total() const { return ml_bytes + acc_bytes; }
};
DecodePlan plan_decode(const PoolGeom &p, int32_t num_sessions, int32_t num_q_heads,
                       int32_t max_blocks_per_session);

// Zeroes n (<= 64) 32-bit counters on the stream with a one-wave kernel (not
// a memset, so that the call can be captured in a graph).
hipError_t launch_clear_counters(uint32_t *counters, int n, hipStream_t stream);

// Kernel launchers (each returns the hipError_t of its launch).
// Copies the slabs of layers [layer_begin, layer_begin + layer_count) of blocks
// ids[0..n): staging block i holds stage_block_slabs slabs, layer_begin's is
// its stage_layer0-th.
// max_gbps > 0: a paced copy of at most that many GB/s of payload.
hipError_t launch_block_copy(const PoolGeom &p, int32_t n, const int32_t *ids, uint8_t *staging,
                             int32_t layer_begin, int32_t layer_count, int32_t stage_block_slabs,
                             int32_t stage_layer0, bool to_pool, double max_gbps,
                             unsigned int *err, hipStream_t stream);
hipError_t launch_append_prefill(const PoolGeom &p, int layer, int32_t num_sessions, int32_t total_tokens,
                                 int32_t max_new_len, const uint16_t *k_new, const uint16_t *v_new,
                                 const int32_t *cu_new_lens, const int32_t *reused_lens,
                                 const int32_t *block_tables, int32_t max_blocks, unsigned int *err,
                                 hipStream_t stream);
// With k_new / v_new (both non-null) the step's own token is attended from
// them and written to its pool slot by the decode kernel itself.
// The schedule paged_attn_decode runs for a batch: tokens per split, planned
// on the host (from context_lens_host) or in the kernel, merge kernel or not.
struct DecodeSchedule {
    int split_tokens;
    bool host_planned;
    bool merge;
};
DecodeSchedule decode_schedule(const PoolGeom &p, int32_t num_sessions, const int32_t *context_lens_host,
                               int32_t appended, const DecodePlan &plan, hipStream_t stream);

// With context_lens_host (the same lengths on the host) the split-K schedule
// is planned on the host; the split merge is launched only if some session is
// split.
hipError_t launch_decode(const PoolGeom &p, int layer, int32_t num_sessions, int32_t num_q_heads,
                         const uint16_t *q, const uint16_t *k_new, const uint16_t *v_new,
                         const int32_t *block_tables,
                         int32_t max_blocks, const int32_t *context_lens, const int32_t *context_lens_host,
                         float scale, uint16_t *out, void *workspace, const DecodePlan &plan,
                         unsigned int *err, hipStream_t stream);
hipError_t launch_prefill(const PoolGeom &p, int layer, int32_t num_sessions, int32_t num_q_heads,
                          const uint16_t *q, const int32_t *cu_new_lens,
                          const int32_t *reused_lens, const int32_t *lens_host, int32_t total_tokens,
                          int32_t max_new_len, const int32_t *block_tables, int32_t max_blocks,
                          float scale, uint16_t *out, uint32_t *queue, unsigned int *err, hipStream_t stream);

// ---------------------------------------------------------------------------
// Device helpers
// ---------------------------------------------------------------------------
__device__ __forceinline__ void flag_error(unsigned int *err, unsigned int bits) {
    if (err) atomicOr(err, bits);
}

// Round-to-nearest-even fp32 -> bf16 bits (inputs here are finite or +-inf).
__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) {
    return (uint32_t)__builtin_bit_cast(unsigned short, (__bf16)f);
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    return f32_to_bf16_bits(lo) | (f32_to_bf16_bits(hi) << 16);
}

}  // namespace ls
