// Paged-attention decode: one query token per session attends to its whole
// paged context — the batched decode step of the thinker/talker
// autoregressive decoders (LiveServe §2.1; continuous-batching decode loop of
// §6) over per-session block tables (block-level KV allocation, §5.1).
//
// Work decomposition (split-K): workgroup = (split k, KV head g, session s),
// covering tokens [k*T, (k+1)*T) of the session.  Its 4 wavefronts take the
// split's 16-token blocks round-robin; each keeps a wavefront-level online
// softmax state (running max m, running sum l, unnormalised output O) for the
// G query heads of group g.  The waves merge through LDS.  A session that fits
// one split is written directly; otherwise each split leaves (m, l, O) in the
// workspace and a second, small kernel merges the splits with the log-sum-exp
// rule (kernel boundaries order the two, so no cross-workgroup fences).
//
// Per block, the GQA group's contraction runs on MFMA 16x16 tiles:
//   S^T[16 tokens x 16 heads] = K[16 x D] . Q^T[D x 16]     (16x16x32 bf16)
//   O^T[16 dims   x 16 heads] += V^T[16 x 16 tokens] . P^T     (16x16x16 bf16)
// The MFMA accumulator layout of S^T (lane: head = lane%16, tokens 4*(lane/16)+i)
// is exactly the B-operand layout PV needs, so the probabilities never leave
// registers.  K tiles are token-major and V tiles dim-major in the pool, so both
// operands load straight from HBM into their MFMA lanes (16- and 8-byte
// coalesced buffer loads), prefetched two blocks ahead.  The split's block ids
// are read once into a register and broadcast with readlane, so the load
// stream never waits on an index fetch; a block that does not exist is loaded
// through a zero-size buffer descriptor (no memory traffic, no branch).  Heads
// beyond G in the 16-wide tile carry q = 0 and are never written.
#include "common.h"

namespace ls {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kDecThreads = 256;
constexpr int kDecWaves = kDecThreads / kWave;
constexpr int kMaxSplitTokens = 512;
constexpr int kMaxPerWave = kMaxSplitTokens / (kDecWaves * kBlock);   // blocks per wave per split
constexpr float kLog2e = 1.4426950408889634f;
constexpr int kBufferDword3 = 0x00020000;   // raw buffer, 32-bit data format
constexpr float kMaxFloor = -1.0e30f;       // initial running max (finite, below any score)

struct DecodeArgs {
    const uint16_t *pool;          // layer base
    int64_t num_blocks;
    int32_t num_kv_heads;
    int32_t group;                 // G = Hq / Hkv (<= 16)
    const uint16_t *q;             // [S][Hq][D]
    uint16_t *out;                 // [S][Hq][D]
    const int32_t *block_tables;   // [S][max_blocks]
    int32_t max_blocks;
    const int32_t *lens;           // tokens already in the pool
    int32_t appended;              // 1: the step's own token was appended at lens[s]
    float scale_log2;              // scale * log2(e)
    int32_t split_tokens;          // multiple of 64, at most kMaxSplitTokens
    int32_t max_splits;
    float *part_ml;                // [S][Hkv][max_splits][G][2]
    float *part_acc;               // [S][Hkv][max_splits][G][D]
    unsigned int *err;             // device error word
};

template <int D>
struct BlockRegs {
    u32x4 k[D / 32];               // K[token lane%16][8 dims of k-step ks]
    u32x2 v[D / 16];               // V^T[dim 16*dt + lane%16][tokens 4*(lane/16) .. +3]
};

__device__ __forceinline__ float wave_max_xor_16_32(float x) {
    x = fmaxf(x, __shfl_xor(x, 16));
    return fmaxf(x, __shfl_xor(x, 32));
}

__device__ __forceinline__ float wave_sum_xor_16_32(float x) {
    x += __shfl_xor(x, 16);
    return x + __shfl_xor(x, 32);
}

// Tokens of session s that attention covers (clipped to the table, flagged).
// Kept branch-free so that the compiler sees a wave-uniform value.
__device__ __forceinline__ int attended_len(const DecodeArgs &a, int s, bool may_flag) {
    const int raw = a.lens[s] + a.appended;
    const int cap = a.max_blocks * kBlock;
    if (may_flag && raw > cap) flag_error(a.err, LS_DEVERR_LENGTH);
    return min(raw, cap);
}

// Issue the loads of one block (blk < 0: a zero-size descriptor, nothing fetched).
template <int D>
__device__ __forceinline__ void load_block(BlockRegs<D> &r, const uint16_t *pool, int32_t num_kv_heads,
                                           int32_t g, int32_t blk, const int (&koff)[D / 32],
                                           const int (&voff)[D / 16]) {
    constexpr int kTileElems = kBlock * D;
    const bool valid = blk >= 0;
    const uint16_t *kt = pool + ((int64_t)(valid ? blk : 0) * 2 * num_kv_heads + g) * kTileElems;
    const uint16_t *vt = kt + (int64_t)num_kv_heads * kTileElems;
    const int bytes = valid ? kTileElems * 2 : 0;
    const __amdgpu_buffer_rsrc_t rk = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t *>(kt), 0, bytes, kBufferDword3);
    const __amdgpu_buffer_rsrc_t rv = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t *>(vt), 0, bytes, kBufferDword3);
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) r.k[ks] = __builtin_amdgcn_raw_buffer_load_b128(rk, koff[ks], 0, 0);
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt) r.v[dt] = __builtin_amdgcn_raw_buffer_load_b64(rv, voff[dt], 0, 0);
}

// Online-softmax update with one 16-token block held in registers.
template <int D>
__device__ __forceinline__ void process_block(BlockRegs<D> &r, const bf16x8 (&qop)[D / 32],
                                              int tok_base, int L, float scale_log2, int g4,
                                              float &m, float &lsum, f32x4 (&o)[D / 16]) {
    f32x4 sacc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks)
        sacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, r.k[ks]),
                                                       qop[ks], sacc, 0, 0, 0);
    const bool partial = tok_base + kBlock > L;     // some slot of this block is not a key
    float x[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        x[i] = sacc[i] * scale_log2;
        if (partial && tok_base + 4 * g4 + i >= L) x[i] = -INFINITY;
    }
    float bm = wave_max_xor_16_32(fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3])));
    const float m_new = fmaxf(m, bm);
    if (__any(m_new > m)) {
        const float alpha = __builtin_amdgcn_exp2f(m - m_new);
        lsum *= alpha;
#pragma unroll
        for (int dt = 0; dt < D / 16; ++dt) o[dt] *= alpha;
        m = m_new;
    }
    float p[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) p[i] = __builtin_amdgcn_exp2f(x[i] - m);
    lsum += (p[0] + p[1]) + (p[2] + p[3]);
    const uint32_t p01 = pack_bf16x2(p[0], p[1]);
    const uint32_t p23 = pack_bf16x2(p[2], p[3]);
    const s16x4 pb = __builtin_bit_cast(s16x4, make_uint2(p01, p23));
    if (partial) {
        // Slots at or past L may hold anything (NaN included): zero them so that
        // 0 * V cannot turn into NaN.
        const int valid = L - tok_base - 4 * g4;      // tokens of this lane's 4 that exist
        const uint32_t lo = valid >= 2 ? 0xFFFFFFFFu : (valid == 1 ? 0x0000FFFFu : 0u);
        const uint32_t hi = valid >= 4 ? 0xFFFFFFFFu : (valid == 3 ? 0x0000FFFFu : 0u);
#pragma unroll
        for (int dt = 0; dt < D / 16; ++dt) {
            r.v[dt].x &= lo;
            r.v[dt].y &= hi;
        }
    }
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt)
        o[dt] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(s16x4, r.v[dt]), pb,
                                                          o[dt], 0, 0, 0);
}

template <int D, int kDepth>
__global__ __launch_bounds__(kDecThreads) void decode_kernel(DecodeArgs a) {
    const int split = blockIdx.x;
    const int g = blockIdx.y;
    const int s = blockIdx.z;
    const int tid = threadIdx.x;
    const int G = a.group;
    const int hq_total = a.num_kv_heads * G;

    const int L = attended_len(a, s, split == 0 && tid == 0 && g == 0);
    if (L <= 0) {
        // Softmax over no key is undefined: write zeros and flag the length.
        if (split == 0) {
            if (tid == 0 && g == 0) flag_error(a.err, LS_DEVERR_LENGTH);
            for (int idx = tid; idx < G * D; idx += kDecThreads)
                a.out[((int64_t)s * hq_total + g * G) * D + idx] = 0;
        }
        return;
    }
    const int t0 = split * a.split_tokens;
    if (t0 >= L) return;
    const int t1 = min(L, t0 + a.split_tokens);
    const int nsplit = (L + a.split_tokens - 1) / a.split_tokens;
    const int blk0 = t0 / kBlock;
    const int nblk = (t1 + kBlock - 1) / kBlock - blk0;     // <= kMaxSplitTokens / 16

    const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
    const int lane = tid % kWave;
    const int c16 = lane & 15;
    const int g4 = lane >> 4;

    // Block ids of the split, one per lane; out-of-range ids become -1.
    int id_lane = -1;
    if (lane < nblk) {
        const int32_t b = a.block_tables[(int64_t)s * a.max_blocks + blk0 + lane];
        if (b >= 0 && b < a.num_blocks) {
            id_lane = b;
        } else if (wave == 0) {
            flag_error(a.err, LS_DEVERR_BLOCK_ID);
        }
    }
    const int my_n = wave < nblk ? (nblk - wave + kDecWaves - 1) / kDecWaves : 0;
    auto bid = [&](int it) -> int {
        const int idx = wave + it * kDecWaves;
        return idx < nblk ? __builtin_amdgcn_readlane(id_lane, idx) : -1;
    };

    // Q^T operand: column = query head c16 of the group (zero beyond G).
    bf16x8 qop[D / 32];
    {
        const bool active = c16 < G;
        const uint16_t *qrow = a.q + ((int64_t)s * hq_total + g * G + (active ? c16 : 0)) * D;
#pragma unroll
        for (int ks = 0; ks < D / 32; ++ks) {
            uint4 v = *reinterpret_cast<const uint4 *>(qrow + ks * 32 + g4 * 8);
            if (!active) v = make_uint4(0, 0, 0, 0);
            qop[ks] = __builtin_bit_cast(bf16x8, v);
        }
    }
    int koff[D / 32], voff[D / 16];
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) koff[ks] = (c16 * D + ks * 32 + g4 * 8) * 2;
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt) voff[dt] = ((dt * 16 + c16) * kBlock + g4 * 4) * 2;

    // The running max starts at a finite floor: a block whose keys are all
    // masked then leaves (m, l, O) unchanged instead of producing NaN.
    float m = kMaxFloor, lsum = 0.f;
    f32x4 o[D / 16];
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};

    // kDepth blocks in flight per wave.  The per-wave block sequence is fully
    // unrolled (at most kMaxPerWave blocks) with forward-only exits, so the
    // compiler sees straight-line code and waits only for the block it is about
    // to use.  A block with a bad id is processed as fully masked (0 keys).
    BlockRegs<D> r[kDepth];
    int bb[kDepth];
#pragma unroll
    for (int j = 0; j < kDepth; ++j) {
        bb[j] = bid(j);
        load_block<D>(r[j], a.pool, a.num_kv_heads, g, bb[j], koff, voff);
    }
#pragma unroll
    for (int i = 0; i < kMaxPerWave; ++i) {
        if (i >= my_n) break;
        const int j = i % kDepth;
        const int tb = (blk0 + wave + i * kDecWaves) * kBlock;
        process_block<D>(r[j], qop, tb, bb[j] >= 0 ? L : 0, a.scale_log2, g4, m, lsum, o);
        if (i + kDepth < kMaxPerWave) {
            bb[j] = bid(i + kDepth);
            load_block<D>(r[j], a.pool, a.num_kv_heads, g, bb[j], koff, voff);
        }
    }
    lsum = wave_sum_xor_16_32(lsum);

    // Merge the 4 waves through LDS.
    __shared__ float sm_m[kDecWaves][16];
    __shared__ float sm_l[kDecWaves][16];
    __shared__ float sm_o[kDecWaves][16][D];
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt)
#pragma unroll
        for (int i = 0; i < 4; ++i) sm_o[wave][c16][dt * 16 + g4 * 4 + i] = o[dt][i];
    if (g4 == 0) {
        sm_m[wave][c16] = m;
        sm_l[wave][c16] = lsum;
    }
    __syncthreads();

    const int64_t part = ((int64_t)s * a.num_kv_heads + g) * a.max_splits + split;
    for (int idx = tid; idx < G * D; idx += kDecThreads) {
        const int h = idx / D, d = idx % D;
        float M = sm_m[0][h];
#pragma unroll
        for (int w = 1; w < kDecWaves; ++w) M = fmaxf(M, sm_m[w][h]);
        float wsum = 0.f, acc = 0.f;
#pragma unroll
        for (int w = 0; w < kDecWaves; ++w) {
            const float e = __builtin_amdgcn_exp2f(sm_m[w][h] - M);
            wsum += e * sm_l[w][h];
            acc += e * sm_o[w][h][d];
        }
        if (nsplit == 1) {
            a.out[((int64_t)s * hq_total + g * G + h) * D + d] = (uint16_t)f32_to_bf16_bits(acc / wsum);
        } else {
            a.part_acc[(part * G + h) * D + d] = acc;
            if (d == 0) {
                a.part_ml[(part * G + h) * 2 + 0] = M;
                a.part_ml[(part * G + h) * 2 + 1] = wsum;
            }
        }
    }
}

// Log-sum-exp merge of the splits of every (session, KV head) with more than one.
template <int D>
__global__ __launch_bounds__(kDecThreads) void decode_combine_kernel(DecodeArgs a) {
    const int g = blockIdx.x;
    const int s = blockIdx.y;
    const int L = attended_len(a, s, false);
    if (L <= 0) return;
    const int nsplit = (L + a.split_tokens - 1) / a.split_tokens;
    if (nsplit <= 1) return;
    const int G = a.group;
    const int hq_total = a.num_kv_heads * G;
    const int64_t part = ((int64_t)s * a.num_kv_heads + g) * a.max_splits;
    for (int idx = threadIdx.x; idx < G * D; idx += kDecThreads) {
        const int h = idx / D, d = idx % D;
        float M = -INFINITY;
        for (int k = 0; k < nsplit; ++k) M = fmaxf(M, a.part_ml[((part + k) * G + h) * 2]);
        float wsum = 0.f, acc = 0.f;
        for (int k = 0; k < nsplit; ++k) {
            const float e = __builtin_amdgcn_exp2f(a.part_ml[((part + k) * G + h) * 2] - M);
            wsum += e * a.part_ml[((part + k) * G + h) * 2 + 1];
            acc += e * a.part_acc[((part + k) * G + h) * D + d];
        }
        a.out[((int64_t)s * hq_total + g * G + h) * D + d] = (uint16_t)f32_to_bf16_bits(acc / wsum);
    }
}

}  // namespace

DecodePlan plan_decode(const PoolGeom &p, int32_t num_sessions, int32_t num_q_heads,
                       int32_t max_blocks_per_session) {
    DecodePlan plan{};
    const int64_t max_tokens = (int64_t)max_blocks_per_session * kBlock;
    const int64_t work = (int64_t)num_sessions * p.num_kv_heads * max_tokens;
    // Aim for several workgroups per CU (256 CUs x 2 resident) when the batch is
    // large, smaller splits when it is not.
    int T = 512;
    if (work < 256LL * 2 * 4 * 512) T = 256;
    if (work < 256LL * 2 * 4 * 128) T = 128;
    plan.split_tokens = T;
    plan.max_splits = (int)((max_tokens + T - 1) / T);
    if (plan.max_splits < 1) plan.max_splits = 1;
    const int G = p.num_kv_heads > 0 ? num_q_heads / p.num_kv_heads : 0;
    const int64_t sg = (int64_t)num_sessions * p.num_kv_heads;
    auto pad = [](size_t b) { return (b + 255) & ~(size_t)255; };
    plan.ml_bytes = pad((size_t)sg * plan.max_splits * G * 2 * sizeof(float));
    plan.acc_bytes = pad((size_t)sg * plan.max_splits * G * p.head_dim * sizeof(float));
    return plan;
}

hipError_t launch_decode(const PoolGeom &p, int layer, int32_t num_sessions, int32_t num_q_heads,
                         const uint16_t *q, bool appended, const int32_t *block_tables,
                         int32_t max_blocks, const int32_t *context_lens, float scale,
                         uint16_t *out, void *workspace, const DecodePlan &plan,
                         unsigned int *err, hipStream_t stream) {
    DecodeArgs a;
    a.pool = p.layer_base(layer);
    a.num_blocks = p.num_blocks;
    a.num_kv_heads = p.num_kv_heads;
    a.group = num_q_heads / p.num_kv_heads;
    a.q = q;
    a.out = out;
    a.block_tables = block_tables;
    a.max_blocks = max_blocks;
    a.lens = context_lens;
    a.appended = appended ? 1 : 0;
    a.scale_log2 = scale * kLog2e;
    a.err = err;
    a.split_tokens = plan.split_tokens;
    a.max_splits = plan.max_splits;
    uint8_t *ws = static_cast<uint8_t *>(workspace);
    a.part_ml = reinterpret_cast<float *>(ws);
    a.part_acc = reinterpret_cast<float *>(ws + plan.ml_bytes);
    dim3 grid(plan.max_splits, p.num_kv_heads, num_sessions);
    if (p.head_dim == 128)
        hipLaunchKernelGGL((decode_kernel<128, 2>), grid, dim3(kDecThreads), 0, stream, a);
    else
        hipLaunchKernelGGL((decode_kernel<64, 2>), grid, dim3(kDecThreads), 0, stream, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || plan.max_splits == 1) return e;
    dim3 cgrid(p.num_kv_heads, num_sessions);
    if (p.head_dim == 128)
        hipLaunchKernelGGL(decode_combine_kernel<128>, cgrid, dim3(kDecThreads), 0, stream, a);
    else
        hipLaunchKernelGGL(decode_combine_kernel<64>, cgrid, dim3(kDecThreads), 0, stream, a);
    return hipGetLastError();
}

}  // namespace ls
