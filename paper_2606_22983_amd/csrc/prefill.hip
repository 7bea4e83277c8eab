// Next-turn (chunked) prefill over reused multi-turn context: the n_s tokens of
// a session's new turn attend causally to its c_s cached tokens plus the turn's
// own earlier tokens (LiveServe §5: reusing LLM-stage KV avoids re-prefilling
// history; §3: current-turn prefill).  Row j of the turn sees keys
// 0 .. c_s + j (bottom-right causal alignment); the turn's K/V has already been
// appended to the pool, so every key is read through the block table.
//
// Workgroup = (q-tile, KV head g, session s).  The tile packs the GQA group into
// the row dimension: 128 rows = (128 / G) new tokens x G query heads sharing
// KV head g, so each K/V tile staged in LDS feeds 128 query rows.  Four
// wavefronts own 32 rows each (two 16-row MFMA tiles).  Keys stream in tiles
// of 64 (four 16-token blocks): global -> registers -> LDS (double buffered,
// one barrier per tile), K token-major with an XOR swizzle, V dim-major.
//
//   S^T[16 keys x 16 rows] = K[16 x D] . Q^T          (MFMA 16x16x32 bf16)
//   O^T[16 dims x 16 rows] += V^T[16 x 32 keys] . P^T  (MFMA 16x16x32 bf16)
// The S^T accumulator layout (lane: row = lane%16, keys 4*(lane/16)+i) is the
// B-operand layout of the PV product, so P stays in registers (rounded to bf16);
// softmax statistics stay in fp32.
#include "common.h"

namespace ls {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kPreThreads = 256;
constexpr int kBufferDword3P = 0x00020000;   // raw buffer, 32-bit data format
constexpr int kPreRows = 128;            // query rows per workgroup
constexpr int kKeyTile = 64;             // keys per staged tile (4 blocks)
constexpr float kLog2eP = 1.4426950408889634f;

struct PrefillArgs {
    const uint16_t *pool;          // layer base
    int64_t num_blocks;
    int32_t num_kv_heads;
    int32_t group;
    const uint16_t *q;             // [T][Hq][D]
    uint16_t *out;                 // [T][Hq][D]
    const int32_t *cu;             // [S+1]
    const int32_t *ctx;            // [S]
    const int32_t *block_tables;
    int32_t max_blocks;
    float scale_log2;
    unsigned int *err;
};

__device__ __forceinline__ float xmax16_32(float x) {
    x = fmaxf(x, __shfl_xor(x, 16));
    return fmaxf(x, __shfl_xor(x, 32));
}
__device__ __forceinline__ float xsum16_32(float x) {
    x += __shfl_xor(x, 16);
    return x + __shfl_xor(x, 32);
}

template <int D>
struct TileRegs {
    static constexpr int kChunks = (2 * kKeyTile * D * 2) / (16 * kPreThreads);  // 16-byte chunks per thread
    u32x4 c[kChunks];
};

// Issue the loads of one key tile (K then V of 4 blocks) into registers.  Blocks
// past the session's keys (or with an id outside the pool) are read through a
// zero-size buffer descriptor: no memory traffic, zeros returned.
template <int D>
__device__ __forceinline__ void load_tile(TileRegs<D> &r, const PrefillArgs &a, const int32_t *table,
                                          int nblk_valid, int g, int kt, int tid) {
    constexpr int kChunksPerTile = kBlock * D * 2 / 16;      // 16-byte chunks in a K (or V) tile
    constexpr int kPerKV = 4 * kChunksPerTile;               // chunks of 4 K tiles
    constexpr int kTileElems = kBlock * D;
#pragma unroll
    for (int u = 0; u < TileRegs<D>::kChunks; ++u) {
        const int c = tid + u * kPreThreads;
        const int is_v = __builtin_amdgcn_readfirstlane(c >= kPerKV ? 1 : 0);
        const int cc = c - is_v * kPerKV;
        const int bi = __builtin_amdgcn_readfirstlane(cc / kChunksPerTile);   // uniform per wave
        const int within = cc % kChunksPerTile;
        const int jb = kt * 4 + bi;
        int32_t b = jb < nblk_valid ? table[jb] : -1;
        const bool valid = b >= 0 && b < a.num_blocks;
        const uint16_t *base = a.pool + (((int64_t)(valid ? b : 0) * 2 + is_v) * a.num_kv_heads + g) * kTileElems;
        const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<uint16_t *>(base), 0, valid ? kTileElems * 2 : 0, kBufferDword3P);
        r.c[u] = __builtin_amdgcn_raw_buffer_load_b128(rsrc, within * 16, 0, 0);
    }
}

// Write a loaded tile to LDS.  Slots at or past the session's last key (kv_len)
// are zeroed here so that masked keys contribute exact zeros (never NaN) to PV.
template <int D>
__device__ __forceinline__ void store_tile(TileRegs<D> &r, uint8_t *lds_k, uint8_t *lds_v, int tid,
                                           int kt, int kv_len) {
    constexpr int kChunksPerTile = kBlock * D * 2 / 16;
    constexpr int kPerKV = 4 * kChunksPerTile;
    constexpr int kRowChunks = D / 8;
    const bool tail = (kt + 1) * kKeyTile > kv_len;
#pragma unroll
    for (int u = 0; u < TileRegs<D>::kChunks; ++u) {
        const int c = tid + u * kPreThreads;
        u32x4 v = r.c[u];
        if (c < kPerKV) {
            const int bi = c / kChunksPerTile;
            const int within = c % kChunksPerTile;
            const int token = within / kRowChunks;
            const int ch = within % kRowChunks;
            if (tail && kt * kKeyTile + bi * kBlock + token >= kv_len) v = u32x4{0u, 0u, 0u, 0u};
            const int slot = ch ^ (token & (kRowChunks - 1));
            *reinterpret_cast<u32x4 *>(lds_k + bi * (kBlock * D * 2) + token * (D * 2) + slot * 16) = v;
        } else {
            const int cv = c - kPerKV;
            if (tail) {
                // V chunk: 8 consecutive tokens of one dim
                const int bi = cv / kChunksPerTile;
                const int t0 = kt * kKeyTile + bi * kBlock + (cv & 1) * 8;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int t = t0 + 2 * e;
                    const uint32_t mask = t + 1 < kv_len ? 0xFFFFFFFFu : (t < kv_len ? 0x0000FFFFu : 0u);
                    v[e] &= mask;
                }
            }
            *reinterpret_cast<u32x4 *>(lds_v + cv * 16) = v;
        }
    }
}

template <int D>
__global__ __launch_bounds__(kPreThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void prefill_kernel(PrefillArgs a) {
    constexpr int KS = D / 32;           // 32-dim k-steps of QK
    constexpr int NDT = D / 16;          // 16-dim output tiles
    constexpr int kRowChunks = D / 8;
    constexpr int kTileBytes = kBlock * D * 2;
    __shared__ __attribute__((aligned(16))) uint8_t lds[2][2][4 * kTileBytes];

    const int qt = blockIdx.x;
    const int g = blockIdx.y;
    const int s = blockIdx.z;
    const int G = a.group;
    const int qtok = kPreRows / G;       // new tokens per tile
    const int n = a.cu[s + 1] - a.cu[s];
    const int j0 = qt * qtok;
    if (j0 >= n) return;
    const int c = a.ctx[s];
    const int j_last = min(j0 + qtok, n) - 1;
    const int kv_len = c + n;
    int nblk_valid = (kv_len + kBlock - 1) / kBlock;
    if (nblk_valid > a.max_blocks) {
        nblk_valid = a.max_blocks;
        if (threadIdx.x == 0) flag_error(a.err, LS_DEVERR_LENGTH);
    }
    const int kv_end = c + j_last + 1;                    // keys this tile can see
    const int ntiles = (kv_end + kKeyTile - 1) / kKeyTile;

    const int tid = threadIdx.x;
    const int wave = tid / kWave;
    const int lane = tid % kWave;
    const int c16 = lane & 15;
    const int g4 = lane >> 4;
    const int hq_total = a.num_kv_heads * G;

    // Rows of this lane (one per 16-row tile): r = wave*32 + rt*16 + c16.
    int row_lim[2];
    int64_t row_out[2];
    bool row_ok[2];
    bf16x8 qop[2][KS];
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
        const int r = wave * 32 + rt * 16 + c16;
        const int jl = j0 + r / G;
        const int h = r % G;
        row_ok[rt] = jl < n;
        const int jc = min(jl, n - 1);
        row_lim[rt] = c + jc;
        const int64_t tok = (int64_t)a.cu[s] + jc;
        row_out[rt] = (tok * hq_total + g * G + h) * D;
        const uint16_t *qrow = a.q + row_out[rt];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
            qop[rt][ks] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4 *>(qrow + ks * 32 + g4 * 8));
    }
    const int wave_lim_min = c + min(j0 + (wave * 32) / G, n - 1);

    float m[2] = {-INFINITY, -INFINITY};
    float lsum[2] = {0.f, 0.f};
    f32x4 o[2][NDT];
#pragma unroll
    for (int rt = 0; rt < 2; ++rt)
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) o[rt][dt] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int32_t *table = a.block_tables + (int64_t)s * a.max_blocks;
    TileRegs<D> regs;
    load_tile<D>(regs, a, table, nblk_valid, g, 0, tid);

    for (int kt = 0; kt < ntiles; ++kt) {
        uint8_t *lk = lds[kt & 1][0];
        uint8_t *lv = lds[kt & 1][1];
        store_tile<D>(regs, lk, lv, tid, kt, kv_len);
        __syncthreads();
        load_tile<D>(regs, a, table, kt + 1 < ntiles ? nblk_valid : 0, g, kt + 1, tid);

        // ---- S^T = K Q^T for 4 key sub-tiles x 2 row tiles
        f32x4 sacc[2][4];
#pragma unroll
        for (int sub = 0; sub < 4; ++sub) {
            sacc[0][sub] = f32x4{0.f, 0.f, 0.f, 0.f};
            sacc[1][sub] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                const int ch = ks * 4 + g4;
                const int slot = ch ^ (c16 & (kRowChunks - 1));
                const bf16x8 kop = __builtin_bit_cast(
                    bf16x8, *reinterpret_cast<const uint4 *>(lk + sub * kTileBytes + c16 * (D * 2) + slot * 16));
                sacc[0][sub] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kop, qop[0][ks], sacc[0][sub], 0, 0, 0);
                sacc[1][sub] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kop, qop[1][ks], sacc[1][sub], 0, 0, 0);
            }
        }

        // ---- online softmax per row
        const int key0 = kt * kKeyTile;
        const bool diag = key0 + kKeyTile - 1 > wave_lim_min;
        bf16x8 pop[2][2];
#pragma unroll
        for (int rt = 0; rt < 2; ++rt) {
            float x[4][4];
            float bm = -INFINITY;
#pragma unroll
            for (int sub = 0; sub < 4; ++sub)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    float v = sacc[rt][sub][i] * a.scale_log2;
                    if (diag && key0 + sub * 16 + g4 * 4 + i > row_lim[rt]) v = -INFINITY;
                    x[sub][i] = v;
                    bm = fmaxf(bm, v);
                }
            bm = xmax16_32(bm);
            const float m_new = fmaxf(m[rt], bm);
            if (__any(m_new > m[rt])) {
                const float alpha = __builtin_amdgcn_exp2f(m[rt] - m_new);
                lsum[rt] *= alpha;
#pragma unroll
                for (int dt = 0; dt < NDT; ++dt) o[rt][dt] *= alpha;
                m[rt] = m_new;
            }
            float ps = 0.f;
            float p[4][4];
#pragma unroll
            for (int sub = 0; sub < 4; ++sub)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    p[sub][i] = __builtin_amdgcn_exp2f(x[sub][i] - m[rt]);
                    ps += p[sub][i];
                }
            lsum[rt] += ps;
#pragma unroll
            for (int k2 = 0; k2 < 2; ++k2) {
                const uint4 w = make_uint4(pack_bf16x2(p[2 * k2][0], p[2 * k2][1]),
                                           pack_bf16x2(p[2 * k2][2], p[2 * k2][3]),
                                           pack_bf16x2(p[2 * k2 + 1][0], p[2 * k2 + 1][1]),
                                           pack_bf16x2(p[2 * k2 + 1][2], p[2 * k2 + 1][3]));
                pop[rt][k2] = __builtin_bit_cast(bf16x8, w);
            }
        }

        // ---- O^T += V^T P^T
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) {
#pragma unroll
            for (int k2 = 0; k2 < 2; ++k2) {
                const uint2 va = *reinterpret_cast<const uint2 *>(lv + (2 * k2) * kTileBytes + (dt * 16 + c16) * 32 + g4 * 8);
                const uint2 vb = *reinterpret_cast<const uint2 *>(lv + (2 * k2 + 1) * kTileBytes + (dt * 16 + c16) * 32 + g4 * 8);
                const bf16x8 vop = __builtin_bit_cast(bf16x8, make_uint4(va.x, va.y, vb.x, vb.y));
                o[0][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vop, pop[0][k2], o[0][dt], 0, 0, 0);
                o[1][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vop, pop[1][k2], o[1][dt], 0, 0, 0);
            }
        }
    }

    // ---- normalise and write
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
        const float inv = 1.f / xsum16_32(lsum[rt]);
        if (!row_ok[rt]) continue;
        uint16_t *orow = a.out + row_out[rt];
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) {
            const uint2 w = make_uint2(pack_bf16x2(o[rt][dt][0] * inv, o[rt][dt][1] * inv),
                                       pack_bf16x2(o[rt][dt][2] * inv, o[rt][dt][3] * inv));
            *reinterpret_cast<uint2 *>(orow + dt * 16 + g4 * 4) = w;
        }
    }
}

}  // namespace

hipError_t launch_prefill(const PoolGeom &p, int layer, int32_t num_sessions, int32_t num_q_heads,
                          const uint16_t *q, const int32_t *cu_new_lens,
                          const int32_t *reused_lens, int32_t max_new_len,
                          const int32_t *block_tables, int32_t max_blocks, float scale,
                          uint16_t *out, unsigned int *err, hipStream_t stream) {
    if (num_sessions <= 0 || max_new_len <= 0) return hipSuccess;
    PrefillArgs a;
    a.pool = p.layer_base(layer);
    a.num_blocks = p.num_blocks;
    a.num_kv_heads = p.num_kv_heads;
    a.group = num_q_heads / p.num_kv_heads;
    a.q = q;
    a.out = out;
    a.cu = cu_new_lens;
    a.ctx = reused_lens;
    a.block_tables = block_tables;
    a.max_blocks = max_blocks;
    a.scale_log2 = scale * kLog2eP;
    a.err = err;
    const int qtok = kPreRows / a.group;
    dim3 grid((max_new_len + qtok - 1) / qtok, p.num_kv_heads, num_sessions);
    if (p.head_dim == 128)
        hipLaunchKernelGGL(prefill_kernel<128>, grid, dim3(kPreThreads), 0, stream, a);
    else
        hipLaunchKernelGGL(prefill_kernel<64>, grid, dim3(kPreThreads), 0, stream, a);
    return hipGetLastError();
}

}  // namespace ls
