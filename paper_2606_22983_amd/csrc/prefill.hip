// Next-turn (chunked) prefill over reused multi-turn context: the n_s tokens of
// a session's new turn attend causally to its c_s cached tokens plus the turn's
// own earlier tokens (LiveServe §5: reusing LLM-stage KV avoids re-prefilling
// history; §3: current-turn prefill).  Row j of the turn sees keys
// 0 .. c_s + j (bottom-right causal alignment); the turn's K/V has already been
// appended to the pool, so every key is read through the block table.
//
// Workgroup = (session, KV head g, query tile).  The tile packs the GQA group
// into the row dimension: 256 rows = (256 / G) new tokens x G query heads
// sharing KV head g, so each K/V tile staged in LDS feeds 256 query rows.
// Eight wavefronts own 32 rows each (two 16-row MFMA tiles).  Keys stream in
// tiles of 64 (four 16-token blocks): buffer loads into registers two tiles
// ahead, then LDS (double buffered, one barrier per tile).
//
//   S^T[16 keys x 16 rows] = K[16 x D] . Q^T          (MFMA 16x16x32 bf16)
//   O^T[16 dims x 16 rows] += V^T[16 x 32 keys] . P^T  (MFMA 16x16x32 bf16)
// The S^T accumulator layout (lane: row = lane%16, keys 4*(lane/16)+i) is the
// B-operand layout of the PV product, so P stays in registers (rounded to
// bf16; the row sums add up the same rounded values); softmax statistics stay
// in fp32.  A row's running max is raised (and its O and l
// rescaled) only when a tile's max exceeds it by more than 2^8, which keeps
// every probability at most 256 and makes rescales rare.
//
// Workgroups run longest session first and, within a session, latest query
// tile first (longest-processing-time order against the tail).  Consecutive
// query tiles of one (session, KV head) are placed on the same XCD so that
// they share its L2.
#include "common.h"

namespace ls {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kPreThreads = 512;
constexpr int kPreRows = 256;            // query rows per workgroup
constexpr int kKeyTile = 64;             // keys per staged tile (4 blocks)
constexpr int kBufferDword3P = 0x00020000;   // raw buffer, 32-bit data format
constexpr float kLog2eP = 1.4426950408889634f;
constexpr float kRescaleSlack = 8.0f;    // log2 units a row max may lag behind
constexpr int kXcds = 8;                 // workgroups are dispatched round-robin over XCDs
constexpr int kXcdChunk = 8;             // consecutive items kept on one XCD
constexpr int kMaxSortSessions = 128;    // larger batches run in index order

struct PrefillArgs {
    const uint16_t *pool;          // layer base
    int64_t num_blocks;
    int32_t num_kv_heads;
    int32_t group;
    int32_t num_sessions;
    int32_t qtiles;                // query tiles of the longest turn
    const uint16_t *q;             // [T][Hq][D]
    uint16_t *out;                 // [T][Hq][D]
    const int32_t *cu;             // [S+1]
    const int32_t *ctx;            // [S]
    const int32_t *block_tables;
    int32_t max_blocks;
    float scale_log2;
    unsigned int *err;
};

// NaN-propagating maxima (v_maximum3_f32 on gfx950: no operand canonicalisation).
__device__ __forceinline__ float fmax3(float a, float b, float c) {
    return __builtin_elementwise_maximum(__builtin_elementwise_maximum(a, b), c);
}

// Max over the four lanes l, l^16, l^32, l^48 (the lanes holding one row's
// scores) with the gfx950 row-swap permutes: VALU only, no LDS round trip.
__device__ __forceinline__ float xmax16_32(float x) {
    const unsigned int u = __float_as_uint(x);
    const auto a = __builtin_amdgcn_permlane32_swap(u, u, false, false);
    const float y = __builtin_elementwise_maximum(__uint_as_float(a[0]), __uint_as_float(a[1]));
    const unsigned int w = __float_as_uint(y);
    const auto b = __builtin_amdgcn_permlane16_swap(w, w, false, false);
    return __builtin_elementwise_maximum(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

__device__ __forceinline__ float xsum16_32(float x) {
    const unsigned int u = __float_as_uint(x);
    const auto a = __builtin_amdgcn_permlane32_swap(u, u, false, false);
    const float y = __uint_as_float(a[0]) + __uint_as_float(a[1]);
    const unsigned int w = __float_as_uint(y);
    const auto b = __builtin_amdgcn_permlane16_swap(w, w, false, false);
    return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// Thread -> 16-byte chunk assignment of one 64-key tile (4 blocks of K, then
// 4 blocks of V).  K: chunk c = tid + u * threads, block c / kCpt, the chunk's
// bytes are token-major (token = within / (D/8)).  V tiles are dim-major
// ([D][16 tokens], two chunks per dim): each wave covers 32 dims, lanes 0..31
// the first 8 tokens, lanes 32..63 the last 8.  With two V chunks per thread
// (D = 128) a thread holds the same (dim, half) of blocks 2*k2 and 2*k2+1.
template <int D>
struct TileCfg {
    static constexpr int kTileBytes = kBlock * D * 2;                  // one block's K (or V)
    static constexpr int kCpt = kTileBytes / 16;                       // chunks per block tile
    static constexpr int kPerThread = 2 * 4 * kCpt / kPreThreads;      // 4 (D=128) or 2 (D=64)
    static constexpr int kKPer = kPerThread / 2;
    static constexpr int kVPer = kPerThread / 2;
    static_assert(kCpt % 64 == 0, "a wave's chunks must stay inside one block tile");
    static_assert(kVPer == 1 || 4 * kCpt == 2 * kPreThreads, "V pairing needs 2 chunks per thread");
};

template <int D>
struct TileRegs {
    u32x4 c[TileCfg<D>::kPerThread];
};

// Block-table entries behind one thread's chunks of a key tile (uniform per
// wave: every wave's chunks of one load lie in one block).
template <int D>
struct TileIds {
    int32_t b[TileCfg<D>::kPerThread];
};

template <int D>
__device__ __forceinline__ void v_chunk_coords(int tid, int e, int &bi, int &dim, int &h) {
    using C = TileCfg<D>;
    int within;
    if constexpr (C::kVPer == 2) {
        bi = 2 * (tid / C::kCpt) + e;
        within = tid % C::kCpt;
    } else {
        bi = tid / C::kCpt;
        within = tid % C::kCpt;
    }
    dim = (within >> 6) * 32 + (within & 31);
    h = (within >> 5) & 1;
}

// Entry jb of a session's block table, or -1 outside [0, nv).  The table
// does not change during a launch, so it is read through the constant address
// space: a scalar load, whose wait does not also wait for the tile loads in
// flight.  The clamped index keeps the read inside the table row.
__device__ __forceinline__ int32_t table_entry(const int32_t *table, int jb, int nv) {
    typedef const __attribute__((address_space(4))) int32_t const_i32;
    const int jc = max(min(jb, nv - 1), 0);
    const int32_t b = ((const_i32 *)table)[jc];
    // select by mask rather than by branch: the load stays unconditional
    const int32_t keep = -(int32_t)((unsigned)jb < (unsigned)nv);
    return b | ~keep;
}

template <int D>
__device__ __forceinline__ int chunk_block(int tid, int u) {
    using C = TileCfg<D>;
    int bi;
    if (u < C::kKPer) {
        bi = (tid + u * kPreThreads) / C::kCpt;
    } else {
        int dim, h;
        v_chunk_coords<D>(tid, u - C::kKPer, bi, dim, h);
    }
    return __builtin_amdgcn_readfirstlane(bi);   // uniform per wave by construction
}

// Load set t = {K of blocks 4t+2 .. 4t+5, V of blocks 4t .. 4t+3}: the keys
// are staged 32 ahead of the values (see the pipeline in prefill_kernel).
// Read the block ids behind this thread's chunks of set t (scalar loads,
// issued a step before use); blocks outside [0, nb) read as absent.
template <int D>
__device__ __forceinline__ void fetch_ids(TileIds<D> &ids, const int32_t *table, int t, int nb, int tid) {
#pragma unroll
    for (int u = 0; u < TileCfg<D>::kPerThread; ++u) {
        const bool is_k = u < TileCfg<D>::kKPer;
        ids.b[u] = table_entry(table, 4 * t + (is_k ? 2 : 0) + chunk_block<D>(tid, u), nb);
    }
}

// Issue the loads of one load set into registers.  Blocks past the session's
// keys (or with an id outside the pool) are read through a zero-size buffer
// descriptor: no memory traffic, zeros returned.  Every call issues the same
// loads, so outstanding loads can be counted across iterations.
template <int D>
__device__ __forceinline__ void load_tile(TileRegs<D> &r, const TileIds<D> &ids, const PrefillArgs &a,
                                          int g, int tid) {
    using C = TileCfg<D>;
#pragma unroll
    for (int u = 0; u < C::kPerThread; ++u) {
        int off, is_v;
        if (u < C::kKPer) {
            off = ((tid + u * kPreThreads) % C::kCpt) * 16;
            is_v = 0;
        } else {
            int bi, dim, h;
            v_chunk_coords<D>(tid, u - C::kKPer, bi, dim, h);
            off = (dim * 2 + h) * 16;
            is_v = 1;
        }
        const int32_t b = ids.b[u];
        const bool valid = b >= 0 && b < a.num_blocks;
        const uint16_t *base =
            a.pool + (((int64_t)(valid ? b : 0) * 2 + is_v) * a.num_kv_heads + g) * (kBlock * D);
        const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<uint16_t *>(base), 0, valid ? C::kTileBytes : 0, kBufferDword3P);
        r.c[u] = __builtin_amdgcn_raw_buffer_load_b128(rsrc, off, 0, 0);
    }
}

// LDS layouts of staged keys and values (32-key units: unit u = blocks 2u, 2u+1):
//   K: four unit slots, unit u in slot u % 4: [block 2][token 16][D/8 chunks
//      of 16 B], chunk index XOR (token % (D/8)).
//   V: one 64-key tile per buffer: [k2 2][g4 4][dim D] groups of 16 B =
//      {block 2*k2, tokens 4*g4..4*g4+3; block 2*k2+1, the same tokens}: the
//      8 keys one lane feeds the PV MFMA.
// Token slots at or past the session's last key (kv_len) are zeroed here, so
// masked keys contribute exact zeros (never NaN) to PV.
template <int D>
__device__ __forceinline__ void store_tile(const TileRegs<D> &r, uint8_t *lds_k, uint8_t *lds_v,
                                           int tid, int t, int kv_len) {
    using C = TileCfg<D>;
    constexpr int kRowChunks = D / 8;
    const int key_k = (4 * t + 2) * kBlock;          // first key of the set's K blocks
    const int key_v = 4 * t * kBlock;                // first key of its V blocks
    const bool tail_k = key_k + kKeyTile > kv_len;
    const bool tail_v = key_v + kKeyTile > kv_len;
    u32x4 v[C::kVPer];
    int bi_v[C::kVPer], dim = 0, h = 0;
#pragma unroll
    for (int u = 0; u < C::kPerThread; ++u) {
        if (u < C::kKPer) {
            const int c = tid + u * kPreThreads;
            const int bi = c / C::kCpt;
            const int within = c % C::kCpt;
            const int token = within / kRowChunks;
            const int ch = within % kRowChunks;
            u32x4 x = r.c[u];
            if (tail_k && key_k + bi * kBlock + token >= kv_len) x = u32x4{0u, 0u, 0u, 0u};
            const int slot = ch ^ (token & (kRowChunks - 1));
            const int unit_slot = (2 * t + 1 + (bi >> 1)) & 3;
            *reinterpret_cast<u32x4 *>(lds_k + unit_slot * (2 * C::kTileBytes) + (bi & 1) * C::kTileBytes +
                                       token * (D * 2) + slot * 16) = x;
        } else {
            const int e = u - C::kKPer;
            v_chunk_coords<D>(tid, e, bi_v[e], dim, h);
            v[e] = r.c[u];
            if (tail_v) {
                const int t0 = key_v + bi_v[e] * kBlock + h * 8;
#pragma unroll
                for (int w = 0; w < 4; ++w) {
                    const int t = t0 + 2 * w;
                    const uint32_t mask = t + 1 < kv_len ? 0xFFFFFFFFu : (t < kv_len ? 0x0000FFFFu : 0u);
                    v[e][w] &= mask;
                }
            }
        }
    }
    // chunk words 0,1 hold tokens 8h..8h+3 (group g4 = 2h), words 2,3 the next four
    if constexpr (C::kVPer == 2) {
        const int k2 = bi_v[0] >> 1;
        uint8_t *g0 = lds_v + ((k2 * 4 + 2 * h) * D + dim) * 16;
        uint8_t *g1 = lds_v + ((k2 * 4 + 2 * h + 1) * D + dim) * 16;
        *reinterpret_cast<u32x4 *>(g0) = u32x4{v[0][0], v[0][1], v[1][0], v[1][1]};
        *reinterpret_cast<u32x4 *>(g1) = u32x4{v[0][2], v[0][3], v[1][2], v[1][3]};
    } else {
        const int k2 = bi_v[0] >> 1, half = bi_v[0] & 1;
        uint8_t *g0 = lds_v + ((k2 * 4 + 2 * h) * D + dim) * 16 + half * 8;
        uint8_t *g1 = lds_v + ((k2 * 4 + 2 * h + 1) * D + dim) * 16 + half * 8;
        *reinterpret_cast<u32x2 *>(g0) = u32x2{v[0][0], v[0][1]};
        *reinterpret_cast<u32x2 *>(g1) = u32x2{v[0][2], v[0][3]};
    }
}

template <int D>
__global__ __launch_bounds__(kPreThreads) void prefill_kernel(PrefillArgs a) {
    using C = TileCfg<D>;
    constexpr int KS = D / 32;           // 32-dim k-steps of QK
    constexpr int NDT = D / 16;          // 16-dim output tiles
    constexpr int kRowChunks = D / 8;
    __shared__ __attribute__((aligned(16))) uint8_t lds_k[4 * 2 * C::kTileBytes];   // 4 unit slots
    __shared__ __attribute__((aligned(16))) uint8_t lds_v[2][4 * C::kTileBytes];
    __shared__ int64_t sm_work[kMaxSortSessions];
    __shared__ int sm_order[kMaxSortSessions];

    const int tid = threadIdx.x;
    const int S = a.num_sessions;
    const int G = a.group;
    const int qtok = kPreRows / G;       // new tokens per query tile
    const int QT = a.qtiles;
    const int Hkv = a.num_kv_heads;

    // ---- XCD-aware placement: each XCD takes kXcdChunk consecutive items
    const int64_t total = (int64_t)S * Hkv * QT;
    const int64_t hw = blockIdx.x;
    const int64_t slot = hw / kXcds;
    const int64_t logical =
        (slot / kXcdChunk) * (kXcds * kXcdChunk) + (hw % kXcds) * kXcdChunk + slot % kXcdChunk;
    if (logical >= total) return;
    const int qt = QT - 1 - (int)(logical % QT);
    const int g = (int)((logical / QT) % Hkv);
    const int rank = (int)(logical / ((int64_t)QT * Hkv));

    // ---- session of this rank: longest (query tiles x keys) first, ties by index
    int s = rank;
    if (S <= kMaxSortSessions) {
        if (tid < S) {
            const int nt = a.cu[tid + 1] - a.cu[tid];
            sm_work[tid] = (int64_t)((nt + qtok - 1) / qtok) * (a.ctx[tid] + nt);
        }
        __syncthreads();
        if (tid < S) {
            const int64_t w = sm_work[tid];
            int r = 0;
            for (int t = 0; t < S; ++t) {
                const int64_t wt = sm_work[t];
                r += (wt > w) || (wt == w && t < tid);
            }
            sm_order[r] = tid;
        }
        __syncthreads();
        s = sm_order[rank];
    }

    const int n = a.cu[s + 1] - a.cu[s];
    const int j0 = qt * qtok;
    if (j0 >= n) return;
    const int c = a.ctx[s];
    const int j_last = min(j0 + qtok, n) - 1;
    const int kv_len = c + n;
    int nblk_valid = (kv_len + kBlock - 1) / kBlock;
    if (nblk_valid > a.max_blocks) {
        nblk_valid = a.max_blocks;
        if (tid == 0) flag_error(a.err, LS_DEVERR_LENGTH);
    }
    const int kv_end = c + j_last + 1;                    // keys this tile can see
    const int ntiles = (kv_end + kKeyTile - 1) / kKeyTile;

    const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
    const int lane = tid % kWave;
    const int c16 = lane & 15;
    const int g4 = lane >> 4;
    const int hq_total = Hkv * G;

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
            qop[rt][ks] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(qrow + ks * 32 + g4 * 8));
    }
    // Wait for q here, before the first tile loads are issued, so that no wait
    // for q remains inside the key loop (vmcnt(0), other counters untouched).
    __builtin_amdgcn_s_waitcnt(0x0F70);
    // smallest causal limit among this wave's rows: key tiles past it need masking
    const int wave_lim_min = c + min(j0 + (wave * 32) / G, n - 1);

    float m[2] = {-INFINITY, -INFINITY};  // running row maxima (raw scores)
    float nm[2] = {0.f, 0.f};             // -m * scale * log2(e)
    float lsum[2] = {0.f, 0.f};           // this lane's partial row sums
    f32x4 o[2][NDT];
#pragma unroll
    for (int rt = 0; rt < 2; ++rt)
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) o[rt][dt] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int32_t *table = a.block_tables + (int64_t)s * a.max_blocks;
    const float sl2 = a.scale_log2;
    const float slack_raw = kRescaleSlack / sl2;
    const bf16x2 ones2 = {(__bf16)1.0f, (__bf16)1.0f};

    // ---- one 32-key unit of the key stream: S^T = K Q^T for 2 key sub-tiles x
    // 2 row tiles into acc (K unit slot s of lds_k)
    auto qk_unit = [&](f32x4 (&acc)[2][2], int slot_u) {
        const uint8_t *lk = lds_k + slot_u * (2 * C::kTileBytes);
#pragma unroll
        for (int sb = 0; sb < 2; ++sb) {
            const int sub = sb;
            acc[0][sb] = f32x4{0.f, 0.f, 0.f, 0.f};
            acc[1][sb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                const int ch = ks * 4 + g4;
                const int sl = ch ^ (c16 & (kRowChunks - 1));
                const bf16x8 kop = __builtin_bit_cast(
                    bf16x8, *reinterpret_cast<const u32x4 *>(lk + sub * C::kTileBytes + c16 * (D * 2) + sl * 16));
                acc[0][sb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kop, qop[0][ks], acc[0][sb], 0, 0, 0);
                acc[1][sb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kop, qop[1][ks], acc[1][sb], 0, 0, 0);
            }
        }
    };
    // Causal mask of a unit whose first key is key0, then its row maxima; a
    // row max that exceeds the running max by more than the slack raises it
    // and rescales O and l (rare after the first unit).  scale > 0 is checked
    // on the host, so masking and maxima commute with scaling.
    auto max_unit = [&](f32x4 (&acc)[2][2], int key0) {
        const bool diag = key0 + 31 > wave_lim_min;
#pragma unroll
        for (int rt = 0; rt < 2; ++rt) {
            if (diag) {
                // key key0 + sb*16 + 4*g4 + i is visible iff sb*16 + i <= lim
                const int lim = row_lim[rt] - key0 - 4 * g4;
#pragma unroll
                for (int sb = 0; sb < 2; ++sb)
#pragma unroll
                    for (int i = 0; i < 4; ++i)
                        if (sb * 16 + i > lim) acc[rt][sb][i] = -INFINITY;
            }
            const f32x4 x0 = acc[rt][0], x1 = acc[rt][1];
            float bm = fmax3(fmax3(x0[0], x0[1], x0[2]), fmax3(x0[3], x1[0], x1[1]), fmax3(x1[2], x1[3], x1[3]));
            bm = xmax16_32(bm);
            if (__any(bm > m[rt] + slack_raw)) {
                const float m_new = __builtin_elementwise_maximum(m[rt], bm);
                const float alpha = __builtin_amdgcn_exp2f((m[rt] - m_new) * sl2);
                lsum[rt] *= alpha;
#pragma unroll
                for (int dt = 0; dt < NDT; ++dt) o[rt][dt] *= alpha;
                m[rt] = m_new;
                nm[rt] = -m_new * sl2;
            }
        }
    };
    // P = exp2(S * scale * log2 e - m') in bf16 (B operand of PV) and row sums.
    auto exp_unit = [&](const f32x4 (&acc)[2][2], bf16x8 (&pop)[2]) {
#pragma unroll
        for (int rt = 0; rt < 2; ++rt) {
            uint32_t w[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const f32x4 &x = acc[rt][j >> 1];
                const int i0 = 2 * (j & 1);
                const bf16x2 pk = {(__bf16)__builtin_amdgcn_exp2f(__builtin_fmaf(x[i0], sl2, nm[rt])),
                                   (__bf16)__builtin_amdgcn_exp2f(__builtin_fmaf(x[i0 + 1], sl2, nm[rt]))};
                lsum[rt] = __builtin_amdgcn_fdot2_f32_bf16(pk, ones2, lsum[rt], false);
                w[j] = __builtin_bit_cast(uint32_t, pk);
            }
            pop[rt] = __builtin_bit_cast(bf16x8, u32x4{w[0], w[1], w[2], w[3]});
        }
    };
    // O^T += V^T P^T for unit half h of a V tile staged at lv.
    auto pv_unit = [&](const bf16x8 (&pop)[2], const uint8_t *lv, int h) {
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) {
            const bf16x8 vop = __builtin_bit_cast(
                bf16x8, *reinterpret_cast<const u32x4 *>(lv + ((h * 4 + g4) * D + dt * 16 + c16) * 16));
            o[0][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vop, pop[0], o[0][dt], 0, 0, 0);
            o[1][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vop, pop[1], o[1][dt], 0, 0, 0);
        }
    };
    // One pipeline step: the scores of unit u (in cur, masked, max applied)
    // become P and are accumulated while the scores of unit u+1 are computed
    // into nxt.  exp/PV of u and QK of u+1 are independent, so the MFMAs of one
    // interleave with the VALU work of the other.
    auto unit_step = [&](f32x4 (&cur)[2][2], f32x4 (&nxt)[2][2], int slot_next, int key0_next,
                         const uint8_t *lv, int h) {
        bf16x8 pop[2];
        qk_unit(nxt, slot_next);
        exp_unit(cur, pop);
        pv_unit(pop, lv, h);
        max_unit(nxt, key0_next);
    };

    // ---- pipeline over 32-key units.  Step u turns the scores of unit u into
    // P, accumulates P V of unit u and computes the scores of unit u+1, so K
    // is needed one unit ahead of V: while key tile j (units 2j, 2j+1) is
    // processed, LDS holds V(j) in lds_v[j&1] and K units 2j+1, 2j+2 in their
    // slots.  At the end of tile j, load set j+1 (K units 2j+3, 2j+4 and V tile
    // j+1) goes from registers to LDS, into slots and a buffer that tile j
    // does not read; it was loaded two tiles ahead (register sets ra, rb).
    // One barrier per tile.
    const int nb = min(nblk_valid, ntiles * 4);     // blocks any row here can see
    TileRegs<D> ra, rb;
    TileIds<D> ids;
    f32x4 sa[2][2], sb2[2][2];
    fetch_ids<D>(ids, table, -1, nb, tid);          // set -1: K unit 0 only
    load_tile<D>(ra, ids, a, g, tid);
    fetch_ids<D>(ids, table, 0, nb, tid);
    load_tile<D>(rb, ids, a, g, tid);
    fetch_ids<D>(ids, table, 1, nb, tid);
    store_tile<D>(ra, lds_k, lds_v[1], tid, -1, kv_len);
    load_tile<D>(ra, ids, a, g, tid);               // set 1
    fetch_ids<D>(ids, table, 2, nb, tid);
    store_tile<D>(rb, lds_k, lds_v[0], tid, 0, kv_len);
    load_tile<D>(rb, ids, a, g, tid);               // set 2
    __syncthreads();
    qk_unit(sa, 0);
    max_unit(sa, 0);
    // Both halves of the body issue the same loads on every path (only the
    // second tile's compute is conditional), so outstanding loads are counted
    // exactly.  Unit slots: tile j reads slots (2j+1)%4 and (2j+2)%4.
    for (int j = 0; j < ntiles; j += 2) {
        fetch_ids<D>(ids, table, j + 3, nb, tid);
        unit_step(sa, sb2, 1, j * kKeyTile + 32, lds_v[0], 0);
        unit_step(sb2, sa, 2, (j + 1) * kKeyTile, lds_v[0], 1);
        store_tile<D>(ra, lds_k, lds_v[1], tid, j + 1, kv_len);
        load_tile<D>(ra, ids, a, g, tid);           // set j+3
        __syncthreads();
        fetch_ids<D>(ids, table, j + 4, nb, tid);
        if (j + 1 < ntiles) {
            unit_step(sa, sb2, 3, (j + 1) * kKeyTile + 32, lds_v[1], 0);
            unit_step(sb2, sa, 0, (j + 2) * kKeyTile, lds_v[1], 1);
        }
        store_tile<D>(rb, lds_k, lds_v[0], tid, j + 2, kv_len);
        load_tile<D>(rb, ids, a, g, tid);           // set j+4
        __syncthreads();
    }

    // ---- normalise and write
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
        const float inv = 1.f / xsum16_32(lsum[rt]);
        if (!row_ok[rt]) continue;
        uint16_t *orow = a.out + row_out[rt];
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) {
            const u32x2 w = u32x2{pack_bf16x2(o[rt][dt][0] * inv, o[rt][dt][1] * inv),
                                  pack_bf16x2(o[rt][dt][2] * inv, o[rt][dt][3] * inv)};
            *reinterpret_cast<u32x2 *>(orow + dt * 16 + g4 * 4) = w;
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
    a.num_sessions = num_sessions;
    a.q = q;
    a.out = out;
    a.cu = cu_new_lens;
    a.ctx = reused_lens;
    a.block_tables = block_tables;
    a.max_blocks = max_blocks;
    a.scale_log2 = scale * kLog2eP;
    a.err = err;
    const int qtok = kPreRows / a.group;
    a.qtiles = (max_new_len + qtok - 1) / qtok;
    const int64_t items = (int64_t)num_sessions * p.num_kv_heads * a.qtiles;
    // Whole groups of kXcds * kXcdChunk workgroups keep the placement map a
    // bijection onto [0, grid); workgroups past the item count exit at once.
    const int64_t per_group = (int64_t)kXcds * kXcdChunk;
    const int64_t grid = (items + per_group - 1) / per_group * per_group;
    if (grid > 0x7FFFFFFFLL) return hipErrorInvalidConfiguration;
    if (p.head_dim == 128)
        hipLaunchKernelGGL(prefill_kernel<128>, dim3((unsigned)grid), dim3(kPreThreads), 0, stream, a);
    else
        hipLaunchKernelGGL(prefill_kernel<64>, dim3((unsigned)grid), dim3(kPreThreads), 0, stream, a);
    return hipGetLastError();
}

}  // namespace ls
