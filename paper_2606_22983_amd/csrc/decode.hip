// Paged-attention decode: one query token per session attends to its whole
// paged context — the batched decode step of the thinker/talker
// autoregressive decoders (LiveServe §2.1; continuous-batching decode loop of
// §6) over per-session block tables (block-level KV allocation, §5.1).
//
// Work decomposition (split-K): an item = (split k, KV head g, session s),
// covering tokens [k*T, (k+1)*T) of the session (T = 1024 on large batches).
// A persistent grid holds one 8-wave workgroup per CU (one workgroup, so no
// two workgroups on a CU compete for its issue slots: with two 4-wave
// workgroups the second ran ~15% slower and lengthened the tail).  The 8
// wavefronts of a workgroup take an item's 16-token blocks round-robin; each
// keeps a wavefront-level online softmax state (running max m, running sum l,
// unnormalised output O) for the G query heads of group g.  The waves merge
// through LDS.  A session that fits
// one split is written directly; otherwise each split leaves (m, l, O) in the
// workspace and a second, small kernel merges the splits with the log-sum-exp
// rule (kernel boundaries order the two, so no cross-workgroup fences).
//
// Per block, the GQA group's contraction runs on MFMA 16x16 tiles:
//   S^T[16 tokens x 16 heads] = K[16 x D] . Q^T[D x 16]     (16x16x32 bf16)
//   O^T[16 dims   x 16 heads] += V^T[16 x 16 tokens] . P^T     (16x16x16 bf16)
// The MFMA accumulator layout of S^T (lane: head = lane%16, tokens 4*(lane/16)+i)
// is exactly the B-operand layout PV needs, so the probabilities never leave
// registers.  K tiles are chunk-major ([D/8][16 tokens][8 dims]) and V tiles
// dim-major in the pool, so both operands load straight from HBM into their
// MFMA lanes: each K load instruction reads 1 KiB contiguous (lane l: bytes
// 16l .. 16l+15 of the k-step's chunks), each V load 512 contiguous bytes;
// prefetched two blocks ahead.  The split's block ids
// are read once into a register and broadcast with readlane, so the load
// stream never waits on an index fetch; a block that does not exist is loaded
// through a zero-size buffer descriptor (no memory traffic, no branch).  Heads
// beyond G in the 16-wide tile carry q = 0 and are never written.
//
// A step that appends its own token (k_new / v_new given) needs no separate
// append launch: the wave that holds the session's last block masks the
// token's (not yet written) pool slot, attends to the token as a one-token
// tile built from k_new / v_new, and then writes it to the slot for the next
// steps.
#include <algorithm>

#include "common.h"

namespace ls {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kDecThreads = 512;
constexpr int kDecWaves = kDecThreads / kWave;
constexpr int kMaxSplitTokens = 1024;        // 8 blocks per wave (the unrolled sequence)
constexpr int kMaxSplits = 256;              // combine kernel's LDS capacity
constexpr int kMaxBatch = 2048;              // sessions per decode call (LDS prefix sums)
constexpr int kMaxGroup = 8;                 // query heads per KV head
constexpr int kKeyBins = kMaxSplitTokens / kBlock + 1;   // short-split block counts 0..64
static_assert(kMaxBatch * kMaxSplits <= 0xFFFFF && kMaxBatch < 4096,
              "work-row counts must fit the packed scan (20 + 12 bits)");
constexpr int kSpinLimit = 1 << 22;          // bound of the merge-slot wait (~0.1 s)
constexpr float kLog2e = 1.4426950408889634f;
constexpr int kBufferDword3 = 0x00020000;   // raw buffer, 32-bit data format
// Cache policy of the K/V tile loads: non-temporal (each tile is read once per
// call, so it is not kept in the caches; measured 10-15% faster on random
// block streams than the default policy).
constexpr int kStreamLoad = 2;
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
    int32_t appended;              // 1: the step's own token sits at position lens[s]
    const uint16_t *k_new;         // [S][Hkv][D] the step's own K/V (appended == 1), written
    const uint16_t *v_new;         // to the pool by this kernel and attended from here
    float scale_log2;              // scale * log2(e)
    int32_t split_tokens;          // at most kPerWave * kDecWaves * kBlock of the instantiation
    int32_t max_splits;
    float *part_ml;                // [S][Hkv][max_splits][G][2]
    float *part_acc;               // [S][Hkv][max_splits][G][D]
    unsigned int *err;             // device error word
    int32_t num_sessions;
};

template <int D>
struct BlockRegs {
    u32x4 k[D / 32];               // K[token lane%16][8 dims of k-step ks]
    u32x2 v[D / 16];               // V^T[dim 16*dt + lane%16][tokens 4*(lane/16) .. +3]
};

// Max / sum over the lanes l, l^16, l^32, l^48 (one head's four token
// groups) with the gfx950 row-swap permutes: VALU only, no LDS round trip.
__device__ __forceinline__ float wave_max_xor_16_32(float x) {
    const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    const float y = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
    const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(y), __float_as_uint(y), false, false);
    return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

__device__ __forceinline__ float wave_sum_xor_16_32(float x) {
    const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    const float y = __uint_as_float(a[0]) + __uint_as_float(a[1]);
    const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(y), __float_as_uint(y), false, false);
    return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// Tokens of session s that attention covers, clipped to [0, table]; an empty
// context (softmax over no key) and an over-long one are flagged.  Kept
// branch-free so that the compiler sees a wave-uniform value.
__device__ __forceinline__ int attended_len(const DecodeArgs &a, int s, bool may_flag) {
    const int raw = a.lens[s] + a.appended;
    const int cap = a.max_blocks * kBlock;
    if (may_flag && (raw > cap || raw <= 0)) flag_error(a.err, LS_DEVERR_LENGTH);
    return max(min(raw, cap), 0);
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
    for (int ks = 0; ks < D / 32; ++ks) r.k[ks] = __builtin_amdgcn_raw_buffer_load_b128(rk, koff[ks], 0, kStreamLoad);
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt) r.v[dt] = __builtin_amdgcn_raw_buffer_load_b64(rv, voff[dt], 0, kStreamLoad);
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

// Block-wide exclusive scan of one value per thread (kDecThreads threads),
// modulo 2^32.
__device__ __forceinline__ unsigned block_exclusive_scan(unsigned v, unsigned *sm_wave_tot, unsigned &total) {
    const int lane = threadIdx.x % kWave;
    const int wave = threadIdx.x / kWave;
    unsigned x = v;
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
        const unsigned y = __shfl_up(x, off);
        if (lane >= off) x += y;
    }
    if (lane == kWave - 1) sm_wave_tot[wave] = x;
    __syncthreads();
    unsigned before = 0;
    total = 0;
#pragma unroll
    for (int w = 0; w < kDecWaves; ++w) {
        const unsigned t = sm_wave_tot[w];
        if (w < wave) before += t;
        total += t;
    }
    return before + x - v;
}

// Persistent decode: a fixed grid (one workgroup per CU) walks the work
// items (session s, split k, KV head g).  Each workgroup first orders, in LDS,
// the work rows (session, split) longest first: every full split (T tokens),
// then each session's last, shorter split by block count, largest first (an
// empty session's one row is among them).  Items are dealt in snake order:
// round k gives item k*W + w to workgroup w for even k and k*W + W-1-w for odd
// k (W workgroups), so every workgroup receives about the same number of
// tokens; with plain round-robin the workgroups holding one item more than the
// rest decide the call's duration.  Every workgroup derives the same order
// from the lengths, no workgroup is launched for a split that does not exist,
// and each fetches the next item's block ids while it works on the current one.
template <int D, int kDepth, int kMaxPerWave>
__global__ __launch_bounds__(kDecThreads) void decode_kernel(DecodeArgs a) {
    __shared__ int sm_cum[kMaxBatch + 1];       // first full-split row of each session
    __shared__ int sm_len[kMaxBatch];           // attended length of each session
    __shared__ int sm_porder[kMaxBatch];        // sessions of the short-split rows, in row order
    __shared__ int sm_key[kDecThreads];         // block count of a session's short split (-1: none)
    __shared__ unsigned long long sm_kmask[kKeyBins][kDecThreads / 64];  // sessions per short-split key
    __shared__ int sm_kabove[kKeyBins + 1];     // sessions with a larger key (suffix counts)
    __shared__ uint8_t sm_own[kMaxBatch];       // 1: the session's own new token is attended (fits the table)
    __shared__ unsigned sm_wave_tot[kDecWaves];
    // Per-item merge slots (double-buffered): each wave leaves its (m, l, O) of
    // the group's heads, the last wave to arrive merges them.
    __shared__ float sm_m[2][kDecWaves][kMaxGroup];
    __shared__ float sm_l[2][kDecWaves][kMaxGroup];
    __shared__ __attribute__((aligned(16))) float sm_o[2][kDecWaves][kMaxGroup][D];
    __shared__ int sm_arrived[2];               // waves that have filled the slot
    __shared__ int sm_merged[2];                // merges completed on the slot

    const int tid = threadIdx.x;
    const int G = a.group;
    const int hq_total = a.num_kv_heads * G;
    const int S = a.num_sessions;
    const int T = a.split_tokens;

    if (tid < 2) {
        sm_arrived[tid] = 0;
        sm_merged[tid] = 0;
    }
    constexpr int kMaskWords = kDecThreads / 64;
    for (int i = tid; i < kKeyBins * kMaskWords; i += kDecThreads) sm_kmask[i / kMaskWords][i % kMaskWords] = 0ull;
    // ---- work rows: full splits per session (prefix sum) and short splits.
    // Both counts share one unsigned scan: full rows in bits 0..19 (at most
    // kMaxBatch * kMaxSplits = 2^19 in total), short rows (at most kMaxBatch)
    // in bits 20..31.
    const int per_thread = (S + kDecThreads - 1) / kDecThreads;
    const int s_begin = min(S, tid * per_thread);
    const int s_end = min(S, s_begin + per_thread);
    auto has_short = [&](int L) { return L == 0 || L % T != 0; };   // an empty session still owns one row
    unsigned mine = 0;
    for (int s = s_begin; s < s_end; ++s) {
        const int L = attended_len(a, s, blockIdx.x == 0);
        sm_len[s] = L;
        sm_own[s] = a.appended && a.lens[s] >= 0 && a.lens[s] + 1 <= a.max_blocks * kBlock;
        mine += (unsigned)(L / T) + (has_short(L) ? 1u << 20 : 0u);
    }
    unsigned packed_total = 0;
    const unsigned packed_run = block_exclusive_scan(mine, sm_wave_tot, packed_total);
    const int full_rows = (int)(packed_total & 0xFFFFFu);
    const int total_rows = full_rows + (int)(packed_total >> 20);
    {
        int frun = (int)(packed_run & 0xFFFFFu), prun = (int)(packed_run >> 20);
        for (int s = s_begin; s < s_end; ++s) {
            const int L = sm_len[s];
            sm_cum[s] = frun;
            frun += L / T;
            if (has_short(L)) {
                if (S > kDecThreads) sm_porder[prun] = s;         // large batch: session order
                ++prun;
            }
        }
        if (S <= kDecThreads && tid < S) {
            const int L = sm_len[tid];
            sm_key[tid] = has_short(L) ? (L % T + kBlock - 1) / kBlock : -1;
        }
    }
    if (tid == 0) sm_cum[S] = full_rows;
    __syncthreads();
    // Rank of each short row: rows with a larger block count first, then
    // session order.  Keys are block counts 0..T/16, so the rank is the number
    // of sessions with a larger key (suffix sums of per-key counts) plus the
    // sessions before this one with the same key (a popcount of that key's
    // session bitmask); both are built with order-independent LDS atomics, so
    // every workgroup derives the same order.
    const bool ranked = S <= kDecThreads && tid < S && sm_key[tid] >= 0;
    if (ranked) __hip_atomic_fetch_or(&sm_kmask[sm_key[tid]][tid / 64], 1ull << (tid % 64), __ATOMIC_RELAXED,
                                      __HIP_MEMORY_SCOPE_WORKGROUP);
    __syncthreads();
    if (S <= kDecThreads && tid < kWave) {
        // Suffix sums over the key bins, one wave: bins 64*c + lane in chunk c.
        int carry = 0;
        for (int c = (kKeyBins + kWave - 1) / kWave - 1; c >= 0; --c) {
            const int bin = c * kWave + tid;
            int cnt = 0;
            if (bin < kKeyBins)
                for (int w = 0; w < kDecThreads / 64; ++w) cnt += __popcll(sm_kmask[bin][w]);
            // inclusive suffix scan of cnt over the lanes (higher lanes first)
            int x = cnt;
#pragma unroll
            for (int off = 1; off < kWave; off <<= 1) {
                const int y = __shfl_down(x, off);
                if (tid + off < kWave) x += y;
            }
            if (bin < kKeyBins) sm_kabove[bin] = carry + x - cnt;
            carry += __shfl(x, 0);
        }
    }
    __syncthreads();
    if (ranked) {
        const int key = sm_key[tid];
        int rank = sm_kabove[key];
        for (int w = 0; w < tid / 64; ++w) rank += __popcll(sm_kmask[key][w]);
        rank += __popcll(sm_kmask[key][tid / 64] & ((1ull << (tid % 64)) - 1ull));
        sm_porder[rank] = tid;
    }
    __syncthreads();
    const int total_items = total_rows * a.num_kv_heads;
    const int W = (int)gridDim.x;
    auto item_of = [&](int round) { return round * W + ((round & 1) ? W - 1 - (int)blockIdx.x : (int)blockIdx.x); };

    const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
    const int lane = tid % kWave;
    const int c16 = lane & 15;
    const int g4 = lane >> 4;
    int koff[D / 32], voff[D / 16];
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) koff[ks] = ((ks * 4 + g4) * kBlock + c16) * 16;   // = ks*1024 + lane*16
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt) voff[dt] = ((dt * 16 + c16) * kBlock + g4 * 4) * 2;

    // (session, split) of work row r.  A full row: the largest s with
    // sm_cum[s] <= r (a session without full splits shares its sm_cum with the
    // next session, so it is never the largest).  A short row: its session's
    // last split.
    auto locate = [&](int row, int &s_out, int &split_out) {
        if (row >= full_rows) {
            s_out = sm_porder[row - full_rows];
            split_out = sm_len[s_out] / T;
            return;
        }
        int lo = 0, hi = S - 1;
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (sm_cum[mid] <= row) lo = mid; else hi = mid - 1;
        }
        s_out = lo;
        split_out = row - sm_cum[lo];
    };
    // Raw block ids of a split, one per lane.  The load is unconditional (its
    // index clamped into the table row) and the id is validated only when it is
    // used, so nothing waits for this load until the item is processed.
    auto fetch_ids = [&](int s_, int split_) -> int {
        const int j = min(split_ * (T / kBlock) + lane, a.max_blocks - 1);
        return a.block_tables[(int64_t)s_ * a.max_blocks + j];
    };
    // Validated id (or -1) of entry idx of a fetched id register.
    auto checked_id = [&](int ids, int idx, int nb) -> int {
        const int b = __builtin_amdgcn_readlane(ids, min(idx, kWave - 1));
        const bool in_split = idx < nb;
        const bool ok = in_split && b >= 0 && b < a.num_blocks;
        if (in_split && !ok && lane == 0) flag_error(a.err, LS_DEVERR_BLOCK_ID);
        // Scalar result (the flag's lane-0 branch must not make it a vector value).
        return __builtin_amdgcn_readfirstlane(ok ? b : -1);
    };

    // Q^T operand of an item: column = query head c16 of the group (zero beyond G).
    auto load_q = [&](int s_, int g_, bf16x8 (&qo)[D / 32]) {
        const bool active = c16 < G;
        const uint16_t *qrow = a.q + ((int64_t)s_ * hq_total + g_ * G + (active ? c16 : 0)) * D;
#pragma unroll
        for (int ks = 0; ks < D / 32; ++ks) {
            uint4 v = *reinterpret_cast<const uint4 *>(qrow + ks * 32 + g4 * 8);
            if (!active) v = make_uint4(0, 0, 0, 0);
            qo[ks] = __builtin_bit_cast(bf16x8, v);
        }
    };
    // Block count of a split and this wave's it-th block id within it.
    auto split_blocks = [&](int s_, int split_) -> int {
        const int L = sm_len[s_];
        const int t0 = split_ * T;
        return L > t0 ? (min(L, t0 + T) + kBlock - 1) / kBlock - t0 / kBlock : 0;
    };

    // kDepth blocks in flight per wave, carried across items: the next item's
    // first blocks (and its q) are requested before the current item's merge.
    BlockRegs<D> r[kDepth];
    int bb[kDepth];
    bf16x8 qop[D / 32];
    // Each wave keeps the fetched block ids of the current and the next item in
    // its own LDS slots (double-buffered; read back with readlane), so no value
    // loaded from memory is carried around the item loop.
    __shared__ int sm_ids[kDecWaves][2][kMaxSplitTokens / kBlock];
    int item = item_of(0);
    int s = 0, split = 0;
    if (item < total_items) {
        locate(item / a.num_kv_heads, s, split);
        const int ids0 = fetch_ids(s, split);
        if (lane < kMaxSplitTokens / kBlock) sm_ids[wave][0][lane] = ids0;
        load_q(s, item % a.num_kv_heads, qop);
        const int nb = split_blocks(s, split);
#pragma unroll
        for (int j = 0; j < kDepth; ++j) {
            bb[j] = checked_id(ids0, wave + j * kDecWaves, nb);
            load_block<D>(r[j], a.pool, a.num_kv_heads, item % a.num_kv_heads, bb[j], koff, voff);
        }
    }
    for (int k = 0; item < total_items; ++k, item = item_of(k)) {
        const int g = item % a.num_kv_heads;
        const int L = sm_len[s];
        const int own = sm_own[s];
        const int Lp = L - own;            // keys read from the pool; the own token comes from k_new
        const int cur_s = s, cur_split = split;
        const int cur_ids = lane < kMaxSplitTokens / kBlock ? sm_ids[wave][k & 1][lane] : -1;
        // Next item: its (session, split) and block ids, fetched now.
        const int next = item_of(k + 1);
        const bool has_next = next < total_items;
        int next_ids = -1;
        if (has_next) {
            locate(next / a.num_kv_heads, s, split);
            next_ids = fetch_ids(s, split);
        }
        const int t0 = cur_split * T;
        const int nsplit = L > 0 ? (L + T - 1) / T : 1;
        const int blk0 = t0 / kBlock;
        const int nblk = split_blocks(cur_s, cur_split);
        const int my_n = wave < nblk ? (nblk - wave + kDecWaves - 1) / kDecWaves : 0;
        auto bid = [&](int it) -> int { return checked_id(cur_ids, wave + it * kDecWaves, nblk); };

        // The running max starts at a finite floor: a block whose keys are all
        // masked then leaves (m, l, O) unchanged instead of producing NaN.
        float m = kMaxFloor, lsum = 0.f;
        f32x4 o[D / 16];
#pragma unroll
        for (int dt = 0; dt < D / 16; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};

        // The per-wave block sequence is fully unrolled (at most kMaxPerWave
        // blocks) with forward-only exits, so the compiler sees straight-line
        // code and waits only for the block it is about to use.  A block with a
        // bad id is processed as fully masked.
#pragma unroll
        for (int i = 0; i < kMaxPerWave; ++i) {
            if (i >= my_n) break;
            const int j = i % kDepth;
            const int tb = (blk0 + wave + i * kDecWaves) * kBlock;
            process_block<D>(r[j], qop, tb, bb[j] >= 0 ? Lp : 0, a.scale_log2, g4, m, lsum, o);
            if (i + kDepth < kMaxPerWave) {
                bb[j] = bid(i + kDepth);
                load_block<D>(r[j], a.pool, a.num_kv_heads, g, bb[j], koff, voff);
            }
        }
        // The step's own token (position Lp): the wave that held its block attends
        // to it as a one-token tile built from k_new / v_new (its pool slot was
        // masked above) and writes it to that slot for later steps.  No other
        // workgroup reads the slot in this launch, and the same wave already
        // loaded the block, so the write races with no read that matters.
        if (own && cur_split == nsplit - 1) {
            const int bl = Lp / kBlock - blk0;             // the token's block within the split
            if (wave == bl % kDecWaves) {
                const int64_t row = ((int64_t)cur_s * a.num_kv_heads + g) * D;
                BlockRegs<D> nr;
#pragma unroll
                for (int ks = 0; ks < D / 32; ++ks) {
                    const u32x4 kv = *reinterpret_cast<const u32x4 *>(a.k_new + row + ks * 32 + g4 * 8);
                    nr.k[ks] = c16 == 0 ? kv : u32x4{0u, 0u, 0u, 0u};
                }
#pragma unroll
                for (int dt = 0; dt < D / 16; ++dt) {
                    const uint32_t v0 = a.v_new[row + dt * 16 + c16];
                    nr.v[dt] = u32x2{g4 == 0 ? v0 : 0u, 0u};
                }
                process_block<D>(nr, qop, Lp, Lp + 1, a.scale_log2, g4, m, lsum, o);
                const int blk = checked_id(cur_ids, bl, nblk);
                if (blk >= 0) {
                    const int t = Lp % kBlock;
                    uint16_t *pool = const_cast<uint16_t *>(a.pool);
                    const int64_t tile = (int64_t)kBlock * D;
                    uint16_t *kt = pool + ((int64_t)blk * 2 * a.num_kv_heads + g) * tile;
                    uint16_t *vt = kt + (int64_t)a.num_kv_heads * tile;
                    for (int d = lane; d < D; d += kWave) {
                        kt[((d >> 3) * kBlock + t) * 8 + (d & 7)] = a.k_new[row + d];
                        vt[d * kBlock + t] = a.v_new[row + d];
                    }
                }
            }
        }
        // Request the next item's first blocks and q before merging this one.
        if (has_next) {
            if (lane < kMaxSplitTokens / kBlock) sm_ids[wave][(k + 1) & 1][lane] = next_ids;
            const int g_next = next % a.num_kv_heads;
            const int nb = split_blocks(s, split);
            load_q(s, g_next, qop);
#pragma unroll
            for (int j = 0; j < kDepth; ++j) {
                bb[j] = checked_id(next_ids, wave + j * kDecWaves, nb);
                load_block<D>(r[j], a.pool, a.num_kv_heads, g_next, bb[j], koff, voff);
            }
        }
        lsum = wave_sum_xor_16_32(lsum);

        // ---- asynchronous merge of the item's waves: no workgroup barrier.
        const int slot = k & 1;
        // The slot is free once the merge of the item two steps back is done.
        // (Bounded: a wait that never ends would be a bug; it is flagged, not hung on.)
        for (int spin = 0; __hip_atomic_load(&sm_merged[slot], __ATOMIC_ACQUIRE,
                                             __HIP_MEMORY_SCOPE_WORKGROUP) != (k >> 1); ++spin) {
            if (spin == kSpinLimit) {
                if (lane == 0) flag_error(a.err, LS_DEVERR_INTERNAL);
                break;
            }
            __builtin_amdgcn_s_sleep(1);
        }
        if (c16 < G) {
#pragma unroll
            for (int dt = 0; dt < D / 16; ++dt)
                *reinterpret_cast<f32x4 *>(&sm_o[slot][wave][c16][dt * 16 + g4 * 4]) = o[dt];
            if (g4 == 0) {
                sm_m[slot][wave][c16] = m;
                sm_l[slot][wave][c16] = lsum;
            }
        }
        // One arrival per wave (lane 0), broadcast to the whole wave.
        int before = 0;
        if (lane == 0)
            before = __hip_atomic_fetch_add(&sm_arrived[slot], 1, __ATOMIC_ACQ_REL,
                                            __HIP_MEMORY_SCOPE_WORKGROUP);
        before = __builtin_amdgcn_readfirstlane(before);
        if (before == kDecWaves - 1) {
            // Last wave in: merge the item (4 consecutive outputs per lane per step).
            const int64_t part = ((int64_t)cur_s * a.num_kv_heads + g) * a.max_splits + cur_split;
            for (int base = lane * 4; base < G * D && L <= 0; base += kWave * 4)
                // Softmax over no key is undefined: the output is zero (flagged in attended_len).
                *reinterpret_cast<uint2 *>(a.out + ((int64_t)cur_s * hq_total + g * G) * D + base) =
                    make_uint2(0u, 0u);
            for (int base = lane * 4; base < G * D && L > 0; base += kWave * 4) {
                const int h = base / D, d = base % D;
                float M = sm_m[slot][0][h];
#pragma unroll
                for (int w = 1; w < kDecWaves; ++w) M = fmaxf(M, sm_m[slot][w][h]);
                float wsum = 0.f;
                f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int w = 0; w < kDecWaves; ++w) {
                    const float e = __builtin_amdgcn_exp2f(sm_m[slot][w][h] - M);
                    wsum += e * sm_l[slot][w][h];
                    acc += e * *reinterpret_cast<const f32x4 *>(&sm_o[slot][w][h][d]);
                }
                if (nsplit == 1) {
                    const float inv = 1.f / wsum;
                    *reinterpret_cast<uint2 *>(a.out + ((int64_t)cur_s * hq_total + g * G + h) * D + d) =
                        make_uint2(pack_bf16x2(acc[0] * inv, acc[1] * inv), pack_bf16x2(acc[2] * inv, acc[3] * inv));
                } else {
                    *reinterpret_cast<f32x4 *>(a.part_acc + (part * G + h) * D + d) = acc;
                    if (d == 0) {
                        a.part_ml[(part * G + h) * 2 + 0] = M;
                        a.part_ml[(part * G + h) * 2 + 1] = wsum;
                    }
                }
            }
            if (lane == 0) {
                __hip_atomic_store(&sm_arrived[slot], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
                __hip_atomic_fetch_add(&sm_merged[slot], 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
            }
        }
    }
}

// Log-sum-exp merge of the splits of every (session, KV head) with more than
// one.  1024 threads per (session, KV head): four groups of 256 threads each
// sum a quarter of the splits for 4 consecutive outputs, and the groups are
// added through LDS.  The first splits' outputs are requested before the split
// statistics (which do not depend on them), so the two loads share one memory
// latency; meanwhile each of the first G waves reduces one head's statistics
// with shuffles.
constexpr int kCombThreads = 1024;
constexpr int kCombParts = kCombThreads / 256;
constexpr int kCombPre = 8;                  // splits per thread loaded up front (32 per row)

template <int D>
__global__ __launch_bounds__(kCombThreads) void decode_combine_kernel(DecodeArgs a) {
    __shared__ float sm_e[kMaxSplits][kMaxGroup];          // exp2(m_k - M) per split and head
    __shared__ float sm_inv[kMaxGroup];                     // 1 / sum_k exp2(m_k - M) l_k
    __shared__ __attribute__((aligned(16))) float sm_acc[kCombParts - 1][256][4];
    const int g = blockIdx.x;
    const int s = blockIdx.y;
    const int L = attended_len(a, s, false);
    if (L <= 0) return;
    const int nsplit = (L + a.split_tokens - 1) / a.split_tokens;
    if (nsplit <= 1) return;
    const int G = a.group;
    const int hq_total = a.num_kv_heads * G;
    const int64_t part = ((int64_t)s * a.num_kv_heads + g) * a.max_splits;
    const int tid = threadIdx.x;
    const int wave = tid / kWave, lane = tid % kWave;
    const int c = tid % 256;                 // 4 consecutive outputs: base = 4c
    const int pidx = tid / 256;              // this thread sums splits pidx, pidx + 4, ...
    const int base = c * 4;
    const bool active = base < G * D;
    const float *src = a.part_acc + (part * G) * D + base;
    f32x4 pre[kCombPre];
#pragma unroll
    for (int i = 0; i < kCombPre; ++i) {
        const int k = pidx + i * kCombParts;
        pre[i] = active && k < nsplit ? *reinterpret_cast<const f32x4 *>(src + (int64_t)k * G * D)
                                      : f32x4{0.f, 0.f, 0.f, 0.f};
    }

    if (wave < G) {
        const int h = wave;
        float M = -INFINITY;
        for (int k = lane; k < nsplit; k += kWave) M = fmaxf(M, a.part_ml[((part + k) * G + h) * 2]);
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) M = fmaxf(M, __shfl_xor(M, off));
        float wsum = 0.f;
        for (int k = lane; k < nsplit; k += kWave) {
            const float e = __builtin_amdgcn_exp2f(a.part_ml[((part + k) * G + h) * 2] - M);
            sm_e[k][h] = e;
            wsum += e * a.part_ml[((part + k) * G + h) * 2 + 1];
        }
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) wsum += __shfl_xor(wsum, off);
        if (lane == 0) sm_inv[h] = 1.f / wsum;
    }
    __syncthreads();

    const int h = active ? base / D : 0;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    if (active) {
#pragma unroll
        for (int i = 0; i < kCombPre; ++i) {
            const int k = pidx + i * kCombParts;
            if (k < nsplit) acc += sm_e[k][h] * pre[i];
        }
        int k = pidx + kCombPre * kCombParts;
        for (; k + 3 * kCombParts < nsplit; k += 4 * kCombParts) {
            const f32x4 v0 = *reinterpret_cast<const f32x4 *>(src + (int64_t)k * G * D);
            const f32x4 v1 = *reinterpret_cast<const f32x4 *>(src + (int64_t)(k + kCombParts) * G * D);
            const f32x4 v2 = *reinterpret_cast<const f32x4 *>(src + (int64_t)(k + 2 * kCombParts) * G * D);
            const f32x4 v3 = *reinterpret_cast<const f32x4 *>(src + (int64_t)(k + 3 * kCombParts) * G * D);
            acc += sm_e[k][h] * v0 + sm_e[k + kCombParts][h] * v1 + sm_e[k + 2 * kCombParts][h] * v2 +
                   sm_e[k + 3 * kCombParts][h] * v3;
        }
        for (; k < nsplit; k += kCombParts)
            acc += sm_e[k][h] * *reinterpret_cast<const f32x4 *>(src + (int64_t)k * G * D);
    }
    if (pidx > 0) *reinterpret_cast<f32x4 *>(sm_acc[pidx - 1][c]) = acc;
    __syncthreads();
    if (pidx == 0 && active) {
#pragma unroll
        for (int q2 = 0; q2 < kCombParts - 1; ++q2) acc += *reinterpret_cast<const f32x4 *>(sm_acc[q2][c]);
        const float inv = sm_inv[h];
        *reinterpret_cast<uint2 *>(a.out + ((int64_t)s * hq_total + g * G) * D + base) =
            make_uint2(pack_bf16x2(acc[0] * inv, acc[1] * inv), pack_bf16x2(acc[2] * inv, acc[3] * inv));
    }
}

}  // namespace

DecodePlan plan_decode(const PoolGeom &p, int32_t num_sessions, int32_t num_q_heads,
                       int32_t max_blocks_per_session) {
    DecodePlan plan{};
    const int64_t max_tokens = (int64_t)max_blocks_per_session * kBlock;
    const int64_t work = (int64_t)num_sessions * p.num_kv_heads * max_tokens;
    // Splits of 512 or 1024 tokens (4 or 8 blocks per wave): long enough to
    // amortise an item's start-up, short enough to give every CU several items
    // on a large batch.
    int T = 1024;
    if (work < 256LL * 2 * 4 * 512) T = 512;
    while (T < kMaxSplitTokens && (max_tokens + T - 1) / T > kMaxSplits) T *= 2;
    plan.split_tokens = T;
    plan.max_splits = (int)((max_tokens + T - 1) / T);
    if (plan.max_splits < 1) plan.max_splits = 1;
    plan.supported = plan.max_splits <= kMaxSplits && num_sessions <= kMaxBatch;
    const int G = p.num_kv_heads > 0 ? num_q_heads / p.num_kv_heads : 0;
    const int64_t sg = (int64_t)num_sessions * p.num_kv_heads;
    auto pad = [](size_t b) { return (b + 255) & ~(size_t)255; };
    plan.ml_bytes = pad((size_t)sg * plan.max_splits * G * 2 * sizeof(float));
    plan.acc_bytes = pad((size_t)sg * plan.max_splits * G * p.head_dim * sizeof(float));
    return plan;
}

hipError_t launch_decode(const PoolGeom &p, int layer, int32_t num_sessions, int32_t num_q_heads,
                         const uint16_t *q, const uint16_t *k_new, const uint16_t *v_new,
                         const int32_t *block_tables,
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
    a.appended = k_new != nullptr ? 1 : 0;
    a.k_new = k_new;
    a.v_new = v_new;
    a.scale_log2 = scale * kLog2e;
    a.err = err;
    a.split_tokens = plan.split_tokens;
    a.max_splits = plan.max_splits;
    uint8_t *ws = static_cast<uint8_t *>(workspace);
    a.part_ml = reinterpret_cast<float *>(ws);
    a.part_acc = reinterpret_cast<float *>(ws + plan.ml_bytes);
    a.num_sessions = num_sessions;
    const int64_t upper = (int64_t)num_sessions * p.num_kv_heads * plan.max_splits;
    // Persistent grid: one 512-thread workgroup (8 waves, this kernel's
    // occupancy) on every CU the stream may use.
    const int64_t resident = (int64_t)stream_cus(p, stream);
    dim3 grid((unsigned)std::min<int64_t>(upper, resident));
#define LS_DECODE(DD, PW) \
    hipLaunchKernelGGL((decode_kernel<DD, 2, PW>), grid, dim3(kDecThreads), 0, stream, a)
    const int per_wave = plan.split_tokens / (kDecWaves * kBlock);
    if (p.head_dim == 128) {
        if (per_wave == 4) LS_DECODE(128, 4);
        else LS_DECODE(128, 8);
    } else {
        if (per_wave == 4) LS_DECODE(64, 4);
        else LS_DECODE(64, 8);
    }
#undef LS_DECODE
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || plan.max_splits == 1) return e;
    dim3 cgrid(p.num_kv_heads, num_sessions);
    if (p.head_dim == 128)
        hipLaunchKernelGGL(decode_combine_kernel<128>, cgrid, dim3(kCombThreads), 0, stream, a);
    else
        hipLaunchKernelGGL(decode_combine_kernel<64>, cgrid, dim3(kCombThreads), 0, stream, a);
    return hipGetLastError();
}

}  // namespace ls
