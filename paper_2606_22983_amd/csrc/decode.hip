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
#include <cstring>
#include <cstdlib>
#include <type_traits>
#include <vector>

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
constexpr int kMaxDeviceSplit = 2048;       // longest split of the kernel's own schedule (two chunks)
constexpr int kKeyBins = kMaxDeviceSplit / kBlock + 1;   // short-split block counts 0..128
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

// A schedule planned on the host (paged_attn_decode with host lengths),
// passed by value in the kernel arguments: workgroup w runs items
// start[w] .. start[w + 1] - 1.  Items are 32-bit words (session in bits
// 0..11, KV head 12..19, split 20..30, "last split the plan gives the
// session" 31), or, when the start[] entries carry kPlanCompactBit, 16-bit halves of them
// (session 0..9, KV head 10..11, split 12..14, last split 15), which holds
// twice as many items for batches of at most 1024 sessions, 4 KV heads and 8
// splits per session.  Plans that fit go in a ~3 KiB argument block; larger
// batches take a ~16 KiB one (the runtime passes kernel arguments of that
// size intact), so the common launch copies no more than it needs.
constexpr int kPlanMaxWg = 256;
constexpr int kPlanItemsSmall = 640;                   // 32-bit words: 640 or 1280 items
constexpr int kPlanItemsLarge = 3840;                  // 32-bit words: 3840 or 7680 items
constexpr uint32_t kPlanCompactBit = 0x8000u;          // in every start[] entry: 16-bit items
template <int kItems>
struct DecodeHostPlanT {
    uint16_t start[kPlanMaxWg + 2];            // | kPlanCompactBit: 16-bit items; [kPlanMaxWg + 1]: unused
    uint32_t item[kItems];
};
using DecodeHostPlan = DecodeHostPlanT<kPlanItemsSmall>;
using DecodeHostPlanLarge = DecodeHostPlanT<kPlanItemsLarge>;
struct NoPlan {
    int32_t unused;
};
template <bool kHost, int kItems>
using PlanArg = typename std::conditional<kHost, DecodeHostPlanT<kItems>, NoPlan>::type;
// Items [first, end) of workgroup w and the item width: start[w] and
// start[w + 1], read as the two aligned 32-bit words from start[w & ~1] on, in
// one scalar load (those need 4-byte alignment).  Every entry carries the
// width flag, so no other load is needed before the first item's.
template <int kItems>
__device__ __forceinline__ void plan_range(const DecodeHostPlanT<kItems> &p, int w, int &first, int &end,
                                           bool &compact) {
    uint32_t word[2];
    __builtin_memcpy(word, &p.start[w & ~1], sizeof word);
    const uint32_t lo = (w & 1) ? word[0] >> 16 : word[0] & 0xFFFFu;
    const uint32_t hi = (w & 1) ? word[1] & 0xFFFFu : word[0] >> 16;
    first = (int)(lo & ~kPlanCompactBit);
    end = (int)(hi & ~kPlanCompactBit);
    compact = (lo & kPlanCompactBit) != 0;
}
__device__ __forceinline__ void plan_range(const NoPlan &, int, int &first, int &end, bool &compact) {
    first = end = 0;
    compact = false;
}
// Item i in the 32-bit layout: one load either way (the word index is
// selected, not branched on).
template <int kItems>
__device__ __forceinline__ uint32_t plan_item(const DecodeHostPlanT<kItems> &p, int i, bool compact) {
    const uint32_t word = p.item[compact ? i >> 1 : i];
    if (!compact) return word;
    const uint32_t h = (word >> ((i & 1) * 16)) & 0xFFFFu;
    return (h & 0x3FFu) | (((h >> 10) & 3u) << 12) | (((h >> 12) & 7u) << 20) | ((h >> 15) << 31);
}

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
// items (session s, split k, KV head g).
//
// Device-planned schedule (kHost false): each workgroup first orders, in LDS,
// the work rows (session, split) longest first: every full split (T tokens),
// then each session's last, shorter split by block count, largest first (an
// empty session's one row is among them).  Items are dealt in snake order:
// round k gives item k*W + w to workgroup w for even k and k*W + W-1-w for odd
// k (W workgroups), so every workgroup receives about the same number of
// tokens; with plain round-robin the workgroups holding one item more than the
// rest decide the call's duration.  Every workgroup derives the same order
// from the lengths, and no workgroup is launched for a split that does not
// exist.
//
// Host-planned schedule (kHost): the host, which knows the lengths, chose the
// split size and gave each workgroup its list of items in the kernel
// arguments; the workgroup only loads the lengths.  An item may then span
// several chunks of kChunk tokens (8 blocks per wave); the online-softmax
// state is carried from chunk to chunk and the waves merge once per item.
//
// Either way each workgroup fetches the next chunk's block ids while it works
// on the current one, and requests its first blocks before merging.
template <int D, int kDepth, int kMaxPerWave, bool kHost, int kItems = kPlanItemsSmall>
__global__ __launch_bounds__(kDecThreads) void decode_kernel(DecodeArgs a, PlanArg<kHost, kItems> plan) {
    constexpr int kChunk = kMaxPerWave * kDecWaves * kBlock;   // tokens per chunk
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
    int full_rows = 0, total_rows = 0;
    if constexpr (!kHost) {
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
        full_rows = (int)(packed_total & 0xFFFFFu);
        total_rows = full_rows + (int)(packed_total >> 20);
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
    }
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

    // (session, split) of work row r of the device schedule.  A full row: the
    // largest s with sm_cum[s] <= r (a session without full splits shares its
    // sm_cum with the next session, so it is never the largest).  A short row:
    // its session's last split.
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
    // This workgroup's k-th item: (session, KV head, split, last split the
    // plan gives the session), or false past its last item.
    int host_base, host_end;
    bool host_compact;
    plan_range(plan, (int)blockIdx.x, host_base, host_end, host_compact);
    const int host_count = host_end - host_base;
    auto item_at = [&](int k, int &s_out, int &g_out, int &split_out, bool &last_out) -> bool {
        if constexpr (kHost) {
            if (k >= host_count) return false;
            const uint32_t e = plan_item(plan, host_base + k, host_compact);
            s_out = (int)(e & 0xFFFu);
            g_out = (int)((e >> 12) & 0xFFu);
            split_out = (int)((e >> 20) & 0x7FFu);
            last_out = (e >> 31) != 0;
            return true;
        } else {
            const int item = item_of(k);
            if (item >= total_items) return false;
            locate(item / a.num_kv_heads, s_out, split_out);
            g_out = item % a.num_kv_heads;
            last_out = false;
            return true;
        }
    };
    // Raw block ids of chunk c of a split, one per lane.  The load is
    // unconditional (its index clamped into the table row) and the id is
    // validated only when it is used, so nothing waits for this load until the
    // chunk is processed.
    auto fetch_ids = [&](int s_, int split_, int c_) -> int {
        const int j = min(split_ * (T / kBlock) + c_ * (kChunk / kBlock) + lane, a.max_blocks - 1);
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
    // Block count of chunk c of a split: tokens [t0, min(L, split end, t0 + kChunk)).
    auto chunk_blocks = [&](int L, int split_, int c_) -> int {
        const int t0 = split_ * T + c_ * kChunk;
        const int t1 = min(min(L, split_ * T + T), t0 + kChunk);
        return t1 > t0 ? (t1 + kBlock - 1) / kBlock - t0 / kBlock : 0;
    };

    // kDepth blocks in flight per wave, carried across chunks and items: the
    // next chunk's first blocks (and, for a new item, its q) are requested
    // before the current item is merged.
    BlockRegs<D> r[kDepth];
    int bb[kDepth];
    bf16x8 qop[D / 32];
    // Each wave keeps the fetched block ids of the current and the next chunk in
    // its own LDS slots (double-buffered; read back with readlane), so no value
    // loaded from memory is carried around the loop.
    __shared__ int sm_ids[kDecWaves][2][kMaxSplitTokens / kBlock];
    int k = 0, c = 0;                  // current item (index in this workgroup's list) and chunk
    int s = 0, g = 0, split = 0;
    bool last_planned = false;
    bool have = item_at(0, s, g, split, last_planned);
    int ids_pre = have ? fetch_ids(s, split, 0) : -1;
    if (have) load_q(s, g, qop);
    if constexpr (kHost) {
        // The schedule came with the arguments, so only the lengths are needed.
        // They are loaded after the first item's block ids and q, whose loads
        // are then already in flight.
        for (int i = tid; i < S; i += kDecThreads) {
            sm_len[i] = attended_len(a, i, blockIdx.x == 0);
            sm_own[i] = a.appended && a.lens[i] >= 0 && a.lens[i] + 1 <= a.max_blocks * kBlock;
        }
        __syncthreads();
    }
    if (have) {
        if (lane < kMaxSplitTokens / kBlock) sm_ids[wave][0][lane] = ids_pre;
        const int nb = chunk_blocks(sm_len[s], split, 0);
#pragma unroll
        for (int j = 0; j < kDepth; ++j) {
            bb[j] = checked_id(ids_pre, wave + j * kDecWaves, nb);
            load_block<D>(r[j], a.pool, a.num_kv_heads, g, bb[j], koff, voff);
        }
    }
    float m = kMaxFloor, lsum = 0.f;
    f32x4 o[D / 16];
    int merges = 0;
    for (int u = 0; have; ++u) {
        const int L = sm_len[s];
        const int own = sm_own[s];
        const int Lp = L - own;            // keys read from the pool; the own token comes from k_new
        const int cur_s = s, cur_g = g, cur_split = split, cur_c = c;
        const bool cur_last_planned = last_planned;
        const int cur_ids = lane < kMaxSplitTokens / kBlock ? sm_ids[wave][u & 1][lane] : -1;
        const int t_split_end = min(L, cur_split * T + T);
        const int t0 = cur_split * T + cur_c * kChunk;
        const bool last_chunk = t0 + kChunk >= t_split_end;
        // Next chunk: the same item's, or the next item's first; its ids fetched now.
        int next_ids = -1;
        if (last_chunk) {
            ++k;
            c = 0;
            have = item_at(k, s, g, split, last_planned);
        } else {
            ++c;
        }
        if (have) next_ids = fetch_ids(s, split, c);
        const int nsplit = L > 0 ? (L + T - 1) / T : 1;
        const int blk0 = t0 / kBlock;
        const int nblk = chunk_blocks(L, cur_split, cur_c);
        const int my_n = wave < nblk ? (nblk - wave + kDecWaves - 1) / kDecWaves : 0;
        auto bid = [&](int it) -> int { return checked_id(cur_ids, wave + it * kDecWaves, nblk); };

        // A new item's running max starts at a finite floor: a block whose keys
        // are all masked then leaves (m, l, O) unchanged instead of producing NaN.
        if (cur_c == 0) {
            m = kMaxFloor;
            lsum = 0.f;
#pragma unroll
            for (int dt = 0; dt < D / 16; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
        }

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
                load_block<D>(r[j], a.pool, a.num_kv_heads, cur_g, bb[j], koff, voff);
            }
        }
        // The step's own token (position Lp): the wave that held its block attends
        // to it as a one-token tile built from k_new / v_new (its pool slot was
        // masked above) and writes it to that slot for later steps.  No other
        // workgroup reads the slot in this launch, and the same wave already
        // loaded the block, so the write races with no read that matters.
        if (own && cur_split == nsplit - 1 && last_chunk) {
            const int bl = Lp / kBlock - blk0;             // the token's block within the chunk
            if (wave == bl % kDecWaves) {
                const int64_t row = ((int64_t)cur_s * a.num_kv_heads + cur_g) * D;
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
                    uint16_t *kt = pool + ((int64_t)blk * 2 * a.num_kv_heads + cur_g) * tile;
                    uint16_t *vt = kt + (int64_t)a.num_kv_heads * tile;
                    for (int d = lane; d < D; d += kWave) {
                        kt[((d >> 3) * kBlock + t) * 8 + (d & 7)] = a.k_new[row + d];
                        vt[d * kBlock + t] = a.v_new[row + d];
                    }
                }
            }
        }
        // Request the next chunk's first blocks (and a new item's q) before
        // merging this item.
        if (have) {
            if (lane < kMaxSplitTokens / kBlock) sm_ids[wave][(u + 1) & 1][lane] = next_ids;
            const int nb = chunk_blocks(sm_len[s], split, c);
            if (c == 0) load_q(s, g, qop);
#pragma unroll
            for (int j = 0; j < kDepth; ++j) {
                bb[j] = checked_id(next_ids, wave + j * kDecWaves, nb);
                load_block<D>(r[j], a.pool, a.num_kv_heads, g, bb[j], koff, voff);
            }
        }
        if (!last_chunk) continue;         // the item goes on: (m, l, O) carry over
        // A host plan that stops short of the session's keys leaves them
        // unattended: flagged (the device lengths differ from the host's).
        if (kHost && cur_last_planned && cur_split * T + T < L && lane == 0 && wave == 0)
            flag_error(a.err, LS_DEVERR_LENGTH);
        const float lsum_w = wave_sum_xor_16_32(lsum);

        // ---- asynchronous merge of the item's waves: no workgroup barrier.
        const int slot = merges & 1;
        // The slot is free once the merge of the item two merges back is done.
        // (Bounded: a wait that never ends would be a bug; it is flagged, not hung on.)
        for (int spin = 0; __hip_atomic_load(&sm_merged[slot], __ATOMIC_ACQUIRE,
                                             __HIP_MEMORY_SCOPE_WORKGROUP) != (merges >> 1); ++spin) {
            if (spin == kSpinLimit) {
                if (lane == 0) flag_error(a.err, LS_DEVERR_INTERNAL);
                break;
            }
            __builtin_amdgcn_s_sleep(1);
        }
        ++merges;
        if (c16 < G) {
#pragma unroll
            for (int dt = 0; dt < D / 16; ++dt)
                *reinterpret_cast<f32x4 *>(&sm_o[slot][wave][c16][dt * 16 + g4 * 4]) = o[dt];
            if (g4 == 0) {
                sm_m[slot][wave][c16] = m;
                sm_l[slot][wave][c16] = lsum_w;
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
            // A split past the session's last (device lengths shorter than the
            // host plan assumed) writes nothing.
            const int64_t part = ((int64_t)cur_s * a.num_kv_heads + cur_g) * a.max_splits + cur_split;
            const bool writes = cur_split < nsplit;
            for (int base = lane * 4; base < G * D && L <= 0; base += kWave * 4)
                // Softmax over no key is undefined: the output is zero (flagged in attended_len).
                *reinterpret_cast<uint2 *>(a.out + ((int64_t)cur_s * hq_total + cur_g * G) * D + base) =
                    make_uint2(0u, 0u);
            for (int base = lane * 4; base < G * D && L > 0 && writes; base += kWave * 4) {
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
                    *reinterpret_cast<uint2 *>(a.out + ((int64_t)cur_s * hq_total + cur_g * G + h) * D + d) =
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
    // Splits of 512, 1024 or 2048 tokens (4 or 8 blocks per wave per 1024-token
    // chunk): long enough to amortise an item's start-up and the merges, short
    // enough to give every CU several items.  2048 when the batch would still
    // give every CU at least three items of that size (thinker batch: 142.7 ->
    // 134.4 us per call, talker step: 116.5 -> 110.4 us, against 1024).
    const int64_t cus = p.num_cus > 0 ? p.num_cus : 256;
    int T = 1024;
    if (work < 256LL * 2 * 4 * 512) T = 512;
    else if ((int64_t)num_sessions * p.num_kv_heads * ((max_tokens + kMaxDeviceSplit - 1) / kMaxDeviceSplit) >=
             3 * cus)
        T = kMaxDeviceSplit;
    while (T < kMaxSplitTokens && (max_tokens + T - 1) / T > kMaxSplits) T *= 2;
    plan.split_tokens = T;
    plan.max_splits = (int)((max_tokens + T - 1) / T);
    if (plan.max_splits < 1) plan.max_splits = 1;
    // Tables of up to kMaxSplits splits of the 1024-token chunk (16384 blocks),
    // whatever split size this batch gets.
    plan.supported = plan.max_splits <= kMaxSplits && num_sessions <= kMaxBatch &&
                     max_tokens <= (int64_t)kMaxSplits * kMaxSplitTokens;
    const int G = p.num_kv_heads > 0 ? num_q_heads / p.num_kv_heads : 0;
    const int64_t sg = (int64_t)num_sessions * p.num_kv_heads;
    auto pad = [](size_t b) { return (b + 255) & ~(size_t)255; };
    plan.ml_bytes = pad((size_t)sg * plan.max_splits * G * 2 * sizeof(float));
    plan.acc_bytes = pad((size_t)sg * plan.max_splits * G * p.head_dim * sizeof(float));
    return plan;
}

namespace {

// Host-side schedule (see DecodeHostPlan).  Chooses the split size T (a
// multiple of 1024 tokens, at least t_min) among: no split at all (T covers
// the longest session), 2048, 3072 and 4096, by the cost of a longest-first
// assignment of the items to the workgroups: the most loaded workgroup's
// tokens plus a fixed cost per item, plus the merge kernel's cost when some
// session is split.  Items then go, longest first, to the least loaded
// workgroup; each workgroup runs its items in that order.  Gives up (false)
// when the batch does not fit the argument block (more workgroups or items),
// or when the device's own schedule (split size t_dev, snake-dealt rows; its
// merge launched whenever dev_merges) is estimated to finish no later.
constexpr int64_t kItemCostTokens = 64;      // per-item start-up, in tokens of streaming
constexpr int64_t kMergeCostTokens = 256;    // the split merge launch, in tokens
constexpr int64_t kScheduleCostTokens = 128; // the device schedule in the kernel prologue, in tokens

// Least-loaded-first assignment over W workgroups: a binary min-heap of keys
// load * 512 + workgroup (W <= 256), ties to the lower workgroup.
struct LoadHeap {
    uint64_t key[kPlanMaxWg];
    int n;
    void reset(int W) {
        n = W;
        for (int w = 0; w < W; ++w) key[w] = (uint64_t)w;     // already a heap
    }
    // Adds `cost` to the least loaded workgroup; returns it and its new load.
    int add(int64_t cost, int64_t &new_load) {
        const uint64_t k = key[0] + ((uint64_t)cost << 9);
        const int w = (int)(k & 511u);
        new_load = (int64_t)(k >> 9);
        int i = 0;                               // sift the grown key down
        for (;;) {
            const int l = 2 * i + 1;
            if (l >= n) break;
            const int m = (l + 1 < n && key[l + 1] < key[l]) ? l + 1 : l;
            if (key[m] >= k) break;
            key[i] = key[m];
            i = m;
        }
        key[i] = k;
        return w;
    }
};

struct PlanRow {
    int32_t tokens, s, split;
};

bool plan_decode_host(int S, int num_kv_heads, const int32_t *lens_host, int appended, int W, int t_min,
                      int t_dev, bool dev_merges, DecodeHostPlanLarge &plan, int &t_out, bool &any_split) {
    if (W < 1 || W > kPlanMaxWg || S > 4096 || num_kv_heads > 255) return false;
    int64_t max_len = 1;
    for (int s = 0; s < S; ++s) max_len = std::max<int64_t>(max_len, (int64_t)lens_host[s] + appended);
    auto len_of = [&](int s) { return std::max<int64_t>((int64_t)lens_host[s] + appended, 1); };
    // The device schedule's estimated makespan: rows of full splits in session
    // order, then the short rows by block count (largest first), each row's
    // heads consecutive, dealt in snake order.
    static thread_local std::vector<int64_t> dev_load;
    static thread_local std::vector<int32_t> shorts;
    dev_load.assign(W, 0);
    shorts.clear();
    int dw = 0, dround = 0;                     // snake position: round parity and slot
    auto deal = [&](int64_t tokens) {
        for (int g = 0; g < num_kv_heads; ++g) {
            dev_load[(dround & 1) ? W - 1 - dw : dw] += tokens + kItemCostTokens;
            if (++dw == W) {
                dw = 0;
                ++dround;
            }
        }
    };
    for (int s = 0; s < S; ++s) {
        const int64_t L = std::max<int64_t>((int64_t)lens_host[s] + appended, 0);
        for (int64_t k = 0; k < L / t_dev; ++k) deal(t_dev);
        if (L == 0 || L % t_dev) shorts.push_back((int32_t)((L % t_dev + kBlock - 1) / kBlock));
    }
    std::stable_sort(shorts.begin(), shorts.end(), std::greater<int32_t>());
    for (int32_t b : shorts) deal((int64_t)b * kBlock);
    const int64_t dev_cost = *std::max_element(dev_load.begin(), dev_load.end()) + kScheduleCostTokens +
                             (dev_merges ? kMergeCostTokens : 0);

    // Rows (session, split) of a split size, longest first (ties: session, split).
    static thread_local std::vector<PlanRow> rows;
    static thread_local LoadHeap heap;
    bool compact = false;
    auto build = [&](int T) -> bool {
        rows.clear();
        const int64_t ns_max = (max_len + T - 1) / T;
        compact = S <= 1024 && num_kv_heads <= 4 && ns_max <= 8;
        const int64_t cap = compact ? 2 * kPlanItemsLarge : kPlanItemsLarge;
        if (ns_max > 2047) return false;
        int64_t n_items = 0;
        for (int s = 0; s < S; ++s) {
            const int64_t L = len_of(s);
            const int ns = (int)((L + T - 1) / T);
            n_items += (int64_t)ns * num_kv_heads;
            if (n_items > cap) return false;
            for (int k = 0; k < ns; ++k)
                rows.push_back({(int32_t)(std::min<int64_t>(L, (int64_t)(k + 1) * T) - (int64_t)k * T), s, k});
        }
        std::sort(rows.begin(), rows.end(), [](const PlanRow &x, const PlanRow &y) {
            return x.tokens != y.tokens ? x.tokens > y.tokens : (x.s != y.s ? x.s < y.s : x.split < y.split);
        });
        return true;
    };
    // LPT over the rows' items; optionally records the plan.  With a bound it
    // stops as soon as the makespan reaches it.
    auto assign = [&](int64_t bound, bool record) -> int64_t {
        heap.reset(W);
        int64_t worst = 0;
        int slot_of[kPlanMaxWg];
        static thread_local std::vector<uint32_t> order;    // (workgroup << 16 | item) per item, in order
        if (record) order.clear();
        for (const PlanRow &r : rows)
            for (int g = 0; g < num_kv_heads; ++g) {
                int64_t nl;
                const int w = heap.add(r.tokens + kItemCostTokens, nl);
                worst = std::max(worst, nl);
                if (!record && worst >= bound) return worst;    // cannot win
                if (record) order.push_back(((uint32_t)w << 16) | (uint32_t)order.size());
            }
        if (!record) return worst;
        // Per-workgroup item lists in assignment order.
        int count[kPlanMaxWg + 1] = {0};
        for (uint32_t o : order) ++count[(o >> 16) + 1];
        for (int w = 0; w < W; ++w) count[w + 1] += count[w];
        for (int w = 0; w <= W; ++w) plan.start[w] = (uint16_t)(count[w] | (compact ? kPlanCompactBit : 0u));
        plan.start[kPlanMaxWg + 1] = 0;
        for (int w = 0; w < W; ++w) slot_of[w] = count[w];
        size_t i = 0;
        for (const PlanRow &r : rows) {
            const bool last = (int64_t)(r.split + 1) * t_out >= len_of(r.s);
            for (int g = 0; g < num_kv_heads; ++g, ++i) {
                const int slot = slot_of[order[i] >> 16]++;
                if (compact) {
                    const uint32_t h = (uint32_t)r.s | ((uint32_t)g << 10) | ((uint32_t)r.split << 12) |
                                       (last ? 0x8000u : 0u);
                    uint32_t &word = plan.item[slot >> 1];
                    const int sh = (slot & 1) * 16;
                    word = (word & ~(0xFFFFu << sh)) | (h << sh);
                } else {
                    plan.item[slot] = (uint32_t)r.s | ((uint32_t)g << 12) | ((uint32_t)r.split << 20) |
                                      (last ? 0x80000000u : 0u);
                }
            }
        }
        return worst;
    };
    // Candidates are ranked by the snake dealing of their rows' items (linear
    // time); the chosen one is then assigned longest-first to the least loaded
    // workgroup, and kept only if that still beats the device schedule.
    auto snake = [&]() -> int64_t {
        static thread_local std::vector<int64_t> load;
        load.assign(W, 0);
        int w = 0, round = 0;
        for (const PlanRow &r : rows)
            for (int g = 0; g < num_kv_heads; ++g) {
                load[(round & 1) ? W - 1 - w : w] += r.tokens + kItemCostTokens;
                if (++w == W) {
                    w = 0;
                    ++round;
                }
            }
        return *std::max_element(load.begin(), load.end());
    };
    const int unit = 1024;
    const int t_whole = (int)((max_len + unit - 1) / unit * unit);
    const int cands[4] = {t_whole, 2048, 3072, 4096};
    int best_t = 0;
    int64_t best_est = INT64_MAX;
    for (int T : cands) {
        T = std::max(T, t_min);
        if (T % unit || T > t_whole) continue;
        if (!build(T)) continue;
        const int64_t est = snake() + (T < max_len ? kMergeCostTokens : 0);
        if (est < best_est) {
            best_est = est;
            best_t = T;
        }
    }
    if (!best_t || !build(best_t)) return false;
    t_out = best_t;
    any_split = best_t < max_len;
    const int64_t cost = assign(INT64_MAX, true) + (any_split ? kMergeCostTokens : 0);
    return cost < dev_cost;
}

// The last host plans (one per batch shape), reused while every session keeps
// its split count and the batch's tokens stay within 1/32 of the planned
// ones: a decode loop's lengths grow by one token per step, which changes
// neither the items nor, noticeably, their balance.
struct CachedPlan {
    bool used = false, host = false, split = false;
    bool large = false;                        // the plan needs the large argument block
    int S = 0, hkv = 0, appended = 0, W = 0, t_min = 0, t_dev = 0, T = 0;
    bool dev_merges = false;
    int64_t tokens = 0;
    std::vector<uint16_t> nsplits;
    DecodeHostPlanLarge plan;
    DecodeHostPlan small;                      // the same plan, when it fits
};

const CachedPlan *cached_decode_plan(int S, int hkv, const int32_t *lens_host, int appended, int W, int t_min,
                                    int t_dev, bool dev_merges) {
    static thread_local CachedPlan cache[4];
    static thread_local int next_victim = 0;
    int64_t tokens = 0;
    for (int s = 0; s < S; ++s) tokens += (int64_t)lens_host[s] + appended;
    for (CachedPlan &c : cache) {
        if (!c.used || c.S != S || c.hkv != hkv || c.appended != appended || c.W != W || c.t_min != t_min ||
            c.t_dev != t_dev || c.dev_merges != dev_merges)
            continue;
        if (std::llabs(tokens - c.tokens) * 32 > c.tokens) continue;
        const int T = c.host ? c.T : t_dev;
        bool same = true;
        for (int s = 0; s < S && same; ++s) {
            const int64_t L = std::max<int64_t>((int64_t)lens_host[s] + appended, 1);
            same = (L + T - 1) / T == c.nsplits[s];
        }
        if (same) return &c;
    }
    CachedPlan &c = cache[next_victim];
    next_victim = (next_victim + 1) % 4;
    c.used = true;
    c.S = S;
    c.hkv = hkv;
    c.appended = appended;
    c.W = W;
    c.t_min = t_min;
    c.t_dev = t_dev;
    c.dev_merges = dev_merges;
    c.tokens = tokens;
    c.host = plan_decode_host(S, hkv, lens_host, appended, W, t_min, t_dev, dev_merges, c.plan, c.T, c.split);
    if (c.host) {
        const int items = c.plan.start[W] & ~kPlanCompactBit;
        const int words = (c.plan.start[W] & kPlanCompactBit) ? (items + 1) / 2 : items;
        c.large = words > kPlanItemsSmall;
        if (!c.large) {
            std::memcpy(c.small.start, c.plan.start, sizeof c.small.start);
            std::memcpy(c.small.item, c.plan.item, sizeof(uint32_t) * (size_t)words);
        }
    }
    const int T = c.host ? c.T : t_dev;
    c.nsplits.resize(S);
    for (int s = 0; s < S; ++s) {
        const int64_t L = std::max<int64_t>((int64_t)lens_host[s] + appended, 1);
        c.nsplits[s] = (uint16_t)std::min<int64_t>((L + T - 1) / T, 65535);
    }
    return &c;
}

}  // namespace

DecodeSchedule decode_schedule(const PoolGeom &p, int32_t num_sessions, const int32_t *context_lens_host,
                               int32_t appended, const DecodePlan &plan, hipStream_t stream) {
    DecodeSchedule sc{plan.split_tokens, false, plan.max_splits > 1};
    if (context_lens_host) {
        const CachedPlan *c = cached_decode_plan(num_sessions, p.num_kv_heads, context_lens_host, appended,
                                                 stream_cus(p, stream), std::max(plan.split_tokens, 1024),
                                                 plan.split_tokens, plan.max_splits > 1);
        if (c->host) sc = DecodeSchedule{c->T, true, c->split};
    }
    return sc;
}

hipError_t launch_decode(const PoolGeom &p, int layer, int32_t num_sessions, int32_t num_q_heads,
                         const uint16_t *q, const uint16_t *k_new, const uint16_t *v_new,
                         const int32_t *block_tables,
                         int32_t max_blocks, const int32_t *context_lens, const int32_t *context_lens_host,
                         float scale, uint16_t *out, void *workspace, const DecodePlan &plan,
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
    const int64_t resident = (int64_t)stream_cus(p, stream);
    dim3 cgrid(p.num_kv_heads, num_sessions);
    // Host lengths: the schedule is planned here and passed with the arguments.
    if (context_lens_host) {
        const CachedPlan *c = cached_decode_plan(num_sessions, p.num_kv_heads, context_lens_host, a.appended,
                                                 (int)resident, std::max(plan.split_tokens, 1024),
                                                 plan.split_tokens, plan.max_splits > 1);
        if (c->host) {
            const bool split = c->split;
            a.split_tokens = c->T;
            const dim3 grid((unsigned)resident);
            if (!c->large) {
                if (p.head_dim == 128)
                    hipLaunchKernelGGL((decode_kernel<128, 2, 8, true>), grid, dim3(kDecThreads), 0, stream, a, c->small);
                else
                    hipLaunchKernelGGL((decode_kernel<64, 2, 8, true>), grid, dim3(kDecThreads), 0, stream, a, c->small);
            } else if (p.head_dim == 128) {
                hipLaunchKernelGGL((decode_kernel<128, 2, 8, true, kPlanItemsLarge>), grid, dim3(kDecThreads), 0,
                                   stream, a, c->plan);
            } else {
                hipLaunchKernelGGL((decode_kernel<64, 2, 8, true, kPlanItemsLarge>), grid, dim3(kDecThreads), 0,
                                   stream, a, c->plan);
            }
            hipError_t e = hipGetLastError();
            if (e != hipSuccess || !split) return e;
            if (p.head_dim == 128)
                hipLaunchKernelGGL(decode_combine_kernel<128>, cgrid, dim3(kCombThreads), 0, stream, a);
            else
                hipLaunchKernelGGL(decode_combine_kernel<64>, cgrid, dim3(kCombThreads), 0, stream, a);
            return hipGetLastError();
        }
    }
    const int64_t upper = (int64_t)num_sessions * p.num_kv_heads * plan.max_splits;
    // Persistent grid: one 512-thread workgroup (8 waves, this kernel's
    // occupancy) on every CU the stream may use.
    dim3 grid((unsigned)std::min<int64_t>(upper, resident));
    const NoPlan none{0};
#define LS_DECODE(DD, PW) \
    hipLaunchKernelGGL((decode_kernel<DD, 2, PW, false>), grid, dim3(kDecThreads), 0, stream, a, none)
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
    if (p.head_dim == 128)
        hipLaunchKernelGGL(decode_combine_kernel<128>, cgrid, dim3(kCombThreads), 0, stream, a);
    else
        hipLaunchKernelGGL(decode_combine_kernel<64>, cgrid, dim3(kCombThreads), 0, stream, a);
    return hipGetLastError();
}

}  // namespace ls
