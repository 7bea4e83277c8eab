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
// Each wavefront owns kRT 16-row MFMA tiles.
//
// Keys stream in 32-key units (two 16-token blocks):
//   S^T[16 keys x 16 rows] = K[16 x D] . Q^T          (MFMA 16x16x32 bf16)
//   O^T[16 dims x 16 rows] += V^T[16 x 32 keys] . P^T  (MFMA 16x16x32 bf16)
// The 16 A-rows of each S^T MFMA are chosen so that lane group g4 (lanes
// 16*g4 .. 16*g4+15) ends up holding the scores of keys 8*g4 .. 8*g4+7 of the
// unit: those 8 keys are the 8 k-slots the same lane supplies as the B operand
// of PV, and they are 8 consecutive tokens of one block, i.e. one 16-byte
// chunk of the block's dim-major V tile.  So P stays in registers (rounded to
// bf16; the row sums add up the same rounded values) and every MFMA operand is
// one 16-byte LDS read.  Scores are exact fp32 sums of bf16 products; the
// softmax scale is applied in fp32 (folding it into q before the MFMA would
// round q * scale to bf16, an error that grows with the score magnitude).
// Softmax statistics stay in fp32.  A row's running max m' is set from its
// first 32 keys and raised only when a unit's probabilities, summed per lane,
// exceed 2^16 (those sums are needed for the row sums anyway, so the common
// path computes no maxima): then O and l are rescaled and the unit's
// probabilities recomputed before its P V, so every probability that reaches
// O is below 2^16.
//
// Pipeline: K runs one unit ahead of P, and P one phase ahead of its P V.
// Each 32-key unit takes two phases: A computes the scores of unit u+1 while
// turning the exp2 arguments of unit u into P; B accumulates P V of unit u-1
// while it scales the scores of unit u+1 into exp2 arguments
// (S * scale * log2(e) - m'); after B the sums of unit u's P are tested, a
// whole phase after they were computed, before unit u's P V in the next B.
// Each MFMA is followed by its share of the phase's VALU work, and the
// operands of the next phase are read from LDS during the current one, so the
// softmax arithmetic issues while the matrix core is busy and LDS latency
// stays hidden.  Data moves from HBM straight into LDS (buffer loads with the
// LDS-destination form: no register staging, no LDS write instructions) two
// 64-key stages ahead, into four stage buffers (a stage's V is read until the
// tile after it), one barrier per 64 keys.
//
// Scheduling: all query tiles of one (session, KV head) pair run on one XCD,
// so they stream the same keys through its L2; pairs are dealt to XCDs
// longest first, by the kernel or, given the lengths on the host, by the host
// (see the schedule in prefill_kernel).  With a counter workspace, XCDs that
// run faster take over the slower ones' last tiles.
#include <algorithm>
#include <type_traits>

#include "common.h"

namespace ls {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;

constexpr int kPreRows = 256;            // query rows per workgroup
constexpr int kRT = 2;                   // 16-row MFMA tiles per wavefront
constexpr int kWaveRows = 16 * kRT;
constexpr int kPreWaves = kPreRows / kWaveRows;
constexpr int kPreThreads = kPreWaves * kWave;
constexpr int kKeyTile = 64;             // keys per pipeline stage (4 blocks)
constexpr int kBufferDword3P = 0x00020000;   // raw buffer, 32-bit data format
constexpr float kLog2eP = 1.4426950408889634f;
constexpr float kSumLimit = 65536.0f;    // per-lane sum of a unit's P above which m' is raised
constexpr int kXcds = 8;                 // workgroups are dispatched round-robin over XCDs
constexpr int kMaxPairs = 512;           // (session, KV head) pairs scheduled; more run in index order
constexpr int kPlanPairs = 256;          // pairs (and sessions) a host-dealt schedule holds

struct PrefillArgs {
    const uint16_t *pool;          // layer base
    int64_t num_blocks;
    int32_t num_kv_heads;
    int32_t group;
    int32_t num_sessions;
    int32_t qtiles;                // query tiles of the longest turn
    int32_t total;                 // new tokens of the call (rows of q and out)
    const uint16_t *q;             // [T][Hq][D]
    uint16_t *out;                 // [T][Hq][D]
    const int32_t *cu;             // [S+1]
    const int32_t *ctx;            // [S]
    const int32_t *block_tables;
    int32_t max_blocks;
    float scale_log2;
    unsigned int *err;
    uint32_t *queue;               // per-XCD item counters (resident workgroups), or null
};

// Schedule dealt on the host when the caller passes the lengths there: every
// XCD's (session, KV head) pairs in the order that XCD runs them, with the
// items (query tiles) of the XCD's entries before each one.
struct PrefillHostPlan {
    uint16_t start[kXcds + 1];           // XCD x runs entries [start[x], start[x + 1])
    uint16_t pair[kPlanPairs];           // s * num_kv_heads + g
    uint16_t session_items[kPlanPairs];  // query tiles planned for session s
    uint32_t before[kPlanPairs];         // items of the XCD's entries before this one
    uint32_t total[kXcds];               // items of XCD x
};
struct PrefillNoPlan {
    int32_t unused;
};
template <bool kHost>
using PrefillPlanArg = typename std::conditional<kHost, PrefillHostPlan, PrefillNoPlan>::type;

// NaN-propagating maxima (v_maximum3_f32 on gfx950: no operand canonicalisation).
__device__ __forceinline__ float fmax3(float a, float b, float c) {
    return __builtin_elementwise_maximum(__builtin_elementwise_maximum(a, b), c);
}

// Max / sum over the four lanes l, l^16, l^32, l^48 (the lanes holding one
// row's scores) with the gfx950 row-swap permutes: VALU only.
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

// Entry jb of a session's block table, or -1 outside [0, nv).  The table does
// not change during a launch, so it is read through the constant address
// space: a scalar load, whose wait does not also wait for vector loads in
// flight.  The clamped index keeps the read inside the table row.
__device__ __forceinline__ int32_t table_entry(const int32_t *table, int jb, int nv) {
    typedef const __attribute__((address_space(4))) int32_t const_i32;
    const int jc = max(min(jb, nv - 1), 0);
    const int32_t b = ((const_i32 *)table)[jc];
    // select by mask rather than by branch: the load stays unconditional
    const int32_t keep = -(int32_t)((unsigned)jb < (unsigned)nv);
    return b | ~keep;
}

// Geometry of one pipeline stage ("load set" t = K of blocks 4t+2 .. 4t+5,
// i.e. units 2t+1 and 2t+2, and V of blocks 4t .. 4t+3, i.e. key tile t).
// Each wave moves whole kilobytes: 64 lanes x 16 bytes per load.
template <int D>
struct Geo {
    static constexpr int kBlockBytes = kBlock * D * 2;           // one block's K (or V) of one head
    static constexpr int kRowChunks = D / 8;                      // 16-byte chunks per K token row
    static constexpr int kUnitBytes = 2 * kBlockBytes;            // K of one 32-key unit
    static constexpr int kStageBytes = 4 * kBlockBytes;           // K (or V) of one stage
    static constexpr int kKbPerBlock = kBlockBytes / 1024;        // 4 (D=128) or 2 (D=64)
    static constexpr int kLoadsK = 4 * kKbPerBlock / kPreWaves;   // per wave per stage: 2 or 1
    static constexpr int kLoads = 2 * kLoadsK;                    // K and V loads per wave per stage
    static_assert(kLoadsK >= 1 && (4 * kKbPerBlock) % kPreWaves == 0, "stage must split evenly");
};

// K LDS layout of one block: [token 16][D/8 chunks], chunk ch of token t in
// slot ch ^ kswz(block-in-unit, t).  The swizzle makes the 16 rows one S^T
// MFMA reads (tokens {0..3, 8..11} + 4*sb of both blocks) hit distinct banks.
template <int D>
__device__ __forceinline__ int kswz(int b, int t) {
    return ((t & 3) | (((t >> 3) & 1) << 2) | (b << 3)) & (Geo<D>::kRowChunks - 1);
}

// V LDS layout of one block: 16-byte chunks (dim, half) = tokens 8*half ..
// 8*half+7 of one dim, chunk at position half*D + dim: the 16 lanes that read
// one (half, 16 dims) read 256 contiguous bytes.

// One wave's load of one kilobyte of a block into LDS (lane l writes bytes
// 16*l .. 16*l+15 of dst).  head_base is this KV head's K (or V) tile in
// block 0 of the layer; a block's tile is slab_elems further per block id,
// one 32 x 32 -> 64-bit multiply.  Absent blocks (id -1 or outside the pool)
// are read through a zero-size buffer descriptor: no memory traffic.
template <int D>
__device__ __forceinline__ void load_kb(const uint16_t *head_base, uint32_t slab_elems, uint32_t nblocks,
                                             int32_t b, uint8_t *dst, int voff) {
    const bool valid = (uint32_t)b < nblocks;
    const uint16_t *base = head_base + (uint64_t)(valid ? (uint32_t)b : 0u) * slab_elems;
    const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t *>(base), 0, valid ? Geo<D>::kBlockBytes : 0, kBufferDword3P);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (lds_void *)dst, 16, voff, 0, 0, 0);
}

// Barrier between pipeline stages.  Each wave first waits until its loads of
// the next stage have landed (only the kLoads loads of the stage after it may
// still be in flight) and its LDS reads have returned; the barrier then
// publishes the next stage to all waves and frees the stage just read.  No
// memory fence: a fence would also wait for the loads two stages ahead.
template <int D>
__device__ __forceinline__ void stage_barrier() {
    // s_waitcnt vmcnt(kLoads) expcnt(7) lgkmcnt(0)
    __builtin_amdgcn_s_waitcnt(0x0070 | Geo<D>::kLoads);
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// Scheduling constraint for one phase of N MFMAs: MFMA i is followed by one
// LDS read (even i, while reads remain), its share of the phase's plain VALU
// instructions, then its share of the transcendental ones.  With the plain
// ones first, the conversion of a pair of exp results issues after the next
// MFMA instead of right behind the second exp, where it would need a wait
// state (1.3% faster on the next-turn workload).
template <int I, int N, int Reads, int Trans, int Valu>
__device__ __forceinline__ void order_phase() {
    if constexpr (I < N) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        if constexpr (I % 2 == 0 && I / 2 < Reads) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        constexpr int t = (I + 1) * Trans / N - I * Trans / N;
        constexpr int v = (I + 1) * Valu / N - I * Valu / N;
        if constexpr (v > 0) __builtin_amdgcn_sched_group_barrier(0x002, v, 0);
        if constexpr (t > 0) __builtin_amdgcn_sched_group_barrier(0x400, t, 0);
        order_phase<I + 1, N, Reads, Trans, Valu>();
    }
}

template <int D, bool kHost>
__global__ __launch_bounds__(kPreThreads) void prefill_kernel(PrefillArgs a, PrefillPlanArg<kHost> plan) {
    using C = Geo<D>;
    constexpr int KS = D / 32;           // 32-dim k-steps of QK
    constexpr int NDT = D / 16;          // 16-dim output tiles
    // Four stage buffers (stage t in buffer t % 4); separate arrays let the
    // compiler track each one's loads.
    __shared__ __attribute__((aligned(1024))) uint8_t k0[C::kStageBytes];
    __shared__ __attribute__((aligned(1024))) uint8_t k1[C::kStageBytes];
    __shared__ __attribute__((aligned(1024))) uint8_t k2[C::kStageBytes];
    __shared__ __attribute__((aligned(1024))) uint8_t k3[C::kStageBytes];
    __shared__ __attribute__((aligned(1024))) uint8_t v0[C::kStageBytes];
    __shared__ __attribute__((aligned(1024))) uint8_t v1[C::kStageBytes];
    __shared__ __attribute__((aligned(1024))) uint8_t v2[C::kStageBytes];
    __shared__ __attribute__((aligned(1024))) uint8_t v3[C::kStageBytes];
    __shared__ __attribute__((aligned(16))) int64_t sm_work[kMaxPairs];
    __shared__ int sm_items[kMaxPairs];
    __shared__ int sm_order[kMaxPairs];
    __shared__ float sm_rank_work[kMaxPairs];
    __shared__ int sm_grab[2];

    const int tid = threadIdx.x;
    const int S = a.num_sessions;
    const int G = a.group;
    const int qtok = kPreRows / G;       // new tokens per query tile
    const int QT = a.qtiles;
    const int Hkv = a.num_kv_heads;

    // ---- one item: rows of query tile qt of session s, KV head g.
    auto run_item = [&](const int s, const int g, const int qt) {
        const int n = a.cu[s + 1] - a.cu[s];
        const int j0 = qt * qtok;
        if (j0 >= n || a.cu[s] < 0 || a.cu[s + 1] > a.total) return;   // (lengths outside q: flagged above)
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
        const int nb = min(nblk_valid, ntiles * 4);           // blocks any row here can see

        const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
        const int lane = tid % kWave;
        const int c16 = lane & 15;
        const int g4 = lane >> 4;
        const int hq_total = Hkv * G;

        // Rows of this lane (one per 16-row tile): r = wave*32 + rt*16 + c16.
        int row_lim[kRT];
        int64_t row_out[kRT];
        bool row_ok[kRT];
        bf16x8 qop[kRT][KS];
    #pragma unroll
        for (int rt = 0; rt < kRT; ++rt) {
            const int r = wave * kWaveRows + rt * 16 + c16;
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
        // Wait for q here, before the first stage loads are issued, so that no
        // wait for q remains inside the key loop (vmcnt(0), other counters untouched).
        __builtin_amdgcn_s_waitcnt(0x0F70);
        // smallest causal limit among this wave's rows: units past it need masking
        const int wave_lim_min = c + min(j0 + (wave * kWaveRows) / G, n - 1);

        // ---- this wave's share of every stage: kLoadsK kilobytes of one K block
        // and of one V block (block 'blk' of the stage), at fixed lane offsets.
        const int blk = (wave * C::kLoadsK) / C::kKbPerBlock;
        int k_voff[C::kLoadsK], v_voff[C::kLoadsK], kb_off[C::kLoadsK];
    #pragma unroll
        for (int e = 0; e < C::kLoadsK; ++e) {
            const int q = (wave * C::kLoadsK + e) % C::kKbPerBlock;       // kilobyte within the block
            kb_off[e] = blk * C::kBlockBytes + q * 1024;
            // K: lane -> (token, slot); fetch the chunk that belongs in that slot
            const int t = q * (1024 / (D * 2)) + lane / C::kRowChunks;
            const int sl = lane % C::kRowChunks;
            k_voff[e] = ((sl ^ kswz<D>(blk & 1, t)) * kBlock + t) * 16;   // chunk-major K tile
            // V: lane -> chunk position p = half*D + dim
            const int p = q * 64 + lane;
            v_voff[e] = (p % D) * 32 + (p / D) * 16;
        }
        const int32_t *table = a.block_tables + (int64_t)s * a.max_blocks;
        const uint32_t slab_elems = (uint32_t)(2 * Hkv * kBlock * D);
        const uint32_t nblocks32 = (uint32_t)min(a.num_blocks, (int64_t)0x7fffffff);
        const uint16_t *kbase = a.pool + (int64_t)g * (kBlock * D);
        const uint16_t *vbase = kbase + (int64_t)Hkv * (kBlock * D);
        auto load_k = [&](uint8_t *stage, int32_t b) {
    #pragma unroll
            for (int e = 0; e < C::kLoadsK; ++e) load_kb<D>(kbase, slab_elems, nblocks32, b, stage + kb_off[e], k_voff[e]);
        };
        auto load_v = [&](uint8_t *stage, int32_t b) {
    #pragma unroll
            for (int e = 0; e < C::kLoadsK; ++e) load_kb<D>(vbase, slab_elems, nblocks32, b, stage + kb_off[e], v_voff[e]);
        };
        auto id_k = [&](int t) { return table_entry(table, 4 * t + 2 + blk, nb); };
        auto id_v = [&](int t) { return table_entry(table, 4 * t + blk, nb); };

        float nm[kRT], lsum[kRT];             // -m' (running row max * scale * log2 e),
        f32x4 o[kRT][NDT];                    // partial row sums, unnormalised output
    #pragma unroll
        for (int rt = 0; rt < kRT; ++rt) {
            nm[rt] = 0.f;
            lsum[rt] = 0.f;
        }
    #pragma unroll
        for (int rt = 0; rt < kRT; ++rt)
    #pragma unroll
            for (int dt = 0; dt < NDT; ++dt) o[rt][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
        const float sl2 = a.scale_log2;
        const bf16x2 ones2 = {(__bf16)1.0f, (__bf16)1.0f};

        // ---- S^T = K Q^T of one 32-key unit for 2 key sub-tiles x 2 row tiles.
        // A-row r of sub-tile sb is token 8*((r>>2)&1) + 4*sb + (r&3) of block
        // r>>3, i.e. unit key 8*(r>>2) + 4*sb + (r&3).  Per-lane byte offsets of
        // the K rows read for sub-tile sb and k-step ks, relative to the unit.
        // They are made opaque to the compiler so that no constant part is split
        // off the address: the split loses the LDS alias information that lets
        // these reads overlap the loads still in flight.
        int kroff[2][KS];
    #pragma unroll
        for (int sb = 0; sb < 2; ++sb) {
            const int b = c16 >> 3;
            const int t = 8 * ((c16 >> 2) & 1) + 4 * sb + (c16 & 3);
            const int sw = kswz<D>(b, t);
    #pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                kroff[sb][ks] = b * C::kBlockBytes + t * (D * 2) + ((ks * 4 + g4) ^ sw) * 16;
                asm volatile("" : "+v"(kroff[sb][ks]));
            }
        }
        // Operands are read from LDS one phase before the MFMAs that use them:
        // kop (K of the next unit) while the current P V runs, vop (V of the
        // current unit) while the next scores are computed.
        bf16x8 kop[2][KS];
        bf16x8 vop[NDT];
        auto read_k = [&](const uint8_t *lk) {
    #pragma unroll
            for (int sb = 0; sb < 2; ++sb)
    #pragma unroll
                for (int ks = 0; ks < KS; ++ks)
                    kop[sb][ks] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(lk + kroff[sb][ks]));
        };
        auto qk_mfma = [&](f32x4 (&acc)[kRT][2]) {
    #pragma unroll
            for (int sb = 0; sb < 2; ++sb) {
    #pragma unroll
                for (int rt = 0; rt < kRT; ++rt) acc[rt][sb] = f32x4{0.f, 0.f, 0.f, 0.f};
    #pragma unroll
                for (int ks = 0; ks < KS; ++ks)
    #pragma unroll
                    for (int rt = 0; rt < kRT; ++rt)
                        acc[rt][sb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kop[sb][ks], qop[rt][ks], acc[rt][sb], 0, 0, 0);
            }
        };
        // Causal mask of a unit whose first key is key0 (lane group g4 holds unit
        // keys 8*g4 + 4*sb + i); only units that reach past the smallest causal
        // limit of the wave's rows need it.
        auto mask_unit = [&](f32x4 (&acc)[kRT][2], int key0) {
            if (key0 + 31 <= wave_lim_min) return;
    #pragma unroll
            for (int rt = 0; rt < kRT; ++rt) {
                const int lim = row_lim[rt] - key0 - 8 * g4;
    #pragma unroll
                for (int sb = 0; sb < 2; ++sb)
    #pragma unroll
                    for (int i = 0; i < 4; ++i)
                        if (4 * sb + i > lim) acc[rt][sb][i] = -INFINITY;
            }
        };
        // Largest of a lane's 8 values of one row tile (NaN-propagating).
        auto lane_max = [&](const f32x4 (&acc)[2]) {
            const f32x4 x0 = acc[0], x1 = acc[1];
            return fmax3(fmax3(x0[0], x0[1], x0[2]), fmax3(x0[3], x1[0], x1[1]), fmax3(x1[2], x1[3], x1[3]));
        };
        // Scores -> exp2 arguments S * scale * log2(e) - m' (phase B).
        auto scale_unit = [&](f32x4 (&acc)[kRT][2]) {
    #pragma unroll
            for (int rt = 0; rt < kRT; ++rt)
    #pragma unroll
                for (int sb = 0; sb < 2; ++sb)
    #pragma unroll
                    for (int i = 0; i < 4; ++i) acc[rt][sb][i] = __builtin_fmaf(acc[rt][sb][i], sl2, nm[rt]);
        };
        // P = exp2(S * scale * log2 e - m') in bf16 (B operand of PV), and the
        // lane's sum of the rounded values per row tile.
        auto exp_unit = [&](const f32x4 (&acc)[kRT][2], bf16x8 (&pop)[kRT], float (&us)[kRT]) {
    #pragma unroll
            for (int rt = 0; rt < kRT; ++rt) {
                uint32_t w[4];
                us[rt] = 0.f;
    #pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const f32x4 &x = acc[rt][j >> 1];
                    const int i0 = 2 * (j & 1);
                    const bf16x2 pk = {(__bf16)__builtin_amdgcn_exp2f(x[i0]), (__bf16)__builtin_amdgcn_exp2f(x[i0 + 1])};
                    us[rt] = __builtin_amdgcn_fdot2_f32_bf16(pk, ones2, us[rt], false);
                    w[j] = __builtin_bit_cast(uint32_t, pk);
                }
                pop[rt] = __builtin_bit_cast(bf16x8, u32x4{w[0], w[1], w[2], w[3]});
            }
        };
        // After the B phase that follows a unit's P (and before its P V): when
        // some lane's sum exceeds the limit (a probability above 2^13, an infinite
        // one included), the rows' maxima are raised to the unit's row maxima.  O
        // and l (which hold the units before it) are rescaled, the exp2 arguments
        // of the unit and of the next unit (already scaled) shifted, and the unit's
        // P recomputed (at most 1 now).  Rows whose max did not move shift by 0.
        // Then the unit's sums join l.
        auto settle = [&](f32x4 (&acc)[kRT][2], f32x4 (&next)[kRT][2], bf16x8 (&pop)[kRT], float (&us)[kRT]) {
            bool over = false;
    #pragma unroll
            for (int rt = 0; rt < kRT; ++rt) over = over || us[rt] > kSumLimit;
            if (__any(over)) {
    #pragma unroll
                for (int rt = 0; rt < kRT; ++rt) {
                    const float shift = __builtin_elementwise_maximum(xmax16_32(lane_max(acc[rt])), 0.f);
                    const float alpha = __builtin_amdgcn_exp2f(-shift);
                    lsum[rt] *= alpha;
    #pragma unroll
                    for (int dt = 0; dt < NDT; ++dt) o[rt][dt] *= alpha;
                    nm[rt] -= shift;
                    acc[rt][0] -= shift;
                    acc[rt][1] -= shift;
                    next[rt][0] -= shift;
                    next[rt][1] -= shift;
                }
                exp_unit(acc, pop, us);
            }
    #pragma unroll
            for (int rt = 0; rt < kRT; ++rt) lsum[rt] += us[rt];
        };
        // Per-lane byte offset of the V chunk this lane reads, opaque for the same
        // reason as kroff.  Dims dt*16 + c16 of one lane are 256 bytes apart.
        int vroff = (g4 >> 1) * C::kBlockBytes + ((g4 & 1) * D + c16) * 16;
        asm volatile("" : "+v"(vroff));
        auto read_v = [&](const uint8_t *lv, int h) {
            const uint8_t *blkv = lv + 2 * h * C::kBlockBytes + vroff;
    #pragma unroll
            for (int dt = 0; dt < NDT; ++dt)
                vop[dt] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(blkv + dt * 256));
        };
        // O^T += V^T P^T for one unit.
        auto pv_mfma = [&](const bf16x8 (&pop)[kRT]) {
    #pragma unroll
            for (int dt = 0; dt < NDT; ++dt)
    #pragma unroll
                for (int rt = 0; rt < kRT; ++rt)
                    o[rt][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vop[dt], pop[rt], o[rt][dt], 0, 0, 0);
        };
        // Instruction order inside a phase: each MFMA is followed by a share of
        // the phase's VALU work and, every other MFMA, by one operand read for the
        // next phase, so that the softmax arithmetic issues while the matrix core
        // is busy and every LDS read has a whole phase to return.
        constexpr int kPhaseMfma = 2 * KS * kRT;              // == NDT * kRT
        constexpr int kExpTrans = kRT * 4 * 2;                // exp phase: 2 exp ...
        constexpr int kExpValu = kRT * 4 * 2;                 // ... and cvt, dot2 per pair
        constexpr int kScaleValu = kRT * 8;                   // scale phase: the FMAs
        // Keeps the probabilities of a phase from being computed later (after the
        // masking branch that follows the phase).
        auto pin = [&](const bf16x8 (&pop)[kRT]) {
    #pragma unroll
            for (int rt = 0; rt < kRT; ++rt) asm volatile("" ::"v"(pop[rt]));
        };
        // Values of keys at or past kv_len (the rest of the session's last block,
        // or blocks never loaded) are zeroed in the staged V tile of key tile j
        // before it is used, so that 0 * NaN cannot reach O.  Only the last key
        // tile can hold such keys; one extra LDS barrier, once per workgroup.
        auto zero_v_tail = [&](uint8_t *lv, int j) {
            constexpr int kChunks = 4 * 2 * D;                    // (block, half, dim) chunks of 8 tokens
            for (int ci = tid; ci < kChunks; ci += kPreThreads) {
                const int bi = ci / (2 * D), hf = (ci / D) & 1;
                const int t0 = j * kKeyTile + bi * kBlock + hf * 8;
                if (t0 + 8 <= kv_len) continue;
                u32x4 *chunk = reinterpret_cast<u32x4 *>(lv + ci * 16);
                u32x4 x = *chunk;
    #pragma unroll
                for (int w = 0; w < 4; ++w) {
                    const int t = t0 + 2 * w;
                    x[w] &= t + 1 < kv_len ? 0xFFFFFFFFu : (t < kv_len ? 0x0000FFFFu : 0u);
                }
                *chunk = x;
            }
            __builtin_amdgcn_s_waitcnt(0xC07F);                   // lgkmcnt(0) only
            asm volatile("" ::: "memory");
            __builtin_amdgcn_s_barrier();
            asm volatile("" ::: "memory");
        };

        // ---- pipeline over 32-key units.  Key tile j (units 2j, 2j+1) reads
        // stage j: K of units 2j+1, 2j+2 and V of units 2j, 2j+1; it also reads V
        // of unit 2j-1 from stage j-1.  While it is processed, the loads of stage
        // j+2 go into buffer (j+2) % 4, last read in tile j-1.  A tile runs four
        // phases, each followed by the test of the P made one phase before:
        //   A0: scores of unit 2j+1 | P of unit 2j          | read V of unit 2j-1
        //   B0: P V of unit 2j-1    | scale of unit 2j+1    | read K of unit 2j+2
        //       (test P of unit 2j)
        //   A1: scores of unit 2j+2 | P of unit 2j+1        | read V of unit 2j
        //   -- barrier: stage j+1 has landed; stage j-1 is fully read --
        //   B1: P V of unit 2j      | scale of unit 2j+2    | read K of unit 2j+3
        //       (test P of unit 2j+1)
        // The last tile then reads V of its second unit and adds its P V.  A wave
        // in a B phase runs at raised issue priority: of the two waves sharing a
        // SIMD, the one feeding P V (light VALU) then issues its MFMAs first while
        // the other's exp work fills the VALU slots.
        f32x4 sa[kRT][2], sb2[kRT][2];
        bf16x8 pop_e[kRT], pop_o[kRT];        // P of the even and odd unit in flight
        float us_e[kRT], us_o[kRT];
    #pragma unroll
        for (int rt = 0; rt < kRT; ++rt) pop_o[rt] = __builtin_bit_cast(bf16x8, u32x4{0u, 0u, 0u, 0u});
        int32_t idk = id_k(-1), idv = id_v(-1);
        load_k(k3, idk);                      // stage -1: K unit 0 (its V part is empty)
        load_v(v3, idv);
        idk = id_k(0); idv = id_v(0);
        load_k(k0, idk);
        load_v(v0, idv);
        idk = id_k(1); idv = id_v(1);
        load_k(k1, idk);
        load_v(v1, idv);
        idk = id_k(2); idv = id_v(2);
        stage_barrier<D>();                   // stages -1 and 0 have landed
        // V of unit -1 (second half of stage -1's V): zeros, so that the first
        // tile's P V of that unit (with P = 0) adds nothing.
        for (int ci = tid; ci < 2 * C::kBlockBytes / 16; ci += kPreThreads)
            *reinterpret_cast<u32x4 *>(v3 + 2 * C::kBlockBytes + ci * 16) = u32x4{0u, 0u, 0u, 0u};
        read_k(k3 + C::kUnitBytes);           // unit 0 = second unit of stage -1
        qk_mfma(sa);
        read_k(k0);                           // unit 1
        mask_unit(sa, 0);
        // The first unit's row maxima start the running maxima (every row sees key 0).
    #pragma unroll
        for (int rt = 0; rt < kRT; ++rt) nm[rt] = -xmax16_32(lane_max(sa[rt])) * sl2;
        scale_unit(sa);
        __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0): the zeros are written
        asm volatile("" ::: "memory");
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");

        // The loads are issued on every path, so outstanding loads are counted
        // exactly; only the compute of tiles past the last one is skipped.
        auto tile = [&](int j, const uint8_t *ks, uint8_t *vs, const uint8_t *vprev, const uint8_t *knext,
                        uint8_t *kn, uint8_t *vn) {
            const int32_t ik = idk, iv = idv;
            idk = id_k(j + 3);
            idv = id_v(j + 3);
            const bool live = j < ntiles;
            if (live && (j + 1) * kKeyTile > kv_len) zero_v_tail(vs, j);
            load_k(kn, ik);
            load_v(vn, iv);
            if (live) {
                qk_mfma(sb2);                           // A0
                exp_unit(sa, pop_e, us_e);
                read_v(vprev, 1);
                order_phase<0, kPhaseMfma, NDT, kExpTrans, kExpValu>();
                pin(pop_e);
                mask_unit(sb2, j * kKeyTile + 32);
                __builtin_amdgcn_s_setprio(1);          // B phases issue first
                pv_mfma(pop_o);                         // B0
                scale_unit(sb2);
                read_k(ks + C::kUnitBytes);
                order_phase<0, kPhaseMfma, 2 * KS, 0, kScaleValu>();
                __builtin_amdgcn_s_setprio(0);
                settle(sa, sb2, pop_e, us_e);
                qk_mfma(sa);                            // A1
                exp_unit(sb2, pop_o, us_o);
                read_v(vs, 0);
                order_phase<0, kPhaseMfma, NDT, kExpTrans, kExpValu>();
                pin(pop_o);
                mask_unit(sa, (j + 1) * kKeyTile);
            }
            stage_barrier<D>();
            if (live) {
                __builtin_amdgcn_s_setprio(1);
                pv_mfma(pop_e);                         // B1
                scale_unit(sa);
                read_k(knext);                          // (unused when tile j+1 is past the end)
                order_phase<0, kPhaseMfma, 2 * KS, 0, kScaleValu>();
                __builtin_amdgcn_s_setprio(0);
                settle(sb2, sa, pop_o, us_o);
                if (j == ntiles - 1) {                  // the last unit's P V
                    read_v(vs, 1);
                    pv_mfma(pop_o);
                }
            }
        };
        for (int j = 0; j < ntiles; j += 4) {
            tile(j, k0, v0, v3, k1, k2, v2);
            tile(j + 1, k1, v1, v0, k2, k3, v3);
            tile(j + 2, k2, v2, v1, k3, k0, v0);
            tile(j + 3, k3, v3, v2, k0, k1, v1);
        }

        // ---- normalise and write
    #pragma unroll
        for (int rt = 0; rt < kRT; ++rt) {
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
    };

    // ---- schedule.  Items are (session s, KV head g, query tile qt).  All query
    // tiles of one (s, g) pair run on one XCD, so they stream the same keys
    // through its L2 at about the same time.  Pairs are dealt to the 8 XCDs in
    // rounds of 8 in order of decreasing work: in each round the heaviest pair
    // goes to the XCD with the least work so far, the next to the next-least,
    // and so on (a longest-processing-time-first rule; the 4 or 8 KV heads of
    // one session have equal work, and a fixed snake would send them to the
    // same half of the XCDs every round).  An XCD runs its pairs in the order
    // dealt, each pair's latest (longest) query tile first.  Workgroup i is
    // dispatched to XCD i % 8 and is the (i / 8)-th item there; every
    // workgroup derives the same schedule from the lengths.  A schedule dealt
    // on the host (same rule, each XCD's pairs then run longest item first)
    // replaces all of this with one lookup.
    const int P = S * Hkv;
    // A turn longer than its planned query tiles (max_new_len understated, or
    // device lengths longer than the host's), a negative turn or a negative
    // context cannot be attended as given: flagged once, by the first
    // workgroup (rows past the planned tiles are not written).
    if (blockIdx.x == 0)
        for (int sp = tid; sp < S; sp += kPreThreads) {
            const int nt = a.cu[sp + 1] - a.cu[sp];
            int planned = QT;
            if constexpr (kHost) planned = plan.session_items[sp];
            if (nt < 0 || nt > planned * qtok || a.ctx[sp] < 0 || a.cu[sp] < 0 || a.cu[sp + 1] > a.total)
                flag_error(a.err, LS_DEVERR_LENGTH);
        }
    int s, g, qt;
    if constexpr (kHost) {
        // Item `slot` of XCD x's list: the entry of the last pair whose earlier
        // items are at most the slot (entries have items, so 'before' increases;
        // an XCD has at most kPlanPairs / 8 entries, one per lane).
        auto lookup = [&](int x, uint32_t slot) {
            const int b = plan.start[x], m = plan.start[x + 1] - b;
            const int ln = tid % kWave;
            const bool passed = ln < m && plan.before[b + min(ln, m - 1)] <= slot;
            const int e = b + __popcll(__ballot(passed)) - 1;
            const uint32_t items = (e + 1 < b + m ? plan.before[e + 1] : plan.total[x]) - plan.before[e];
            qt = (int)(items - 1 - (slot - plan.before[e]));
            s = plan.pair[e] / Hkv;
            g = plan.pair[e] % Hkv;
        };
        // Without counters, workgroup i takes item i / 8 of XCD i % 8.  With
        // them (a.queue), workgroup i takes the next item of XCD i % 8's list
        // through a counter per XCD, and once that list is exhausted, the next
        // item of the XCD with the most items left (the grid has ~10% more
        // workgroups than items; the ones that find every list exhausted end).
        // XCDs run at different speeds (several percent apart), so with a fixed
        // deal the fast ones idle at the end.  Each list is tried at most once
        // after it ran out, so the search ends.
        const int home = (int)(blockIdx.x % kXcds);
        if (a.queue) {
            if (tid == 0) {
                int gx = -1;
                uint32_t gs = atomicAdd(&a.queue[home], 1u);
                if (gs < plan.total[home]) {
                    gx = home;
                } else {
                    uint32_t tried = 1u << home;
                    while (gx < 0) {
                        int best = -1;
                        int64_t most = 0;
                        for (int y = 0; y < kXcds; ++y) {
                            if ((tried >> y) & 1u) continue;
                            const int64_t left =
                                (int64_t)plan.total[y] -
                                (int64_t)__hip_atomic_load(&a.queue[y], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                            if (left > most) {
                                most = left;
                                best = y;
                            }
                        }
                        if (best < 0) break;                       // every list is exhausted
                        gs = atomicAdd(&a.queue[best], 1u);
                        if (gs < plan.total[best]) gx = best;
                        else tried |= 1u << best;
                    }
                }
                sm_grab[0] = gx;
                sm_grab[1] = (int)gs;
            }
            __syncthreads();
            if (sm_grab[0] < 0) return;
            lookup(sm_grab[0], (uint32_t)sm_grab[1]);
        } else {
            const uint32_t slot = blockIdx.x / kXcds;
            if (slot >= plan.total[home]) return;
            lookup(home, slot);
        }
    } else if (P <= kMaxPairs) {
        for (int p = tid; p < P; p += kPreThreads) {
            const int sp = p / Hkv;
            const int nt = max(a.cu[sp + 1] - a.cu[sp], 0);
            const int items = min((nt + qtok - 1) / qtok, QT);
            sm_items[p] = items;
            sm_work[p] = (int64_t)items * (2 * (int64_t)max(a.ctx[sp], 0) + nt);
        }
        if (tid == 0 && (P & 1)) sm_work[P] = -1;              // pad to 2 (never counts)
        __syncthreads();
        for (int p = tid; p < P; p += kPreThreads) {
            // Two works per LDS read and four reads in flight.
            const int64_t w = sm_work[p];
            int r = 0;
#pragma unroll 4
            for (int q = 0; q < P; q += 2) {
                const longlong2 w2 = *reinterpret_cast<const longlong2 *>(&sm_work[q]);
                r += (w2.x > w) || (w2.x == w && q < p);
                r += (w2.y > w) || (w2.y == w && q + 1 < p);
            }
            sm_order[r] = p;
            sm_rank_work[r] = (float)w;
        }
        __syncthreads();
        const int xcd = (int)(blockIdx.x % kXcds);
        int slot = (int)(blockIdx.x / kXcds);
        int pick = -1;
        // Every wave deals the rounds itself.  Lane 8 xi + xj compares the work
        // of XCD xj with that of XCD xi; the ballot's byte xi then counts the
        // XCDs ahead of XCD xi (less work, or equal work and a lower index),
        // which is XCD xi's place in the round.  Work sums are floats: only
        // their order matters, and every wave adds the same values in the same
        // order.
        const int xi = (tid % kWave) >> 3, xj = tid & 7;
        float done = 0.f;                                 // work dealt to XCD xj so far
        for (int k = 0; kXcds * k < P; ++k) {
            const float di = __shfl(done, xi);            // lane xi holds XCD xi
            const uint64_t ahead = __ballot(done < di || (done == di && xj < xi));
            const int r_j = kXcds * k + __popcll((ahead >> (8 * xj)) & 0xFF);
            if (r_j < P) done += sm_rank_work[r_j];
            const int r = kXcds * k + __popcll((ahead >> (8 * xcd)) & 0xFF);
            if (r >= P) break;
            const int cnt = sm_items[sm_order[r]];
            if (slot < cnt) {
                pick = sm_order[r];
                break;
            }
            slot -= cnt;
        }
        if (pick < 0) return;
        s = pick / Hkv;
        g = pick % Hkv;
        qt = sm_items[pick] - 1 - slot;
    } else {
        const int64_t lg = blockIdx.x;
        if (lg >= (int64_t)S * Hkv * QT) return;
        qt = QT - 1 - (int)(lg % QT);
        g = (int)((lg / QT) % Hkv);
        s = (int)(lg / ((int64_t)QT * Hkv));
    }

    run_item(s, g, qt);
}

}  // namespace

namespace {

// Host dealing of the schedule (the device rule, on exact integer work, with
// each XCD's pairs then ordered by decreasing item length c + n, so that the
// items an XCD ends with are short).  Returns false when the batch exceeds the
// plan's capacity (the device deals the schedule then).
bool plan_prefill_host(int32_t S, int32_t hkv, int32_t qtok, const int32_t *lens, PrefillHostPlan &plan,
                       int32_t &max_items) {
    const int P = S * hkv;
    if (S > kPlanPairs || P > kPlanPairs) return false;
    struct Pair {
        int64_t work, len;
        int32_t p, items, deal;
    };
    Pair pr[kPlanPairs];
    int np = 0;
    for (int s = 0; s < S; ++s) {
        const int32_t n = lens[2 * s], c = lens[2 * s + 1];
        const int32_t items = (int32_t)(((int64_t)n + qtok - 1) / qtok);
        if (items > 0xFFFF) return false;                  // beyond the plan's 16-bit counts
        plan.session_items[s] = (uint16_t)items;
        if (items == 0) continue;
        for (int g = 0; g < hkv; ++g)
            pr[np++] = Pair{(int64_t)items * (2 * (int64_t)c + n), (int64_t)c + n, s * hkv + g, items, 0};
    }
    for (int s = S; s < kPlanPairs; ++s) plan.session_items[s] = 0;
    std::stable_sort(pr, pr + np, [](const Pair &x, const Pair &y) { return x.work > y.work; });
    // Rounds of 8: the round's k-th heaviest pair to the XCD with the k-th least work so far.
    int64_t load[kXcds] = {};
    int xcd_of[kPlanPairs];
    for (int r0 = 0; r0 < np; r0 += kXcds) {
        int rank[kXcds];
        for (int x = 0; x < kXcds; ++x) rank[x] = x;
        std::stable_sort(rank, rank + kXcds, [&](int x, int y) { return load[x] < load[y]; });
        for (int k = 0; k < kXcds && r0 + k < np; ++k) {
            xcd_of[r0 + k] = rank[k];
            pr[r0 + k].deal = r0 + k;
            load[rank[k]] += pr[r0 + k].work;
        }
    }
    // Per XCD, entries by decreasing item length (ties in dealing order).
    int idx[kPlanPairs];
    for (int i = 0; i < np; ++i) idx[i] = i;
    std::stable_sort(idx, idx + np, [&](int i, int j) {
        if (xcd_of[i] != xcd_of[j]) return xcd_of[i] < xcd_of[j];
        return pr[i].len > pr[j].len;
    });
    max_items = 0;
    int e = 0;
    for (int x = 0; x < kXcds; ++x) {
        plan.start[x] = (uint16_t)e;
        uint32_t acc = 0;
        for (; e < np && xcd_of[idx[e]] == x; ++e) {
            plan.pair[e] = (uint16_t)pr[idx[e]].p;
            plan.before[e] = acc;
            acc += (uint32_t)pr[idx[e]].items;
        }
        plan.total[x] = acc;
        max_items = std::max(max_items, (int32_t)acc);
    }
    plan.start[kXcds] = (uint16_t)e;
    return (int64_t)max_items * kXcds <= 0x7FFFFFFF;
}

}  // namespace

__global__ void clear_counters_kernel(uint32_t *counters, int n) {
    if ((int)threadIdx.x < n) counters[threadIdx.x] = 0u;
}

hipError_t launch_clear_counters(uint32_t *counters, int n, hipStream_t stream) {
    hipLaunchKernelGGL(clear_counters_kernel, dim3(1), dim3(kWave), 0, stream, counters, n);
    return hipGetLastError();
}

hipError_t launch_prefill(const PoolGeom &p, int layer, int32_t num_sessions, int32_t num_q_heads,
                          const uint16_t *q, const int32_t *cu_new_lens,
                          const int32_t *reused_lens, const int32_t *lens_host, int32_t total_tokens,
                          int32_t max_new_len, const int32_t *block_tables, int32_t max_blocks,
                          float scale, uint16_t *out, uint32_t *queue, unsigned int *err, hipStream_t stream) {
    if (num_sessions <= 0 || max_new_len <= 0) return hipSuccess;
    PrefillArgs a;
    a.pool = p.layer_base(layer);
    a.num_blocks = p.num_blocks;
    a.num_kv_heads = p.num_kv_heads;
    a.group = num_q_heads / p.num_kv_heads;
    a.num_sessions = num_sessions;
    a.total = total_tokens;
    a.q = q;
    a.out = out;
    a.cu = cu_new_lens;
    a.ctx = reused_lens;
    a.block_tables = block_tables;
    a.max_blocks = max_blocks;
    a.scale_log2 = scale * kLog2eP;
    a.err = err;
    a.queue = nullptr;
    const int qtok = kPreRows / a.group;
    a.qtiles = (max_new_len + qtok - 1) / qtok;
    PrefillHostPlan plan;
    int32_t max_items = 0;
    if (lens_host && plan_prefill_host(num_sessions, p.num_kv_heads, qtok, lens_host, plan, max_items)) {
        if (max_items == 0) return hipSuccess;
        dim3 grid((unsigned)(kXcds * max_items));
        if (queue) {
            // Items are taken through the counters; ~10% more workgroups than
            // items let the faster XCDs take over the slower ones' last items.
            if (hipError_t e = launch_clear_counters(queue, kXcds, stream)) return e;
            a.queue = queue;
            int64_t items = 0;
            for (int x = 0; x < kXcds; ++x) items += plan.total[x];
            const int64_t per_xcd = (items + kXcds - 1) / kXcds + (items + 10 * kXcds - 1) / (10 * kXcds);
            grid = dim3((unsigned)(kXcds * per_xcd));
        }
        if (p.head_dim == 128)
            hipLaunchKernelGGL((prefill_kernel<128, true>), grid, dim3(kPreThreads), 0, stream, a, plan);
        else
            hipLaunchKernelGGL((prefill_kernel<64, true>), grid, dim3(kPreThreads), 0, stream, a, plan);
        return hipGetLastError();
    }
    // An XCD holds at most ceil(pairs / 8) pairs of at most qtiles items each;
    // workgroups past an XCD's item count exit at once.
    const int64_t pairs = (int64_t)num_sessions * p.num_kv_heads;
    const int64_t grid = (pairs + kXcds - 1) / kXcds * kXcds * a.qtiles;
    if (grid > 0x7FFFFFFFLL) return hipErrorInvalidConfiguration;
    const PrefillNoPlan none{0};
    const dim3 g((unsigned)grid);
    if (p.head_dim == 128)
        hipLaunchKernelGGL((prefill_kernel<128, false>), g, dim3(kPreThreads), 0, stream, a, none);
    else
        hipLaunchKernelGGL((prefill_kernel<64, false>), g, dim3(kPreThreads), 0, stream, a, none);
    return hipGetLastError();
}

}  // namespace ls
