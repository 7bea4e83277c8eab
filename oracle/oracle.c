/*
 * CPU oracle for the paged-KV hot path of LiveServe (arXiv 2606.22983).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is a plain, slow, obviously-correct
 * reference.  Only the test suite, the package smoke check and the benchmark's
 * cpu_baseline leg may load it.  It shares no code, header, table or helper
 * with the GPU library; it knows the pool layout only from the written
 * definition below.
 *
 * What it computes (all floating point in fp64; bf16 inputs are widened
 * exactly):
 *
 *   attend   exact softmax attention of one query row over the first n keys
 *            of a session, keys located through the session's block table.
 *            The paper (§2.1, §5) runs the thinker/talker as autoregressive
 *            decoders over a paged, block-allocated KV cache (§5.1 keeps
 *            block-level allocation; §6 extends the paged KV block pool) but
 *            does not restate attention itself; the operation is the textbook
 *            scaled dot-product softmax attention, with grouped query heads
 *            (query head h reads KV head h / (Hq/Hkv)).
 *   append   write new tokens' K and V rows into their pool slots: the slot of
 *            logical token t of session s is (block_table[s][t / B], t % B).
 *   stash    gather whole blocks (every layer, K and V) into a contiguous
 *            staging array, one block after another — the HBM-to-DRAM offload
 *            of idle multi-turn KV (§5, §5.1: eviction stays block-level).
 *   restore  the inverse scatter — the DRAM-to-HBM reload / speech-triggered
 *            preload of §5.2.
 *
 * Pool layout (definition; bf16 stored as uint16):
 *   pool[layer][block][kv][head][tile]   kv = 0 for K, 1 for V
 *   K tile: [chunk d/W in 0..D/W-1][token o in 0..B-1][d%W], W = min(8, D)
 *           (chunk-major)
 *   V tile: [dim d in 0..D-1][token o in 0..B-1]   (dim-major)
 * Staging layout for stash/restore: staging[i][layer][kv][head][tile], i.e.
 * the per-layer (kv, head, tile) slab of block ids[i] for every layer, block
 * after block.
 *
 * Parity is pinned by the CPU tests: reduction to a library attention routine,
 * brute force on tiny inputs, closed forms and invariants.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

static double widen_bf16(uint16_t bits)
{
    uint32_t word = (uint32_t)bits << 16;
    float f;
    memcpy(&f, &word, sizeof f);
    return (double)f;
}

static int64_t k_index(int64_t num_blocks, int num_kv_heads, int head_dim, int block_size,
                       int layer, int64_t block, int head, int token, int dim)
{
    int64_t tile = (((int64_t)layer * num_blocks + block) * 2 + 0) * num_kv_heads + head;
    int w = head_dim < 8 ? head_dim : 8;          /* chunk width in dims */
    return ((tile * (head_dim / w) + dim / w) * block_size + token) * w + dim % w;
}

static int64_t v_index(int64_t num_blocks, int num_kv_heads, int head_dim, int block_size,
                       int layer, int64_t block, int head, int token, int dim)
{
    int64_t tile = (((int64_t)layer * num_blocks + block) * 2 + 1) * num_kv_heads + head;
    return (tile * head_dim + dim) * block_size + token;
}

/*
 * Attention rows.  Row r is a query of session row_session[r] that sees keys
 * 0 .. row_keys[r]-1 of that session; its Hq query heads are
 * q[row_q_index[r]][h][:] and the result goes to out[r][h][:] (fp64).
 * Decode is one row per session with row_keys = context length (plus one when
 * the step's own token was appended); next-turn prefill row j of a session
 * with reused context c sees keys 0 .. c + j (bottom-right causal alignment).
 * Returns 0, or -1 if a row has no key (softmax over an empty set) or a block
 * id lies outside the pool.
 */
int oracle_attend(const uint16_t *pool, int num_layers, int64_t num_blocks, int num_kv_heads,
                  int head_dim, int block_size, int layer, int num_q_heads,
                  const int32_t *block_tables, int max_blocks_per_session,
                  int num_rows, const int32_t *row_session, const int32_t *row_keys,
                  const int64_t *row_q_index, const uint16_t *q, double scale, double *out)
{
    if (layer < 0 || layer >= num_layers) return -1;
    int group = num_q_heads / num_kv_heads;
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : bad)
    for (int64_t job = 0; job < (int64_t)num_rows * num_q_heads; ++job) {
        int r = (int)(job / num_q_heads);
        int h = (int)(job % num_q_heads);
        int s = row_session[r];
        int n = row_keys[r];
        int g = h / group;
        const uint16_t *qrow = q + (row_q_index[r] * num_q_heads + h) * head_dim;
        double *o = out + ((int64_t)r * num_q_heads + h) * head_dim;
        for (int d = 0; d < head_dim; ++d) o[d] = 0.0;
        if (n <= 0 || (n + block_size - 1) / block_size > max_blocks_per_session) {
            bad = 1;
            continue;
        }
        /* scores x_t = scale * <q, k_t> */
        double *x = (double *)malloc(sizeof(double) * (size_t)n);
        if (!x) { bad = 1; continue; }
        double mu = -INFINITY;
        for (int t = 0; t < n; ++t) {
            int64_t b = block_tables[(int64_t)s * max_blocks_per_session + t / block_size];
            if (b < 0 || b >= num_blocks) { bad = 1; mu = NAN; break; }
            double dot = 0.0;
            for (int d = 0; d < head_dim; ++d)
                dot += widen_bf16(qrow[d]) *
                       widen_bf16(pool[k_index(num_blocks, num_kv_heads, head_dim, block_size,
                                               layer, b, g, t % block_size, d)]);
            x[t] = scale * dot;
            if (x[t] > mu) mu = x[t];
        }
        if (isnan(mu)) { free(x); continue; }
        /* softmax weights w_t = exp(x_t - max) and the weighted mean of V */
        double wsum = 0.0;
        for (int t = 0; t < n; ++t) {
            int64_t b = block_tables[(int64_t)s * max_blocks_per_session + t / block_size];
            double w = exp(x[t] - mu);
            wsum += w;
            for (int d = 0; d < head_dim; ++d)
                o[d] += w * widen_bf16(pool[v_index(num_blocks, num_kv_heads, head_dim, block_size,
                                                    layer, b, g, t % block_size, d)]);
        }
        for (int d = 0; d < head_dim; ++d) o[d] /= wsum;
        free(x);
    }
    return bad ? -1 : 0;
}

/*
 * Append: token i (i < num_tokens) belongs to session tok_session[i] at
 * logical position tok_pos[i]; its K row is k_new[i][head][:] and its V row
 * v_new[i][head][:].  Both are written into the pool slot given by the block
 * table.  Returns -1 on an out-of-range slot, 0 otherwise.
 */
int oracle_append(uint16_t *pool, int num_layers, int64_t num_blocks, int num_kv_heads,
                  int head_dim, int block_size, int layer,
                  const int32_t *block_tables, int max_blocks_per_session,
                  int num_tokens, const int32_t *tok_session, const int32_t *tok_pos,
                  const uint16_t *k_new, const uint16_t *v_new)
{
    if (layer < 0 || layer >= num_layers) return -1;
    for (int i = 0; i < num_tokens; ++i) {
        int s = tok_session[i];
        int t = tok_pos[i];
        if (t < 0 || t / block_size >= max_blocks_per_session) return -1;
        int64_t b = block_tables[(int64_t)s * max_blocks_per_session + t / block_size];
        if (b < 0 || b >= num_blocks) return -1;
        for (int g = 0; g < num_kv_heads; ++g)
            for (int d = 0; d < head_dim; ++d) {
                int64_t src = ((int64_t)i * num_kv_heads + g) * head_dim + d;
                pool[k_index(num_blocks, num_kv_heads, head_dim, block_size, layer, b, g,
                             t % block_size, d)] = k_new[src];
                pool[v_index(num_blocks, num_kv_heads, head_dim, block_size, layer, b, g,
                             t % block_size, d)] = v_new[src];
            }
    }
    return 0;
}

/* Bytes of one (layer, block) slab: K and V tiles of every KV head. */
static int64_t slab_bytes(int num_kv_heads, int head_dim, int block_size)
{
    return (int64_t)2 * num_kv_heads * block_size * head_dim * (int64_t)sizeof(uint16_t);
}

/* Stash: staging[i][layer] <- pool[layer][ids[i]] for every layer.  Byte copy. */
int oracle_stash(const uint16_t *pool, int num_layers, int64_t num_blocks, int num_kv_heads,
                 int head_dim, int block_size, int n, const int32_t *ids, uint16_t *staging)
{
    int64_t slab = slab_bytes(num_kv_heads, head_dim, block_size);
    for (int i = 0; i < n; ++i) {
        if (ids[i] < 0 || ids[i] >= num_blocks) return -1;
        for (int l = 0; l < num_layers; ++l)
            memcpy((char *)staging + ((int64_t)i * num_layers + l) * slab,
                   (const char *)pool + ((int64_t)l * num_blocks + ids[i]) * slab, (size_t)slab);
    }
    return 0;
}

/* Restore: pool[layer][ids[i]] <- staging[i][layer] for every layer.  Byte copy. */
int oracle_restore(uint16_t *pool, int num_layers, int64_t num_blocks, int num_kv_heads,
                   int head_dim, int block_size, int n, const int32_t *ids,
                   const uint16_t *staging)
{
    int64_t slab = slab_bytes(num_kv_heads, head_dim, block_size);
    for (int i = 0; i < n; ++i) {
        if (ids[i] < 0 || ids[i] >= num_blocks) return -1;
        for (int l = 0; l < num_layers; ++l)
            memcpy((char *)pool + ((int64_t)l * num_blocks + ids[i]) * slab,
                   (const char *)staging + ((int64_t)i * num_layers + l) * slab, (size_t)slab);
    }
    return 0;
}
