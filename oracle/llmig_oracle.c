/*
 * CPU oracle for multi-stage KV-cache live migration (Llumnix, arXiv
 * 2406.03243).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or
 * call this file; only the test suite, the smoke check and the CPU-baseline
 * leg of the benchmark do.  It shares no code, header, constant or helper
 * with the GPU library: it is a plain, slow, obviously correct restatement
 * of what a migration computes, written against host copies of the pools.
 *
 * What a migration is (Llumnix §4.2, "Live Migration of LLM Requests"): the
 * KV cache of a running request is append-only, so the blocks it already
 * filled can be copied from the source instance's block pool to blocks the
 * destination reserved, stage after stage, while decoding continues; the
 * last stage copies what the final iteration added.  A migration therefore
 * reaches exactly a byte copy of whole KV blocks, and this oracle is that
 * definition written out.
 *
 * Pool layout (vLLM's paged KV cache, Llumnix §2 "Batching and memory
 * management" and §5 "Block fusion"): for every layer l there is one K
 * tensor and one V tensor of shape [num_blocks, block_size, kv_heads,
 * head_dim].  One (layer, K or V, block) tile is tile_bytes = block_size *
 * kv_heads * head_dim * elem_bytes contiguous bytes; token slot s of a block
 * occupies slot_bytes = kv_heads * head_dim * elem_bytes bytes at offset
 * s * slot_bytes inside its tile.
 *
 * Every routine below moves bytes with memcpy/memcmp and never interprets
 * them as numbers, so NaN payloads, signed zeros and subnormals pass through
 * untouched.
 *
 * Error classes (the same classes the library reports, defined here on
 * their own): ORACLE_OK, ORACLE_EINVAL (bad range or argument, duplicate
 * ids), ORACLE_ENOSPC (the destination could not reserve the blocks the
 * stage needs: the failed pre-allocation of the handshake, Llumnix §4.2),
 * ORACLE_ERANGE (a negative block id).
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

#define ORACLE_OK 0
#define ORACLE_EINVAL (-1)
#define ORACLE_ENOSPC (-2)
#define ORACLE_ERANGE (-3)

/*
 * Plan one migration stage (Llumnix §4.2: a stage first reserves its
 * destination blocks, then copies the KV produced since the stage before).
 *
 * The stage covers tokens [from_tok, to_tok) of a request whose first `len`
 * tokens are resident in the source pool.  Logical block j holds tokens
 * [j*bs, (j+1)*bs).  The stage's logical blocks are found by walking the
 * tokens one at a time and recording each block the walk enters; logical
 * block J[k] is paired with the k-th entry of the destination free list
 * (first come, first served).
 *
 * Readings of the paper that this follows:
 *  - a non-final stage copies only whole blocks, so from_tok must sit on a
 *    block boundary, and to_tok must too unless it is the end of the
 *    sequence (the last, partial block is copied by the final stage only);
 *  - the mapping takes destination blocks from the head of the free list in
 *    ascending logical order; the caller advances its free list by *out_n.
 *
 * Checks, in this order (the first failing one decides the result):
 *   1. out_n present                                 (else ORACLE_EINVAL);
 *   2. bs >= 1, 0 <= from_tok <= to_tok <= len;
 *   3. from_tok on a block boundary; to_tok on one unless to_tok == len;
 *   4. no negative table, free-list or output length;
 *   5. the source table holds every block of the first len tokens (and is
 *      present when it must hold any);
 *   6. the free list holds enough blocks            (else ORACLE_ENOSPC);
 *   7. the outputs hold the stage, and the free list and outputs are
 *      present when the stage is not empty;
 *   8. no negative block id among the stage's pairs  (else ORACLE_ERANGE);
 *   9. no block id repeated among the stage's sources, nor among its
 *      destinations.
 * Checks 2-5, 7 and 9 fail with ORACLE_EINVAL.
 * On any error *out_n is 0 (when out_n exists) and nothing else is written.
 */
int oracle_plan(const int32_t *src_table, int64_t src_table_len,
                const int32_t *dst_free_list, int64_t dst_free_len,
                int64_t len, int64_t from_tok, int64_t to_tok, int32_t bs,
                int32_t *out_src, int32_t *out_dst, int64_t out_cap,
                int64_t *out_n)
{
    if (out_n == NULL)
        return ORACLE_EINVAL;
    *out_n = 0;
    if (bs < 1 || len < 0 || from_tok < 0 || from_tok > to_tok || to_tok > len)
        return ORACLE_EINVAL;
    if (from_tok % bs != 0)
        return ORACLE_EINVAL;
    if (to_tok % bs != 0 && to_tok != len)
        return ORACLE_EINVAL;
    if (src_table_len < 0 || dst_free_len < 0 || out_cap < 0)
        return ORACLE_EINVAL;

    /* Blocks that hold the first len tokens: walk every token. */
    int64_t blocks_of_len = 0;
    int64_t last = -1;
    for (int64_t t = 0; t < len; t++) {
        if (t / bs != last) {
            last = t / bs;
            blocks_of_len++;
        }
    }
    if (src_table_len < blocks_of_len)
        return ORACLE_EINVAL;
    if (blocks_of_len > 0 && src_table == NULL)
        return ORACLE_EINVAL;

    /* Blocks the stage touches: walk the stage's tokens. */
    int64_t n = 0;
    int64_t first_block = -1;
    last = -1;
    for (int64_t t = from_tok; t < to_tok; t++) {
        if (t / bs != last) {
            last = t / bs;
            if (first_block < 0)
                first_block = last;
            n++;
        }
    }
    if (n > dst_free_len)
        return ORACLE_ENOSPC;
    if (n > out_cap)
        return ORACLE_EINVAL;
    if (n > 0 && (dst_free_list == NULL || out_src == NULL || out_dst == NULL))
        return ORACLE_EINVAL;

    for (int64_t k = 0; k < n; k++) {
        if (src_table[first_block + k] < 0 || dst_free_list[k] < 0)
            return ORACLE_ERANGE;
    }
    /* Pairwise comparison: slow, but plainly right. */
    for (int64_t a = 0; a < n; a++) {
        for (int64_t b = a + 1; b < n; b++) {
            if (src_table[first_block + a] == src_table[first_block + b])
                return ORACLE_EINVAL;
            if (dst_free_list[a] == dst_free_list[b])
                return ORACLE_EINVAL;
        }
    }

    for (int64_t k = 0; k < n; k++) {
        out_src[k] = src_table[first_block + k];
        out_dst[k] = dst_free_list[k];
    }
    *out_n = n;
    return ORACLE_OK;
}

/*
 * Copy one stage (Llumnix §4.2): for every pair (s, d), every layer l and
 * both K and V, the destination tile d receives the bytes of source tile s.
 * src_k[l], src_v[l], dst_k[l], dst_v[l] are host copies of the layer
 * tensors; tile_bytes is the size of one (layer, K/V, block) tile.
 */
void oracle_copy(uint8_t *const *src_k, uint8_t *const *src_v,
                 uint8_t *const *dst_k, uint8_t *const *dst_v,
                 int32_t num_layers, int64_t tile_bytes,
                 const int32_t *map_src, const int32_t *map_dst, int64_t n)
{
    for (int64_t i = 0; i < n; i++) {
        for (int32_t l = 0; l < num_layers; l++) {
            memcpy(dst_k[l] + (int64_t)map_dst[i] * tile_bytes,
                   src_k[l] + (int64_t)map_src[i] * tile_bytes, (size_t)tile_bytes);
            memcpy(dst_v[l] + (int64_t)map_dst[i] * tile_bytes,
                   src_v[l] + (int64_t)map_src[i] * tile_bytes, (size_t)tile_bytes);
        }
    }
}

/*
 * Block fusion, sending side (Llumnix §5 "Block fusion": the scattered
 * per-layer K/V blocks of a request are gathered into one contiguous buffer
 * so they travel as a single message).  The buffer is laid out
 * [layer][K=0, V=1][i][tile_bytes], i in the order of blocks[].
 */
void oracle_pack(uint8_t *const *pool_k, uint8_t *const *pool_v,
                 int32_t num_layers, int64_t tile_bytes,
                 const int32_t *blocks, int64_t n, uint8_t *staging)
{
    for (int32_t l = 0; l < num_layers; l++) {
        for (int kv = 0; kv < 2; kv++) {
            uint8_t *const *pool = (kv == 0) ? pool_k : pool_v;
            for (int64_t i = 0; i < n; i++) {
                int64_t slot = ((int64_t)l * 2 + kv) * n + i;
                memcpy(staging + slot * tile_bytes,
                       pool[l] + (int64_t)blocks[i] * tile_bytes, (size_t)tile_bytes);
            }
        }
    }
}

/* Block fusion, receiving side: the inverse of oracle_pack. */
void oracle_unpack(uint8_t *const *pool_k, uint8_t *const *pool_v,
                   int32_t num_layers, int64_t tile_bytes,
                   const int32_t *blocks, int64_t n, const uint8_t *staging)
{
    for (int32_t l = 0; l < num_layers; l++) {
        for (int kv = 0; kv < 2; kv++) {
            uint8_t *const *pool = (kv == 0) ? pool_k : pool_v;
            for (int64_t i = 0; i < n; i++) {
                int64_t slot = ((int64_t)l * 2 + kv) * n + i;
                memcpy(pool[l] + (int64_t)blocks[i] * tile_bytes,
                       staging + slot * tile_bytes, (size_t)tile_bytes);
            }
        }
    }
}

/*
 * Decoding appends KV (Llumnix §4.2: each iteration appends the KV of its
 * token and leaves earlier KV unchanged).  Writes tokens
 * [from_tok, from_tok + n_tok) into the pool through the request's block
 * table; data is laid out [layer][K=0, V=1][token][slot_bytes].
 */
void oracle_write_tokens(uint8_t *const *pool_k, uint8_t *const *pool_v,
                         int32_t num_layers, int32_t bs, int64_t slot_bytes,
                         const int32_t *table, int64_t from_tok, int64_t n_tok,
                         const uint8_t *data)
{
    int64_t tile_bytes = (int64_t)bs * slot_bytes;
    for (int32_t l = 0; l < num_layers; l++) {
        for (int kv = 0; kv < 2; kv++) {
            uint8_t *const *pool = (kv == 0) ? pool_k : pool_v;
            for (int64_t j = 0; j < n_tok; j++) {
                int64_t t = from_tok + j;
                uint8_t *slot = pool[l] + (int64_t)table[t / bs] * tile_bytes
                              + (t % bs) * slot_bytes;
                memcpy(slot, data + (((int64_t)l * 2 + kv) * n_tok + j) * slot_bytes,
                       (size_t)slot_bytes);
            }
        }
    }
}

/*
 * Token identity, the property a migration must establish: for every token
 * t < len, every layer and both K and V, the bytes of t's slot reached
 * through table_a in pool a equal those reached through table_b in pool b.
 * Returns -1 when all match, else the first token that differs.
 */
int64_t oracle_first_token_mismatch(uint8_t *const *a_k, uint8_t *const *a_v,
                                    const int32_t *table_a,
                                    uint8_t *const *b_k, uint8_t *const *b_v,
                                    const int32_t *table_b,
                                    int32_t num_layers, int32_t bs,
                                    int64_t slot_bytes, int64_t len)
{
    int64_t tile_bytes = (int64_t)bs * slot_bytes;
    for (int64_t t = 0; t < len; t++) {
        for (int32_t l = 0; l < num_layers; l++) {
            int64_t off_a = (int64_t)table_a[t / bs] * tile_bytes + (t % bs) * slot_bytes;
            int64_t off_b = (int64_t)table_b[t / bs] * tile_bytes + (t % bs) * slot_bytes;
            if (memcmp(a_k[l] + off_a, b_k[l] + off_b, (size_t)slot_bytes) != 0)
                return t;
            if (memcmp(a_v[l] + off_a, b_v[l] + off_b, (size_t)slot_bytes) != 0)
                return t;
        }
    }
    return -1;
}

/* ------------------------------------------------------------------------
 * Decode attention over the paged pool (the work that runs beside a
 * migration and whose slowdown Llumnix §6.2 measures).  For every layer l,
 * sequence b and query head h (served by KV head g = h / (q_heads /
 * kv_heads), grouped-query attention), with the sequence's ctx tokens
 * reached through its block table:
 *     s_t = scale * sum_d q[l][b][h][d] * K_l[t][g][d]
 *     p_t = exp(s_t - max_t s) / sum_t exp(s_t - max_t s)
 *     out[l][b][h][d] = sum_t p_t * V_l[t][g][d]
 * in double precision; a sequence with ctx = 0 gives zeros.
 * ---------------------------------------------------------------------- */

/* IEEE 754 binary16 bits to double, from the format: 1 sign bit, 5 exponent
 * bits (bias 15), 10 fraction bits; exponent 0 encodes zero and subnormals,
 * 31 infinities and NaNs. */
double oracle_half_to_double(uint16_t h)
{
    int sign = (h >> 15) & 1;
    int exp = (h >> 10) & 0x1f;
    int frac = h & 0x3ff;
    double v;
    if (exp == 0)
        v = ldexp((double)frac, -24);
    else if (exp == 31)
        v = frac ? NAN : INFINITY;
    else
        v = ldexp((double)(frac | 0x400), exp - 25);
    return sign ? -v : v;
}

/* bfloat16 bits to double: the upper half of an IEEE binary32. */
double oracle_bf16_to_double(uint16_t h)
{
    uint32_t bits = (uint32_t)h << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
}

static double elem(const uint8_t *base, int64_t index, int is_bf16)
{
    uint16_t bits;
    memcpy(&bits, base + index * 2, 2);
    return is_bf16 ? oracle_bf16_to_double(bits) : oracle_half_to_double(bits);
}

/* q: [num_layers][batch][q_heads][head_dim] 16-bit; tables: [batch][table_stride]
 * block ids; ctx: [batch]; out: [num_layers][batch][q_heads][head_dim] double. */
void oracle_decode_attention(uint8_t *const *pool_k, uint8_t *const *pool_v, int32_t num_layers,
                             int32_t block_size, int32_t kv_heads, int32_t head_dim, int is_bf16,
                             const uint8_t *q, int32_t batch, int32_t q_heads,
                             const int32_t *tables, int32_t table_stride, const int32_t *ctx,
                             double scale, double *out)
{
    int32_t group = q_heads / kv_heads;
    for (int32_t l = 0; l < num_layers; l++) {
        for (int32_t b = 0; b < batch; b++) {
            for (int32_t h = 0; h < q_heads; h++) {
                int32_t g = h / group;
                int64_t qoff = (((int64_t)l * batch + b) * q_heads + h) * head_dim;
                double *o = out + qoff;
                for (int32_t d = 0; d < head_dim; d++)
                    o[d] = 0.0;
                if (ctx[b] <= 0)
                    continue;
                double smax = -INFINITY;
                for (int32_t t = 0; t < ctx[b]; t++) {
                    int64_t row = ((int64_t)tables[(int64_t)b * table_stride + t / block_size] * block_size
                                   + t % block_size) * kv_heads + g;
                    double s = 0.0;
                    for (int32_t d = 0; d < head_dim; d++)
                        s += elem(q, qoff + d, is_bf16) * elem(pool_k[l], row * head_dim + d, is_bf16);
                    s *= scale;
                    if (s > smax)
                        smax = s;
                }
                double denom = 0.0;
                for (int32_t t = 0; t < ctx[b]; t++) {
                    int64_t row = ((int64_t)tables[(int64_t)b * table_stride + t / block_size] * block_size
                                   + t % block_size) * kv_heads + g;
                    double s = 0.0;
                    for (int32_t d = 0; d < head_dim; d++)
                        s += elem(q, qoff + d, is_bf16) * elem(pool_k[l], row * head_dim + d, is_bf16);
                    double w = exp(s * scale - smax);
                    denom += w;
                    for (int32_t d = 0; d < head_dim; d++)
                        o[d] += w * elem(pool_v[l], row * head_dim + d, is_bf16);
                }
                for (int32_t d = 0; d < head_dim; d++)
                    o[d] /= denom;
            }
        }
    }
}

/* ------------------------------------------------------------------------
 * Cross-layout migration: the source and destination instances keep the
 * (token, head, dim) elements of a tile in different orders.  The copy is
 * then no longer a byte copy of tiles but the same elements placed where
 * the destination's layout puts them; whole tiles still move (a partial
 * last block carries its unused slots along).  Llumnix migrates between
 * instances of one engine (§4.2); this generalisation keeps its definition,
 * element for element.
 *
 * Layouts of one tile of bs tokens, H heads, D dims, e-byte elements
 * (x = 16 / e elements form one 16-byte group of a head's dims):
 *   ORACLE_LAYOUT_NHD  [bs][H][D]         token-major (the vLLM pool above)
 *   ORACLE_LAYOUT_HND  [H][bs][D]         head-major
 *   ORACLE_LAYOUT_HCNX [H][D/x][bs][x]    vLLM paged attention's key cache
 *   ORACLE_LAYOUT_HDN  [H][D][bs]         vLLM paged attention's value cache
 * ---------------------------------------------------------------------- */
#define ORACLE_LAYOUT_NHD 0
#define ORACLE_LAYOUT_HND 1
#define ORACLE_LAYOUT_HCNX 2
#define ORACLE_LAYOUT_HDN 3

/* Byte offset of element (t, h, d) inside a tile, or -1 for an unknown
 * layout or an element size that does not divide 16 (HCNX only). */
int64_t oracle_layout_offset(int32_t layout, int64_t t, int64_t h, int64_t d,
                             int32_t bs, int32_t heads, int32_t head_dim, int32_t elem_bytes)
{
    int64_t index;
    if (layout == ORACLE_LAYOUT_NHD) {
        index = (t * heads + h) * head_dim + d;
    } else if (layout == ORACLE_LAYOUT_HND) {
        index = (h * bs + t) * head_dim + d;
    } else if (layout == ORACLE_LAYOUT_HCNX) {
        if (elem_bytes <= 0 || 16 % elem_bytes != 0)
            return -1;
        int64_t x = 16 / elem_bytes;
        int64_t groups = head_dim / x;
        index = ((h * groups + d / x) * bs + t) * x + d % x;
    } else if (layout == ORACLE_LAYOUT_HDN) {
        index = (h * head_dim + d) * bs + t;
    } else {
        return -1;
    }
    return index * elem_bytes;
}

/* One stage between pools of different layouts: for every pair (s, d),
 * every layer and both K and V, every element (t, h, dim) of source tile s
 * is written to the position the destination layout gives it in tile d.
 * layouts[0] / layouts[1] are the K / V layouts of each side. */
void oracle_copy_layout(uint8_t *const *src_k, uint8_t *const *src_v, const int32_t *src_layouts,
                        uint8_t *const *dst_k, uint8_t *const *dst_v, const int32_t *dst_layouts,
                        int32_t num_layers, int32_t bs, int32_t heads, int32_t head_dim,
                        int32_t elem_bytes, const int32_t *map_src, const int32_t *map_dst, int64_t n)
{
    int64_t tile_bytes = (int64_t)bs * heads * head_dim * elem_bytes;
    for (int64_t i = 0; i < n; i++) {
        for (int32_t l = 0; l < num_layers; l++) {
            for (int kv = 0; kv < 2; kv++) {
                const uint8_t *s = (kv == 0 ? src_k : src_v)[l] + (int64_t)map_src[i] * tile_bytes;
                uint8_t *d = (kv == 0 ? dst_k : dst_v)[l] + (int64_t)map_dst[i] * tile_bytes;
                for (int64_t t = 0; t < bs; t++)
                    for (int64_t h = 0; h < heads; h++)
                        for (int64_t e = 0; e < head_dim; e++)
                            memcpy(d + oracle_layout_offset(dst_layouts[kv], t, h, e, bs, heads,
                                                            head_dim, elem_bytes),
                                   s + oracle_layout_offset(src_layouts[kv], t, h, e, bs, heads,
                                                            head_dim, elem_bytes),
                                   (size_t)elem_bytes);
            }
        }
    }
}

/* Decoding's KV appends into a pool of any layout: data is laid out
 * [layer][K=0, V=1][token][H][D] (each token's K or V in head, dim order)
 * and element (h, dim) of token t goes where the pool's layout puts it in
 * slot t % bs of block table[t / bs]. */
void oracle_write_tokens_layout(uint8_t *const *pool_k, uint8_t *const *pool_v,
                                const int32_t *layouts, int32_t num_layers, int32_t bs,
                                int32_t heads, int32_t head_dim, int32_t elem_bytes,
                                const int32_t *table, int64_t from_tok, int64_t n_tok,
                                const uint8_t *data)
{
    int64_t tile_bytes = (int64_t)bs * heads * head_dim * elem_bytes;
    for (int32_t l = 0; l < num_layers; l++) {
        for (int kv = 0; kv < 2; kv++) {
            uint8_t *const *pool = (kv == 0) ? pool_k : pool_v;
            for (int64_t j = 0; j < n_tok; j++) {
                int64_t t = from_tok + j;
                uint8_t *tile = pool[l] + (int64_t)table[t / bs] * tile_bytes;
                const uint8_t *src = data + (((int64_t)l * 2 + kv) * n_tok + j) * heads * head_dim * elem_bytes;
                for (int64_t h = 0; h < heads; h++)
                    for (int64_t e = 0; e < head_dim; e++)
                        memcpy(tile + oracle_layout_offset(layouts[kv], t % bs, h, e, bs, heads,
                                                           head_dim, elem_bytes),
                               src + (h * head_dim + e) * elem_bytes, (size_t)elem_bytes);
            }
        }
    }
}

/* Token identity across layouts: -1 when every element (t < len, every
 * layer, K and V, every head and dim) read through table_a and a's layouts
 * equals the one read through table_b and b's layouts; else the first token
 * that differs. */
int64_t oracle_first_token_mismatch_layout(uint8_t *const *a_k, uint8_t *const *a_v,
                                           const int32_t *a_layouts, const int32_t *table_a,
                                           uint8_t *const *b_k, uint8_t *const *b_v,
                                           const int32_t *b_layouts, const int32_t *table_b,
                                           int32_t num_layers, int32_t bs, int32_t heads,
                                           int32_t head_dim, int32_t elem_bytes, int64_t len)
{
    int64_t tile_bytes = (int64_t)bs * heads * head_dim * elem_bytes;
    for (int64_t t = 0; t < len; t++) {
        for (int32_t l = 0; l < num_layers; l++) {
            for (int kv = 0; kv < 2; kv++) {
                const uint8_t *ta = (kv == 0 ? a_k : a_v)[l] + (int64_t)table_a[t / bs] * tile_bytes;
                const uint8_t *tb = (kv == 0 ? b_k : b_v)[l] + (int64_t)table_b[t / bs] * tile_bytes;
                for (int64_t h = 0; h < heads; h++)
                    for (int64_t e = 0; e < head_dim; e++)
                        if (memcmp(ta + oracle_layout_offset(a_layouts[kv], t % bs, h, e, bs, heads,
                                                             head_dim, elem_bytes),
                                   tb + oracle_layout_offset(b_layouts[kv], t % bs, h, e, bs, heads,
                                                             head_dim, elem_bytes),
                                   (size_t)elem_bytes) != 0)
                            return t;
            }
        }
    }
    return -1;
}

/* Block fusion's receiving side between engines of different layouts: the
 * staging buffer (laid out as oracle_pack writes it) holds tiles whose
 * elements follow staging_layouts (K, V); every element (t, h, dim) of
 * slot ((l * 2 + kv) * n + i) lands in tile (l, kv) of pool block
 * blocks[i] where the pool's layouts put it. */
void oracle_unpack_layout(uint8_t *const *pool_k, uint8_t *const *pool_v, const int32_t *pool_layouts,
                          const int32_t *staging_layouts, int32_t num_layers, int32_t bs, int32_t heads,
                          int32_t head_dim, int32_t elem_bytes, const int32_t *blocks, int64_t n,
                          const uint8_t *staging)
{
    int64_t tile_bytes = (int64_t)bs * heads * head_dim * elem_bytes;
    for (int32_t l = 0; l < num_layers; l++) {
        for (int kv = 0; kv < 2; kv++) {
            uint8_t *const *pool = (kv == 0) ? pool_k : pool_v;
            for (int64_t i = 0; i < n; i++) {
                const uint8_t *s = staging + (((int64_t)l * 2 + kv) * n + i) * tile_bytes;
                uint8_t *d = pool[l] + (int64_t)blocks[i] * tile_bytes;
                for (int64_t t = 0; t < bs; t++)
                    for (int64_t h = 0; h < heads; h++)
                        for (int64_t e = 0; e < head_dim; e++)
                            memcpy(d + oracle_layout_offset(pool_layouts[kv], t, h, e, bs, heads,
                                                            head_dim, elem_bytes),
                                   s + oracle_layout_offset(staging_layouts[kv], t, h, e, bs, heads,
                                                            head_dim, elem_bytes),
                                   (size_t)elem_bytes);
            }
        }
    }
}
