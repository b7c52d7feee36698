/*
 * hma_oracle.c -- plain, slow, float64 CPU oracle for the deferred-dequantization
 * decode path of HMA-Serve ("HBM Is Not All You Need", arXiv 2606.29986).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, includes or
 * calls this file; it shares no code, header, table or constant generator with
 * the HIP kernels.  Only the test suite, the package smoke check and the
 * CPU-baseline leg of the benchmark may load it.
 *
 * What it computes (paper section in brackets):
 *   - BF16 <-> float64 conversions used to state results exactly.
 *   - Block-float (BFP8) decode: a per-block shared exponent and a per-element
 *     7-bit mantissa are turned into a BF16 value [Sec. 3.3].  Two independent
 *     routes are given: a value-level definition (exact real value, then
 *     round-to-nearest-even into BF16) and a bit-assembly route (the shifts,
 *     masks and ORs the paper describes).  They must agree on every input.
 *   - BFP8 encode, used only to manufacture test inputs: the paper's prefill
 *     side produces BFP8 KV [Sec. 3.1]; the decode GPU never encodes.
 *   - Page reconstruction: BFP8 pages -> BF16 pages of the paged row-major KV
 *     cache [Sec. 1, Sec. 2.3 Challenge 2, Sec. 3.3].
 *   - Tiled per-chip prefill shards -> BF16 pages (shard merge, post-rotary
 *     key re-layout, decode) and -> raw BFP8 pages with the bytes unchanged
 *     [Sec. 3.3]; the paper gives no tile byte order, the one used is stated
 *     at ora_rebuild_tiled.
 *   - Single-token GQA decode attention over the paged cache, where each page
 *     is either raw BFP8 (decoded on read) or already BF16 [Sec. 3.3, Fig. 2],
 *     in float64 from the softmax-attention definition; keys may be stored in
 *     the interleaved rotary order and are then relabelled on read.
 *   - Split-K partials over arbitrary contiguous token ranges and their
 *     log-sum-exp merge (a reformulation of the same softmax; not in the paper).
 *
 * Format readings where the paper is silent (sign, exponent bias, block size,
 * layout) are the ones listed in the design notes: element byte = sign bit 7 +
 * 7-bit magnitude m, block = 16 consecutive head-dim channels of one token,
 * exponent byte E with bias 127, value = (-1)^s * m * 2^(E-133).
 *
 * Layouts (all row-major, little-endian):
 *   mantissa pool  uint8  [pages][Hkv][P][D]
 *   exponent pool  uint8  [pages][Hkv][P][D/16]
 *   BF16 pool      uint16 [pages][Hkv][P][D]
 *   page table     int32  [B][max_pages]; bit 30 set = page lives in the BF16
 *                  pool; physical id = entry & 0x3FFFFFFF; slot = t % P.
 */
#include <math.h>
#include <stdint.h>
#include <stddef.h>
#include <stdlib.h>
#include <string.h>

#define ORA_BLOCK 16          /* channels per shared exponent (reading of Sec. 3.3) */
#define ORA_EXP_OFFSET 133    /* 127 bias + 6: m/64 is the significand of the block max */
#define ORA_TAG_BF16 0x40000000
#define ORA_ID_MASK 0x3FFFFFFF

/* ------------------------------------------------------------------ BF16 */

/* BF16 bits -> float64.  Exact: BF16 is the upper half of an IEEE binary32. */
double ora_bf16_to_f64(uint16_t b)
{
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/* float64 -> BF16 bits, round to nearest, ties to even; overflow -> +-Inf,
 * NaN -> quiet NaN.  Written from the definition of the binary16-brain format:
 * 8 exponent bits (bias 127), 7 stored fraction bits, subnormals at 2^-133
 * spacing. */
uint16_t ora_f64_to_bf16(double v)
{
    if (isnan(v))
        return (uint16_t)(signbit(v) ? 0xFFC0 : 0x7FC0);
    uint16_t sign = signbit(v) ? 0x8000 : 0;
    double a = fabs(v);
    if (isinf(a))
        return (uint16_t)(sign | 0x7F80);
    if (a == 0.0)
        return sign;
    if (a < ldexp(1.0, -126)) {
        /* subnormal range: value = q * 2^-133, q in [0,128]; q = 128 is the
         * smallest normal and its bit pattern is exactly 0x0080 */
        double q = nearbyint(ldexp(a, 133));   /* default mode: ties to even */
        return (uint16_t)(sign | (uint16_t)q);
    }
    int e;
    double f = frexp(a, &e);                   /* a = f * 2^e, f in [0.5, 1) */
    double q = nearbyint(ldexp(f, 8));         /* 8 significant bits: [128, 256] */
    if (q == 256.0) {
        q = 128.0;
        e += 1;
    }
    int field = e - 1 + 127;
    if (field >= 255)
        return (uint16_t)(sign | 0x7F80);
    return (uint16_t)(sign | (uint16_t)(field << 7) | (uint16_t)((int)q - 128));
}

/* --------------------------------------------------------- BFP8 decode */

/* Value-level decode of one element [Sec. 3.3: shared exponent + 7-bit mantissa].
 * x = (-1)^s * m * 2^(E-133), computed exactly in float64 and rounded to BF16.
 * The rounding is exact for every E <= 254; E = 255 with m >= 64 overflows to
 * Inf, and m = 0 gives a zero carrying the sign bit. */
uint16_t ora_bfp8_decode_value(uint8_t E, uint8_t byte)
{
    int s = byte >> 7;
    int m = byte & 0x7F;
    double v = ldexp((double)m, (int)E - ORA_EXP_OFFSET);
    if (s)
        v = -v;                      /* m = 0 gives -0.0, which keeps its sign */
    return ora_f64_to_bf16(v);
}

/* Bit-assembly decode of one element: the shifts / masks / ORs route the paper
 * names [Sec. 3.3, Sec. 2.3 Challenge 2].  Independent of the value-level route;
 * the two are cross-checked on all 65,536 (E, byte) pairs. */
uint16_t ora_bfp8_decode_bits(uint8_t E, uint8_t byte)
{
    uint32_t s = (uint32_t)(byte >> 7);
    uint32_t m = (uint32_t)(byte & 0x7F);
    if (m == 0)
        return (uint16_t)(s << 15);
    int lz = 0;                       /* leading zeros of m inside its 7-bit field */
    while (!(m & (0x40u >> lz)))
        lz++;
    int e = (int)E - lz;              /* biased exponent of the normalised value */
    if (e >= 255)
        return (uint16_t)((s << 15) | 0x7F80);
    if (e >= 1) {
        uint32_t frac = (m << (lz + 1)) & 0x7F;   /* drop the leading one */
        return (uint16_t)((s << 15) | ((uint32_t)e << 7) | frac);
    }
    /* BF16 subnormal: stored fraction = value / 2^-133 = m * 2^E */
    return (uint16_t)((s << 15) | (m << E));
}

/* --------------------------------------------------------- BFP8 encode */

/* Encode one block of 16 finite BF16 values (test-input manufacture only).
 *   E    = largest exponent field in the block (0 if all zero / subnormal)
 *   m_i  = round-half-even(|x_i| * 2^(133-E)), clamped to 127
 *   s_i  = sign of x_i, cleared when m_i = 0
 * Returns 0, or -1 if an input is NaN or Inf (nothing is written then). */
int ora_bfp8_encode_block(const uint16_t *x, uint8_t *E_out, uint8_t *bytes_out)
{
    int E = 0;
    for (int i = 0; i < ORA_BLOCK; i++) {
        int field = (x[i] >> 7) & 0xFF;
        if (field == 0xFF)
            return -1;
        if (field > E)
            E = field;
    }
    for (int i = 0; i < ORA_BLOCK; i++) {
        double a = fabs(ora_bf16_to_f64(x[i]));
        double q = nearbyint(ldexp(a, ORA_EXP_OFFSET - E));   /* exact scaling, RNE */
        if (q > 127.0)
            q = 127.0;
        int m = (int)q;
        int s = (x[i] >> 15) & 1;
        if (m == 0)
            s = 0;
        bytes_out[i] = (uint8_t)((s << 7) | m);
    }
    *E_out = (uint8_t)E;
    return 0;
}

/* Encode n_blocks consecutive 16-element blocks: block k reads x[16k..16k+15],
 * writes bytes[16k..16k+15] and exps[k].  With the page layouts above, encoding
 * a whole BF16 pool in order yields the matching mantissa and exponent pools.
 * Returns 0, or -1 if any input is non-finite (the blocks holding one are left
 * unwritten). */
int ora_bfp8_encode_blocks(const uint16_t *x, int64_t n_blocks, uint8_t *bytes, uint8_t *exps)
{
    int bad = 0;
    #pragma omp parallel for schedule(static) reduction(|:bad)
    for (int64_t k = 0; k < n_blocks; k++)
        bad |= ora_bfp8_encode_block(x + k * ORA_BLOCK, exps + k, bytes + k * ORA_BLOCK) != 0;
    return bad ? -1 : 0;
}

/* Decode n_blocks consecutive blocks with the value-level route. */
void ora_bfp8_decode_blocks(const uint8_t *bytes, const uint8_t *exps, int64_t n_blocks, uint16_t *out)
{
    #pragma omp parallel for schedule(static)
    for (int64_t k = 0; k < n_blocks; k++)
        for (int i = 0; i < ORA_BLOCK; i++)
            out[k * ORA_BLOCK + i] = ora_bfp8_decode_value(exps[k], bytes[k * ORA_BLOCK + i]);
}

/* Decode n_blocks consecutive blocks with the bit-assembly route. */
void ora_bfp8_decode_blocks_bits(const uint8_t *bytes, const uint8_t *exps, int64_t n_blocks, uint16_t *out)
{
    for (int64_t k = 0; k < n_blocks; k++)
        for (int i = 0; i < ORA_BLOCK; i++)
            out[k * ORA_BLOCK + i] = ora_bfp8_decode_bits(exps[k], bytes[k * ORA_BLOCK + i]);
}

/* ----------------------------------------------- page reconstruction */

/* Lazy reconstruction of BFP8 pages into the paged BF16 cache [Sec. 3.3].
 * For every pool p in [0, n_pools) and pair i in [0, n_pages): the (page,
 * all heads) tile src_pages[i] of BFP8 pool p is decoded into page
 * dst_pages[i] of BF16 pool p.  Pool p starts src_pool_stride_pages pages
 * after pool 0 (mantissa and exponent pools alike) and dst_pool_stride_pages
 * pages after BF16 pool 0.  Pages not named in dst_pages are left untouched. */
void ora_dequant_pages(const uint8_t *src_mant, const uint8_t *src_exp, uint16_t *dst,
                       const int32_t *src_pages, const int32_t *dst_pages, int32_t n_pages,
                       int32_t n_pools, int64_t src_pool_stride_pages, int64_t dst_pool_stride_pages,
                       int32_t num_kv_heads, int32_t head_dim, int32_t page_size)
{
    const int64_t page_elems = (int64_t)num_kv_heads * page_size * head_dim;
    const int64_t page_blocks = page_elems / ORA_BLOCK;
    #pragma omp parallel for collapse(2) schedule(static)
    for (int32_t p = 0; p < n_pools; p++)
        for (int32_t i = 0; i < n_pages; i++) {
            const uint8_t *mant = src_mant + (p * src_pool_stride_pages + src_pages[i]) * page_elems;
            const uint8_t *ex = src_exp + (p * src_pool_stride_pages + src_pages[i]) * page_blocks;
            uint16_t *out = dst + (p * dst_pool_stride_pages + dst_pages[i]) * page_elems;
            for (int64_t k = 0; k < page_blocks; k++)
                for (int c = 0; c < ORA_BLOCK; c++)
                    out[k * ORA_BLOCK + c] = ora_bfp8_decode_value(ex[k], mant[k * ORA_BLOCK + c]);
        }
}

/* ------------------------------------- tiled shards -> BF16 pages */

/* The decoder's single reconstruction pass also turns the prefill side's
 * tiled layout into row-major pages, merges the per-chip KV shards, and
 * moves keys from the interleaved rotary order to the half-split order
 * [Sec. 3.3; Sec. 2.3: the prefill chips work on 32x32 tiles].  The paper
 * gives no byte order for the tiles; the order used here is:
 *   shard t (chip t of n_shards) holds KV heads [t*Hs, (t+1)*Hs), Hs = Hkv/n_shards;
 *   a shard is tiles [local head h][token tile (32 tokens)][channel tile (32 channels)];
 *   a tile is 64 exponent bytes [face][row] followed by 1024 mantissa bytes
 *   [face][row][16]; face f covers tile rows 16*(f/2).. and tile channels
 *   16*(f%2)..; the 16 channels of one face row (one token) share an exponent.
 * Keys leave the prefill side with rotary pairs (2i, 2i+1); the decode side
 * pairs (i, i + D/2).  With rope_reorder set, source channel c lands at c/2
 * (c even) or D/2 + c/2 (c odd); values are untouched.
 * Pool `pool` of the source starts src_pool_stride_bytes after pool 0; its
 * shards follow each other.  Token p of the request (p < n_tokens) lands in
 * slot p % P of page dst_pages[p / P] of BF16 pool `pool`, KV head t*Hs + h. */
void ora_rebuild_tiled(const uint8_t *src, int64_t src_pool_stride_bytes, int32_t n_pools,
                       int32_t n_shards, int32_t n_tokens, int32_t num_kv_heads, int32_t head_dim,
                       int32_t page_size, int32_t rope_reorder, uint16_t *dst,
                       const int32_t *dst_pages, int64_t dst_pool_stride_pages)
{
    const int32_t hs = num_kv_heads / n_shards;
    const int32_t token_tiles = (n_tokens + 31) / 32;
    const int32_t chan_tiles = head_dim / 32;
    const int64_t tile_bytes = 64 + 32 * 32;
    const int64_t shard_bytes = (int64_t)hs * token_tiles * chan_tiles * tile_bytes;
    #pragma omp parallel for collapse(3) schedule(static)
    for (int32_t pool = 0; pool < n_pools; pool++)
        for (int32_t t = 0; t < n_shards; t++)
            for (int32_t h = 0; h < hs; h++)
                for (int32_t p = 0; p < n_tokens; p++)
                    for (int32_t c = 0; c < head_dim; c++) {
                        const int64_t tile_index = ((int64_t)h * token_tiles + p / 32) * chan_tiles + c / 32;
                        const uint8_t *tile = src + pool * src_pool_stride_bytes + t * shard_bytes
                                              + tile_index * tile_bytes;
                        const int rr = p % 32, cc = c % 32;
                        const int face = (rr / 16) * 2 + cc / 16;
                        const uint8_t E = tile[face * 16 + rr % 16];
                        const uint8_t byte = tile[64 + face * 256 + (rr % 16) * 16 + cc % 16];
                        const int c_out = rope_reorder ? (c % 2 == 0 ? c / 2 : head_dim / 2 + c / 2) : c;
                        const int64_t page = pool * dst_pool_stride_pages + dst_pages[p / page_size];
                        const int64_t row = (page * num_kv_heads + (int64_t)t * hs + h) * page_size + p % page_size;
                        dst[row * head_dim + c_out] = ora_bfp8_decode_value(E, byte);
                    }
}

/* Tiled shards -> BFP8 pages, bytes unchanged: the layout half of the pass
 * above, for a decoder that keeps the raw BFP8 pages and decodes them inside
 * attention [Sec. 3.3].  Keys keep the interleaved rotary order (a 16-channel
 * block cannot be relabelled without re-encoding); attention accounts for it
 * (key_order).  Token p goes to slot p % P of page dst_pages[p / P] of pool
 * `pool` (mantissa pool [pages][Hkv][P][D], exponent pool [pages][Hkv][P][D/16]). */
void ora_pack_tiled(const uint8_t *src, int64_t src_pool_stride_bytes, int32_t n_pools,
                    int32_t n_shards, int32_t n_tokens, int32_t num_kv_heads, int32_t head_dim,
                    int32_t page_size, uint8_t *dst_mant, uint8_t *dst_exp,
                    const int32_t *dst_pages, int64_t dst_pool_stride_pages)
{
    const int32_t hs = num_kv_heads / n_shards;
    const int32_t token_tiles = (n_tokens + 31) / 32;
    const int32_t chan_tiles = head_dim / 32;
    const int64_t tile_bytes = 64 + 32 * 32;
    const int64_t shard_bytes = (int64_t)hs * token_tiles * chan_tiles * tile_bytes;
    for (int32_t pool = 0; pool < n_pools; pool++)
        for (int32_t t = 0; t < n_shards; t++)
            for (int32_t h = 0; h < hs; h++)
                for (int32_t p = 0; p < n_tokens; p++) {
                    const int64_t page = pool * dst_pool_stride_pages + dst_pages[p / page_size];
                    const int64_t row = (page * num_kv_heads + (int64_t)t * hs + h) * page_size + p % page_size;
                    for (int32_t c = 0; c < head_dim; c++) {
                        const int64_t tile_index = ((int64_t)h * token_tiles + p / 32) * chan_tiles + c / 32;
                        const uint8_t *tile = src + pool * src_pool_stride_bytes + t * shard_bytes
                                              + tile_index * tile_bytes;
                        const int rr = p % 32, cc = c % 32;
                        const int face = (rr / 16) * 2 + cc / 16;
                        dst_mant[row * head_dim + c] = tile[64 + face * 256 + (rr % 16) * 16 + cc % 16];
                        if (c % ORA_BLOCK == 0)
                            dst_exp[row * (head_dim / ORA_BLOCK) + c / ORA_BLOCK] = tile[face * 16 + rr % 16];
                    }
                }
}

/* ----------------------------------------------------- paged attention */

typedef struct {
    const uint8_t *k_mant, *k_exp, *v_mant, *v_exp;
    const uint16_t *k_bf16, *v_bf16;
    const int32_t *page_table;
    int32_t max_pages_per_seq, num_kv_heads, head_dim, page_size;
    int32_t key_order;   /* 1: K rows stored in the interleaved rotary order */
} ora_kv;

/* Gather one K or V row of logical token t of sequence b, kv head j, into
 * row[head_dim] as float64 [Sec. 3.3: BFP8 pages decoded on read, BF16 pages
 * read as stored].  With key_order set, K rows are stored as the prefill side
 * leaves them (rotary pairs (2i, 2i+1)) and are relabelled into the
 * half-split order of the queries (pairs (i, i + D/2)) [Sec. 3.3: post-RoPE
 * key re-layout]: stored channel 2i is key channel i, 2i+1 is D/2 + i. */
static void ora_gather_row_stored(const ora_kv *kv, int is_v, int b, int j, int t, double *row);

static void ora_gather_row(const ora_kv *kv, int is_v, int b, int j, int t, double *row)
{
    if (is_v || !kv->key_order) {
        ora_gather_row_stored(kv, is_v, b, j, t, row);
        return;
    }
    const int D = kv->head_dim;
    double stored[D];
    ora_gather_row_stored(kv, is_v, b, j, t, stored);
    for (int i = 0; i < D / 2; i++) {
        row[i] = stored[2 * i];
        row[D / 2 + i] = stored[2 * i + 1];
    }
}

static void ora_gather_row_stored(const ora_kv *kv, int is_v, int b, int j, int t, double *row)
{
    int32_t entry = kv->page_table[(int64_t)b * kv->max_pages_per_seq + t / kv->page_size];
    int slot = t % kv->page_size;
    int64_t id = entry & ORA_ID_MASK;
    int64_t tok = (id * kv->num_kv_heads + j) * kv->page_size + slot;
    if (entry & ORA_TAG_BF16) {
        const uint16_t *src = (is_v ? kv->v_bf16 : kv->k_bf16) + tok * kv->head_dim;
        for (int d = 0; d < kv->head_dim; d++)
            row[d] = ora_bf16_to_f64(src[d]);
    } else {
        const uint8_t *mant = (is_v ? kv->v_mant : kv->k_mant) + tok * kv->head_dim;
        const uint8_t *ex = (is_v ? kv->v_exp : kv->k_exp) + tok * (kv->head_dim / ORA_BLOCK);
        for (int d = 0; d < kv->head_dim; d++)
            row[d] = ora_bf16_to_f64(ora_bfp8_decode_value(ex[d / ORA_BLOCK], mant[d]));
    }
}

/* Softmax attention of one query row over tokens [t0, t1) of sequence b,
 * kv head j, in float64:
 *   s_t = scale * <q, k_t>,  m = max_t s_t,  w_t = exp(s_t - m),
 *   l = sum_t w_t,  o = sum_t w_t v_t / l.
 * An empty range gives m = -inf, l = 0, o = 0.  Returns nothing; writes
 * (*m_out, *l_out, o[head_dim]). */
static void ora_attend_range(const ora_kv *kv, const uint16_t *q, double scale,
                             int b, int j, int t0, int t1,
                             double *m_out, double *l_out, double *o, double *scores, double *row)
{
    const int D = kv->head_dim;
    for (int d = 0; d < D; d++)
        o[d] = 0.0;
    if (t1 <= t0) {
        *m_out = -INFINITY;
        *l_out = 0.0;
        return;
    }
    double m = -INFINITY;
    for (int t = t0; t < t1; t++) {
        ora_gather_row(kv, 0, b, j, t, row);
        double s = 0.0;
        for (int d = 0; d < D; d++)
            s += ora_bf16_to_f64(q[d]) * row[d];
        s *= scale;
        scores[t - t0] = s;
        if (s > m)
            m = s;
    }
    double l = 0.0;
    for (int t = t0; t < t1; t++) {
        double w = exp(scores[t - t0] - m);
        l += w;
        ora_gather_row(kv, 1, b, j, t, row);
        for (int d = 0; d < D; d++)
            o[d] += w * row[d];
    }
    for (int d = 0; d < D; d++)
        o[d] /= l;
    *m_out = m;
    *l_out = l;
}

/* Log-sum-exp merge of n partials (m_s, l_s, o_s[D]) of one query row:
 *   M = max_s m_s,  w_s = l_s e^(m_s - M),  o = sum_s w_s o_s / sum_s w_s,
 *   lse = M + ln sum_s w_s.
 * Partials with l_s = 0 (empty ranges) are skipped; if all are empty the
 * result is o = 0, lse = -inf. */
void ora_merge_partials(int32_t n, const double *m, const double *l, const double *o, int32_t head_dim,
                        double *out, double *lse)
{
    double M = -INFINITY;
    for (int s = 0; s < n; s++)
        if (l[s] > 0.0 && m[s] > M)
            M = m[s];
    for (int d = 0; d < head_dim; d++)
        out[d] = 0.0;
    if (M == -INFINITY) {
        *lse = -INFINITY;
        return;
    }
    double W = 0.0;
    for (int s = 0; s < n; s++) {
        if (!(l[s] > 0.0))
            continue;
        double w = l[s] * exp(m[s] - M);
        W += w;
        for (int d = 0; d < head_dim; d++)
            out[d] += w * o[(int64_t)s * head_dim + d];
    }
    for (int d = 0; d < head_dim; d++)
        out[d] /= W;
    *lse = M + log(W);
}

/* Single-token GQA decode attention over the paged, mixed-format KV cache.
 *   q [B][Hq][D] BF16, out [B][Hq][D] float64, lse [B][Hq] float64 (natural log).
 * Query head h reads kv head floor(h / (Hq/Hkv)).  Sequence b attends to its
 * logical tokens [0, context_lens[b]); context 0 gives out = 0, lse = -inf.
 * The scale is applied to the float64 dot product.  Returns 0, or -1 on a bad
 * argument. */
int ora_decode_attn(const uint16_t *q,
                    const uint8_t *k_mant, const uint8_t *k_exp, const uint8_t *v_mant, const uint8_t *v_exp,
                    const uint16_t *k_bf16, const uint16_t *v_bf16,
                    const int32_t *page_table, int32_t max_pages_per_seq, const int32_t *context_lens,
                    int32_t batch, int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                    int32_t page_size, double scale, int32_t key_order, double *out, double *lse)
{
    if (num_kv_heads <= 0 || num_q_heads % num_kv_heads != 0 || head_dim % ORA_BLOCK != 0)
        return -1;
    ora_kv kv = {k_mant, k_exp, v_mant, v_exp, k_bf16, v_bf16, page_table,
                 max_pages_per_seq, num_kv_heads, head_dim, page_size, key_order};
    const int g = num_q_heads / num_kv_heads;
    int max_ctx = 0;
    for (int b = 0; b < batch; b++)
        if (context_lens[b] > max_ctx)
            max_ctx = context_lens[b];
    int bad = 0;
    #pragma omp parallel
    {
        double *scores = (double *)malloc(sizeof(double) * (size_t)(max_ctx > 0 ? max_ctx : 1));
        double *row = (double *)malloc(sizeof(double) * (size_t)head_dim);
        if (!scores || !row) {
            #pragma omp atomic write
            bad = 1;
        } else {
            #pragma omp for collapse(2) schedule(dynamic)
            for (int b = 0; b < batch; b++)
                for (int h = 0; h < num_q_heads; h++) {
                    int64_t qo = ((int64_t)b * num_q_heads + h) * head_dim;
                    double m, l;
                    ora_attend_range(&kv, q + qo, scale, b, h / g, 0, context_lens[b],
                                     &m, &l, out + qo, scores, row);
                    lse[(int64_t)b * num_q_heads + h] = (l > 0.0) ? m + log(l) : -INFINITY;
                }
        }
        free(scores);
        free(row);
    }
    return bad ? -1 : 0;
}

/* Split reference: for one (b, h), attend each contiguous range
 * [bounds[s], bounds[s+1]) separately, then merge with ora_merge_partials.
 * bounds has n_splits + 1 nondecreasing entries from 0 to context_lens[b].
 * Also returns the per-split partials (m, l, o) so a test can inspect them.
 * Returns 0, or -1 on a bad partition or allocation failure. */
int ora_decode_attn_split_one(const uint16_t *q,
                              const uint8_t *k_mant, const uint8_t *k_exp, const uint8_t *v_mant,
                              const uint8_t *v_exp, const uint16_t *k_bf16, const uint16_t *v_bf16,
                              const int32_t *page_table, int32_t max_pages_per_seq,
                              const int32_t *context_lens, int32_t num_q_heads, int32_t num_kv_heads,
                              int32_t head_dim, int32_t page_size, double scale, int32_t b, int32_t h,
                              const int32_t *bounds, int32_t n_splits,
                              double *part_m, double *part_l, double *part_o, double *out, double *lse)
{
    if (n_splits < 1 || bounds[0] != 0 || bounds[n_splits] != context_lens[b])
        return -1;
    for (int s = 0; s < n_splits; s++)
        if (bounds[s + 1] < bounds[s])
            return -1;
    ora_kv kv = {k_mant, k_exp, v_mant, v_exp, k_bf16, v_bf16, page_table,
                 max_pages_per_seq, num_kv_heads, head_dim, page_size, 0};
    const int g = num_q_heads / num_kv_heads;
    int ctx = context_lens[b];
    double *scores = (double *)malloc(sizeof(double) * (size_t)(ctx > 0 ? ctx : 1));
    double *row = (double *)malloc(sizeof(double) * (size_t)head_dim);
    if (!scores || !row) {
        free(scores);
        free(row);
        return -1;
    }
    const uint16_t *qr = q + ((int64_t)b * num_q_heads + h) * head_dim;
    for (int s = 0; s < n_splits; s++)
        ora_attend_range(&kv, qr, scale, b, h / g, bounds[s], bounds[s + 1],
                         &part_m[s], &part_l[s], part_o + (int64_t)s * head_dim, scores, row);
    ora_merge_partials(n_splits, part_m, part_l, part_o, head_dim, out, lse);
    free(scores);
    free(row);
    return 0;
}
