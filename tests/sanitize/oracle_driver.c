/* Memory- and UB-sanitizer driver for the oracle (test infrastructure).
 *
 * Built by tests/test_oracle_sanitize.py with -fsanitize=address,undefined
 * and run as a plain process: every oracle entry point is called on buffers
 * of exactly the size its contract names (so any read or write past them is
 * reported), on random contents and ragged shapes.  Also checks that the two
 * independent decoders agree on every (exponent, byte) pair. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

uint16_t ora_bfp8_decode_value(uint8_t E, uint8_t byte);
uint16_t ora_bfp8_decode_bits(uint8_t E, uint8_t byte);
int ora_bfp8_encode_blocks(const uint16_t *x, int64_t n_blocks, uint8_t *bytes, uint8_t *exps);
void ora_bfp8_decode_blocks(const uint8_t *bytes, const uint8_t *exps, int64_t n_blocks, uint16_t *out);
void ora_dequant_pages(const uint8_t *src_mant, const uint8_t *src_exp, uint16_t *dst,
                       const int32_t *src_pages, const int32_t *dst_pages, int32_t n_pages,
                       int32_t n_pools, int64_t src_pool_stride_pages, int64_t dst_pool_stride_pages,
                       int32_t num_kv_heads, int32_t head_dim, int32_t page_size);
void ora_rebuild_tiled(const uint8_t *src, int64_t src_pool_stride_bytes, int32_t n_pools,
                       int32_t n_shards, int32_t n_tokens, int32_t num_kv_heads, int32_t head_dim,
                       int32_t page_size, int32_t rope_reorder, uint16_t *dst,
                       const int32_t *dst_pages, int64_t dst_pool_stride_pages);
void ora_pack_tiled(const uint8_t *src, int64_t src_pool_stride_bytes, int32_t n_pools,
                    int32_t n_shards, int32_t n_tokens, int32_t num_kv_heads, int32_t head_dim,
                    int32_t page_size, uint8_t *dst_mant, uint8_t *dst_exp,
                    const int32_t *dst_pages, int64_t dst_pool_stride_pages);
int ora_decode_attn(const uint16_t *q, const uint8_t *k_mant, const uint8_t *k_exp,
                    const uint8_t *v_mant, const uint8_t *v_exp, const uint16_t *k_bf16,
                    const uint16_t *v_bf16, const int32_t *page_table, int32_t max_pages_per_seq,
                    const int32_t *context_lens, int32_t batch, int32_t num_q_heads, int32_t num_kv_heads,
                    int32_t head_dim, int32_t page_size, double scale, int32_t key_order, double *out,
                    double *lse);
int ora_decode_attn_split_one(const uint16_t *q, const uint8_t *k_mant, const uint8_t *k_exp,
                              const uint8_t *v_mant, const uint8_t *v_exp, const uint16_t *k_bf16,
                              const uint16_t *v_bf16, const int32_t *page_table, int32_t max_pages_per_seq,
                              const int32_t *context_lens, int32_t num_q_heads, int32_t num_kv_heads,
                              int32_t head_dim, int32_t page_size, double scale, int32_t b, int32_t h,
                              const int32_t *bounds, int32_t n_splits, double *part_m, double *part_l,
                              double *part_o, double *out, double *lse);

enum { D = 128, P = 16 };

static uint64_t state = 0x9E3779B97F4A7C15ull;
static uint32_t rnd(void)
{
    state ^= state << 13;
    state ^= state >> 7;
    state ^= state << 17;
    return (uint32_t)(state >> 16);
}

static void *alloc_rand(size_t n)
{
    uint8_t *p = (uint8_t *)malloc(n ? n : 1);
    for (size_t i = 0; i < n; i++)
        p[i] = (uint8_t)rnd();
    return p;
}

/* a shuffled list of n distinct ids drawn from [0, range) */
static int32_t *distinct_ids(int n, int range)
{
    int32_t *all = (int32_t *)malloc(sizeof(int32_t) * (size_t)range);
    for (int i = 0; i < range; i++)
        all[i] = i;
    for (int i = range - 1; i > 0; i--) {
        const int k = (int)(rnd() % (uint32_t)(i + 1));
        const int32_t t = all[i];
        all[i] = all[k];
        all[k] = t;
    }
    int32_t *ids = (int32_t *)malloc(sizeof(int32_t) * (size_t)(n ? n : 1));
    memcpy(ids, all, sizeof(int32_t) * (size_t)n);
    free(all);
    return ids;
}

static int check_decoders(void)
{
    for (int E = 0; E < 256; E++)
        for (int b = 0; b < 256; b++)
            if (ora_bfp8_decode_value((uint8_t)E, (uint8_t)b) != ora_bfp8_decode_bits((uint8_t)E, (uint8_t)b)) {
                printf("decoders disagree at E=%d byte=%d\n", E, b);
                return 1;
            }
    return 0;
}

static void run_codec(void)
{
    const int64_t nb = 333;
    uint16_t *x = (uint16_t *)malloc(sizeof(uint16_t) * (size_t)(nb * 16));
    for (int64_t i = 0; i < nb * 16; i++)     /* finite BF16 patterns */
        x[i] = (uint16_t)(rnd() & 0x7F7F) | (uint16_t)(rnd() & 0x8000);
    uint8_t *bytes = (uint8_t *)malloc((size_t)(nb * 16));
    uint8_t *exps = (uint8_t *)malloc((size_t)nb);
    uint16_t *back = (uint16_t *)malloc(sizeof(uint16_t) * (size_t)(nb * 16));
    ora_bfp8_encode_blocks(x, nb, bytes, exps);
    ora_bfp8_decode_blocks(bytes, exps, nb, back);
    free(x); free(bytes); free(exps); free(back);
}

static void run_dequant(void)
{
    const int hkv = 3, pages = 11, n = 7, pools = 3, dst_pages = 13;
    const size_t pe = (size_t)hkv * P * D;
    uint8_t *mant = (uint8_t *)alloc_rand((size_t)pools * pages * pe);
    uint8_t *ex = (uint8_t *)alloc_rand((size_t)pools * pages * pe / 16);
    uint16_t *dst = (uint16_t *)calloc((size_t)pools * dst_pages * pe, sizeof(uint16_t));
    int32_t *src_ids = distinct_ids(n, pages), *dst_ids = distinct_ids(n, dst_pages);
    ora_dequant_pages(mant, ex, dst, src_ids, dst_ids, n, pools, pages, dst_pages, hkv, D, P);
    free(mant); free(ex); free(dst); free(src_ids); free(dst_ids);
}

static void run_tiled(int n_tokens, int n_shards, int hkv)
{
    const int pools = 2, hs = hkv / n_shards, ttiles = (n_tokens + 31) / 32;
    const size_t shard = (size_t)hs * ttiles * (D / 32) * 1088;
    const size_t stride = shard * n_shards + 32;
    uint8_t *src = (uint8_t *)alloc_rand(stride * (pools - 1) + shard * n_shards);
    const int n_req = (n_tokens + P - 1) / P, pool_pages = n_req + 3;
    int32_t *ids = distinct_ids(n_req, pool_pages);
    uint16_t *dst = (uint16_t *)calloc((size_t)pools * pool_pages * hkv * P * D, sizeof(uint16_t));
    uint8_t *dm = (uint8_t *)calloc((size_t)pools * pool_pages * hkv * P * D, 1);
    uint8_t *de = (uint8_t *)calloc((size_t)pools * pool_pages * hkv * P * D / 16, 1);
    for (int rope = 0; rope < 2; rope++)
        ora_rebuild_tiled(src, (int64_t)stride, pools, n_shards, n_tokens, hkv, D, P, rope, dst, ids, pool_pages);
    ora_pack_tiled(src, (int64_t)stride, pools, n_shards, n_tokens, hkv, D, P, dm, de, ids, pool_pages);
    free(src); free(ids); free(dst); free(dm); free(de);
}

static int run_attention(void)
{
    const int B = 5, hkv = 2, g = 3, hq = hkv * g;
    const int ctx[5] = {0, 1, 17, 100, 33};
    int maxp = 0, total = 0;
    for (int b = 0; b < B; b++) {
        const int np = (ctx[b] + P - 1) / P;
        total += np;
        if (np > maxp)
            maxp = np;
    }
    const size_t pe = (size_t)hkv * P * D;
    uint8_t *km = (uint8_t *)alloc_rand((size_t)total * pe), *vm = (uint8_t *)alloc_rand((size_t)total * pe);
    uint8_t *ke = (uint8_t *)malloc((size_t)total * pe / 16), *ve = (uint8_t *)malloc((size_t)total * pe / 16);
    for (size_t i = 0; i < (size_t)total * pe / 16; i++) {
        ke[i] = (uint8_t)(120 + rnd() % 12);
        ve[i] = (uint8_t)(120 + rnd() % 12);
    }
    uint16_t *kb = (uint16_t *)malloc(sizeof(uint16_t) * (size_t)total * pe);
    uint16_t *vb = (uint16_t *)malloc(sizeof(uint16_t) * (size_t)total * pe);
    for (size_t i = 0; i < (size_t)total * pe; i++) {
        kb[i] = (uint16_t)(rnd() & 0x3FFF);
        vb[i] = (uint16_t)(rnd() & 0x3FFF);
    }
    int32_t *perm = distinct_ids(total, total);
    int32_t *pt = (int32_t *)calloc((size_t)B * (maxp ? maxp : 1), sizeof(int32_t));
    int at = 0;
    for (int b = 0; b < B; b++)
        for (int i = 0; i < (ctx[b] + P - 1) / P; i++)
            pt[b * maxp + i] = perm[at++] | ((rnd() & 1) ? 0x40000000 : 0);
    uint16_t *q = (uint16_t *)malloc(sizeof(uint16_t) * (size_t)B * hq * D);
    for (int i = 0; i < B * hq * D; i++)
        q[i] = (uint16_t)(rnd() & 0x3FFF);
    double *out = (double *)malloc(sizeof(double) * (size_t)B * hq * D);
    double *lse = (double *)malloc(sizeof(double) * (size_t)B * hq);
    int rc = 0;
    for (int ko = 0; ko < 2; ko++)
        rc |= ora_decode_attn(q, km, ke, vm, ve, kb, vb, pt, maxp, ctx, B, hq, hkv, D, P, 0.0883883, ko, out, lse);
    const int bounds[4] = {0, 16, 48, 100};
    double pm[3], pl[3], po[3 * D], o[D], l1;
    rc |= ora_decode_attn_split_one(q, km, ke, vm, ve, kb, vb, pt, maxp, ctx, hq, hkv, D, P, 0.0883883, 3, 4,
                                    bounds, 3, pm, pl, po, o, &l1);
    free(km); free(vm); free(ke); free(ve); free(kb); free(vb); free(perm); free(pt); free(q);
    free(out); free(lse);
    return rc;
}

int main(void)
{
    if (check_decoders())
        return 1;
    run_codec();
    run_dequant();
    run_tiled(1, 1, 8);
    run_tiled(70, 2, 4);
    run_tiled(129, 4, 8);
    if (run_attention()) {
        printf("attention returned an error\n");
        return 1;
    }
    printf("oracle sanitizer run ok\n");
    return 0;
}
