// hma_api.cpp -- the exported C ABI of libhma (declared in include/hma.h).
//
// Every argument is validated on the host before any HIP call, so a rejected
// call enqueues nothing and the checks can run on a machine without a GPU.
#include "hma.h"

#include <limits.h>
#include <stdint.h>

#include <algorithm>

#include "hma_internal.h"

namespace {

constexpr int32_t kSupportedHeadDim = 128;
constexpr int32_t kSupportedPageSize = 16;
constexpr int32_t kMaxGroup = 16;            // query heads per KV head (MFMA N = 16)
constexpr int32_t kSplitQuantum = 16;        // splits hold whole pages
constexpr int32_t kAutoSplitQuantum = 32;
constexpr int64_t kComputeUnits = 256;       // MI355X
// 4-wave workgroups: two per CU already give a CU the eight waves it needs to
// stream at full rate (three fit and take up the splits beyond)
constexpr int64_t kTargetWorkgroups = 2 * kComputeUnits;
constexpr int32_t kMinAutoSplit = 256;
constexpr int32_t kMaxAutoSplit = 2048;
constexpr int32_t kMaxWideSplit = 8192;

constexpr int32_t kSupportedBlock = 16;       // channels per shared exponent

bool aligned(const void *p, uintptr_t a)
{
    return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0;
}

// [a, a + na) and [b, b + nb) share a byte
bool overlaps(const void *a, int64_t na, const void *b, int64_t nb)
{
    const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
    return na > 0 && nb > 0 && x < y + (uintptr_t)nb && y < x + (uintptr_t)na;
}

int32_t round_up(int64_t x, int32_t q)
{
    return (int32_t)(((x + q - 1) / q) * q);
}

bool attn_sizes_ok(int32_t batch, int32_t hq, int32_t hkv, int32_t max_ctx)
{
    return batch >= 0 && hq > 0 && hkv > 0 && hq % hkv == 0 && max_ctx >= 0;
}

int32_t splits_for(int32_t max_ctx, int32_t tps);

// Split length for tokens_per_split = 0.  When every (sequence, KV head) pair
// fits in one pass of one workgroup per CU, the splits are sized for exactly
// that (8-wave workgroups); otherwise they target two 4-wave workgroups per
// CU, from the longest length (the host's only length information).
int32_t auto_tokens_per_split(int32_t batch, int32_t hkv, int32_t max_ctx)
{
    const int64_t pairs = (int64_t)batch * hkv;
    const int32_t whole = round_up(max_ctx > 0 ? max_ctx : 1, kSplitQuantum);
    int64_t wide = (pairs * (int64_t)max_ctx + kComputeUnits - 1) / kComputeUnits;
    wide = round_up(wide, kAutoSplitQuantum);
    if (wide < kMinAutoSplit)
        wide = kMinAutoSplit;
    if (wide > whole)
        wide = whole;
    if (wide <= kMaxWideSplit && pairs * splits_for(max_ctx, (int32_t)wide) <= kComputeUnits)
        return (int32_t)wide;
    int64_t tps = (pairs * (int64_t)max_ctx + kTargetWorkgroups - 1) / kTargetWorkgroups;
    tps = round_up(tps, kAutoSplitQuantum);
    if (tps < kMinAutoSplit)
        tps = kMinAutoSplit;
    if (tps > kMaxAutoSplit)
        tps = kMaxAutoSplit;
    if (tps > whole)
        tps = whole;
    return (int32_t)tps;
}

// Waves per workgroup for a grid of `blocks` workgroups: 8 (one workgroup per
// CU) when the grid fits in one pass over the CUs, else 4.
int32_t waves_for(int64_t blocks)
{
    return blocks <= kComputeUnits ? 8 : 4;
}

int32_t splits_for(int32_t max_ctx, int32_t tps)
{
    return max_ctx <= 0 ? 1 : (int32_t)(((int64_t)max_ctx + tps - 1) / tps);
}

int dequant_checked(const uint8_t *src_mant, const uint8_t *src_exp, uint16_t *dst_bf16,
                    const int32_t *src_pages, const int32_t *dst_pages, int32_t n_pages,
                    int32_t n_pools, int64_t src_pool_stride_pages, int64_t dst_pool_stride_pages,
                    int32_t num_kv_heads, int32_t head_dim, int32_t page_size, void *stream,
                    bool naive)
{
    if (n_pages < 0 || n_pools < 0 || num_kv_heads <= 0)
        return HMA_EINVAL;
    if (head_dim != kSupportedHeadDim || page_size != kSupportedPageSize)
        return HMA_EUNSUPPORTED;
    if (n_pages == 0 || n_pools == 0)
        return HMA_OK;
    if (!src_mant || !src_exp || !dst_bf16)
        return HMA_EINVAL;
    if (!aligned(src_mant, 16) || !aligned(src_exp, 16) || !aligned(dst_bf16, 16))
        return HMA_EINVAL;
    if (n_pools > 1 && (src_pool_stride_pages < 1 || dst_pool_stride_pages < 1))
        return HMA_EINVAL;
    if (src_pool_stride_pages < 0 || dst_pool_stride_pages < 0)
        return HMA_EINVAL;
    // the destination must not overlap the sources over the span the host can
    // bound: pools 0 .. n_pools - 1 at their strides, n_pages pages each (the
    // pages an identity page list touches; explicit lists are the caller's
    // contract)
    {
        const int64_t tile = (int64_t)num_kv_heads * kSupportedPageSize * kSupportedHeadDim;
        const int64_t sp = n_pools > 1 ? (int64_t)(n_pools - 1) * src_pool_stride_pages + n_pages : n_pages;
        const int64_t dp = n_pools > 1 ? (int64_t)(n_pools - 1) * dst_pool_stride_pages + n_pages : n_pages;
        if (overlaps(dst_bf16, dp * tile * 2, src_mant, sp * tile) ||
            overlaps(dst_bf16, dp * tile * 2, src_exp, sp * tile / kSupportedBlock))
            return HMA_EINVAL;
    }
    const int64_t tiles = (int64_t)n_pools * n_pages * num_kv_heads;
    if (tiles / 4 + 1 > (int64_t)INT_MAX)
        return HMA_EINVAL;
    if (naive && (tiles * kSupportedPageSize * kSupportedHeadDim + 255) / 256 > (int64_t)INT_MAX)
        return HMA_EINVAL;
    const hipStream_t s = static_cast<hipStream_t>(stream);
    const int rc = naive ? hma::launch_bfp8_dequant_pages_naive(src_mant, src_exp, dst_bf16, src_pages,
                                                                dst_pages, n_pages, n_pools,
                                                                src_pool_stride_pages,
                                                                dst_pool_stride_pages, num_kv_heads, s)
                         : hma::launch_bfp8_dequant_pages(src_mant, src_exp, dst_bf16, src_pages,
                                                          dst_pages, n_pages, n_pools,
                                                          src_pool_stride_pages,
                                                          dst_pool_stride_pages, num_kv_heads, s);
    return rc == 0 ? HMA_OK : HMA_EHIP;
}

// Host-side decisions of one attention call, shared by the call itself, the
// workspace query and the no-allocation entry point.
struct AttnPlan {
    int32_t tps, n_splits, waves, planned, balanced, slots_per_head;
    int64_t slots;                            // partial slots (0: no merge)
    size_t ticket_bytes, ml_bytes, o_bytes;   // workspace regions, 256-byte multiples but the last
};

size_t align256(size_t x)
{
    return (x + 255) & ~(size_t)255;
}

// ---- vector-ALU comparison kernel: at most 8 query heads per KV head, one
// range length for the whole batch
constexpr int32_t kValuMaxGroup = 8;

bool valu_sizes_ok(int32_t batch, int32_t hq, int32_t hkv, int32_t max_ctx, int32_t tps)
{
    return attn_sizes_ok(batch, hq, hkv, max_ctx) && hq / hkv <= kValuMaxGroup && tps >= 0 &&
           tps % kSplitQuantum == 0 && tps <= hma::kMaxTokensPerSplit;
}

// Automatic range length: one workgroup per compute unit over the batch at
// max_ctx (the kernel's registers leave room for one 8-wave workgroup per
// CU), at most 4096 tokens per range so that a long sequence of a ragged
// batch is spread over several CUs.
constexpr int64_t kValuMaxAutoSplit = 4096;

int32_t valu_tokens_per_split(int32_t batch, int32_t hkv, int32_t max_ctx, int32_t tps)
{
    if (tps)
        return tps;
    const int64_t pairs = (int64_t)batch * hkv;
    const int64_t len = std::max(max_ctx, 1);
    int64_t t = pairs >= kComputeUnits ? len : (pairs * len + kComputeUnits - 1) / kComputeUnits;
    t = std::min(std::min(t, len), kValuMaxAutoSplit);
    return round_up(t, kSplitQuantum);
}

struct ValuPlan {
    int32_t tps, n_splits;
    size_t ml_bytes, o_bytes;
};

ValuPlan valu_plan(int32_t batch, int32_t hq, int32_t hkv, int32_t max_ctx, int32_t tokens_per_split)
{
    ValuPlan pl;
    pl.tps = valu_tokens_per_split(batch, hkv, max_ctx, tokens_per_split);
    pl.n_splits = splits_for(max_ctx, pl.tps);
    const size_t slots = (size_t)batch * hq * pl.n_splits;
    pl.ml_bytes = align256(slots * 2 * sizeof(float));
    pl.o_bytes = slots * kSupportedHeadDim * sizeof(float);
    return pl;
}

AttnPlan attn_plan(int32_t batch, int32_t hq, int32_t hkv, int32_t max_ctx, int32_t tokens_per_split)
{
    AttnPlan pl;
    const int64_t pairs = (int64_t)batch * hkv;
    pl.tps = tokens_per_split ? tokens_per_split : auto_tokens_per_split(batch, hkv, max_ctx);
    pl.n_splits = splits_for(max_ctx, pl.tps);
    pl.waves = waves_for(pairs * pl.n_splits);
    pl.planned = pl.waves == 4 && batch <= hma::kPlanMaxBatch && pl.n_splits < hma::kPlanMaxBatch;
    // with the automatic split, the 4-wave schedule cuts the batch's pages
    // into equal ranges on the device, one per wave (ragged batches balance
    // across CUs)
    pl.balanced = pl.planned && tokens_per_split == 0;
    pl.slots_per_head = 0;
    if (pl.balanced) {
        // ranges per KV head: at most the grid's share (one range per
        // wave), or the count of ranges of the largest size when the pages
        // outnumber that; piece (k, b) is slot k + b
        const int64_t max_pages = ((int64_t)max_ctx + kSupportedPageSize - 1) / kSupportedPageSize;
        const int64_t by_grid = (hma::kBalancedGridCap + hkv - 1) / hkv * hma::kBalancedWaves;
        const int64_t by_size = (batch * max_pages + hma::kMaxChunkPages - 1) / hma::kMaxChunkPages;
        pl.slots_per_head = (int32_t)(std::max(by_grid, by_size) + batch);
        pl.slots = (int64_t)hkv * pl.slots_per_head;
    } else {
        pl.slots = pl.n_splits > 1 ? pairs * pl.n_splits : 0;
    }
    const size_t g = (size_t)(hq / hkv);
    pl.ticket_bytes = pl.slots ? align256((size_t)pairs * sizeof(int32_t)) : 0;
    pl.ml_bytes = pl.slots ? align256((size_t)pl.slots * g * 2 * sizeof(float)) : 0;
    pl.o_bytes = pl.slots ? (size_t)pl.slots * g * kSupportedHeadDim * sizeof(float) : 0;
    return pl;
}

int64_t tiled_shard_bytes(int32_t n_tokens, int32_t heads_per_shard)
{
    return (int64_t)heads_per_shard * ((n_tokens + 31) / 32) * (kSupportedHeadDim / 32) * (64 + 32 * 32);
}

// Shared argument checks of the tiled-source entry points (HMA_OK also when
// there is nothing to do: the caller then returns without launching).
int tiled_check(const uint8_t *src, int64_t src_pool_stride_bytes, int32_t n_pools, int32_t n_shards,
                int32_t n_tokens, const void *dst_a, const void *dst_b, int64_t dst_pool_stride_pages,
                int32_t num_kv_heads, int32_t head_dim, int32_t page_size)
{
    if (n_pools < 0 || n_tokens < 0 || n_shards < 1 || num_kv_heads <= 0)
        return HMA_EINVAL;
    if (head_dim != kSupportedHeadDim || page_size != kSupportedPageSize)
        return HMA_EUNSUPPORTED;
    if (num_kv_heads % n_shards != 0)
        return HMA_EINVAL;
    if (n_pools == 0 || n_tokens == 0)
        return HMA_OK;
    if (!src || !dst_a || !dst_b || !aligned(src, 16) || !aligned(dst_a, 16) || !aligned(dst_b, 16))
        return HMA_EINVAL;
    const int64_t pool_bytes = (int64_t)n_shards * tiled_shard_bytes(n_tokens, num_kv_heads / n_shards);
    if (n_pools > 1 && (src_pool_stride_bytes < pool_bytes || src_pool_stride_bytes % 16 != 0))
        return HMA_EINVAL;
    if (n_pools > 1 && dst_pool_stride_pages < 1)
        return HMA_EINVAL;
    if (dst_pool_stride_pages < 0 || src_pool_stride_bytes < 0)
        return HMA_EINVAL;
    const int64_t units = (int64_t)n_pools * num_kv_heads * ((n_tokens + 31) / 32);
    if (units / 4 + 1 > (int64_t)INT_MAX)
        return HMA_EINVAL;
    return HMA_OK;
}

// Host-side validation of an attention call (no HIP call).
int attn_check(const uint16_t *q, const uint8_t *k_mant, const uint8_t *k_exp, const uint8_t *v_mant,
               const uint8_t *v_exp, const uint16_t *k_bf16, const uint16_t *v_bf16, const int32_t *page_table,
               int32_t max_pages_per_seq, const int32_t *context_lens, int32_t max_context_len, int32_t batch,
               int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim, int32_t page_size, float scale,
               int32_t key_order, int32_t tokens_per_split, const uint16_t *out, const float *lse)
{
    if (!attn_sizes_ok(batch, num_q_heads, num_kv_heads, max_context_len))
        return HMA_EINVAL;
    if (head_dim != kSupportedHeadDim || page_size != kSupportedPageSize)
        return HMA_EUNSUPPORTED;
    if (num_q_heads / num_kv_heads > kMaxGroup)
        return HMA_EUNSUPPORTED;
    if (tokens_per_split < 0 || tokens_per_split % kSplitQuantum != 0 ||
        tokens_per_split > hma::kMaxTokensPerSplit)
        return HMA_EINVAL;
    if (max_pages_per_seq < 0 || (int64_t)max_context_len > (int64_t)max_pages_per_seq * page_size)
        return HMA_EINVAL;
    if (!(scale == scale) || (key_order != 0 && key_order != 1))
        return HMA_EINVAL;
    if (batch == 0)
        return HMA_OK;
    if (!q || !k_mant || !k_exp || !v_mant || !v_exp || !page_table || !context_lens || !out)
        return HMA_EINVAL;
    if ((k_bf16 == nullptr) != (v_bf16 == nullptr))
        return HMA_EINVAL;
    if (!aligned(q, 16) || !aligned(out, 16) || !aligned(k_mant, 16) || !aligned(v_mant, 16) ||
        !aligned(k_exp, 16) || !aligned(v_exp, 16) || !aligned(k_bf16, 16) || !aligned(v_bf16, 16) ||
        !aligned(lse, 4))
        return HMA_EINVAL;
    const AttnPlan pl = attn_plan(batch, num_q_heads, num_kv_heads, max_context_len, tokens_per_split);
    if ((int64_t)batch * num_kv_heads * pl.n_splits > (int64_t)INT_MAX)
        return HMA_EINVAL;
    return HMA_OK;
}

// Launch with the tickets at `tickets` and the partials at `partials` (NULL
// when the plan needs none).
int attn_launch(const uint16_t *q, const uint8_t *k_mant, const uint8_t *k_exp, const uint8_t *v_mant,
                const uint8_t *v_exp, const uint16_t *k_bf16, const uint16_t *v_bf16, const int32_t *page_table,
                int32_t max_pages_per_seq, const int32_t *context_lens, int32_t max_context_len, int32_t batch,
                int32_t num_q_heads, int32_t num_kv_heads, float scale, int32_t key_order, const AttnPlan &pl,
                uint16_t *out, float *lse, uint8_t *tickets, uint8_t *partials, void *stream)
{
    hma::AttnLaunch a;
    a.q = q;
    a.k_mant = k_mant;
    a.k_exp = k_exp;
    a.v_mant = v_mant;
    a.v_exp = v_exp;
    a.k_bf16 = k_bf16;
    a.v_bf16 = v_bf16;
    a.page_table = page_table;
    a.ctx_lens = context_lens;
    a.out = out;
    a.lse = lse;
    a.tickets = pl.slots ? reinterpret_cast<int32_t *>(tickets) : nullptr;
    a.part_ml = pl.slots ? reinterpret_cast<float2 *>(partials) : nullptr;
    a.part_o = pl.slots ? reinterpret_cast<float *>(partials + pl.ml_bytes) : nullptr;
    a.max_pages = max_pages_per_seq;
    a.batch = batch;
    a.hq = num_q_heads;
    a.hkv = num_kv_heads;
    a.tps = pl.tps;
    a.n_splits = pl.n_splits;
    a.max_ctx = max_context_len;
    a.waves = pl.waves;
    a.planned = pl.planned;
    a.balanced = pl.balanced;
    a.slots_per_head = pl.slots_per_head;
    a.scale = scale;
    a.key_interleaved = key_order;
    return hma::launch_decode_attn(a, static_cast<hipStream_t>(stream)) == 0 ? HMA_OK : HMA_EHIP;
}

}  // namespace

extern "C" {

const char *hma_status_string(int status)
{
    switch (status) {
    case HMA_OK:
        return "ok";
    case HMA_EINVAL:
        return "invalid argument (null pointer, bad size, misalignment or aliasing)";
    case HMA_EUNSUPPORTED:
        return "unsupported configuration (head_dim must be 128, page_size 16, "
               "query heads per KV head at most 16)";
    case HMA_EWORKSPACE:
        return "workspace missing or too small";
    case HMA_EHIP:
        return "HIP launch or copy failed";
    case HMA_ESCRATCH:
        return "problem larger than the fixed device scratch of hma_decode_attn_bfp8_noalloc";
    default:
        return "unknown status";
    }
}

int hma_bfp8_dequant_pages(const uint8_t *src_mant, const uint8_t *src_exp, uint16_t *dst_bf16,
                           const int32_t *src_pages, const int32_t *dst_pages, int32_t n_pages,
                           int32_t n_pools, int64_t src_pool_stride_pages,
                           int64_t dst_pool_stride_pages, int32_t num_kv_heads,
                           int32_t head_dim, int32_t page_size, void *stream)
{
    return dequant_checked(src_mant, src_exp, dst_bf16, src_pages, dst_pages, n_pages, n_pools,
                           src_pool_stride_pages, dst_pool_stride_pages, num_kv_heads, head_dim,
                           page_size, stream, false);
}

int hma_bfp8_dequant_pages_naive(const uint8_t *src_mant, const uint8_t *src_exp, uint16_t *dst_bf16,
                                 const int32_t *src_pages, const int32_t *dst_pages, int32_t n_pages,
                                 int32_t n_pools, int64_t src_pool_stride_pages,
                                 int64_t dst_pool_stride_pages, int32_t num_kv_heads,
                                 int32_t head_dim, int32_t page_size, void *stream)
{
    return dequant_checked(src_mant, src_exp, dst_bf16, src_pages, dst_pages, n_pages, n_pools,
                           src_pool_stride_pages, dst_pool_stride_pages, num_kv_heads, head_dim,
                           page_size, stream, true);
}

int hma_ingress_rebuild(const uint8_t *host_mant, const uint8_t *host_exp, uint8_t *stage_mant,
                        uint8_t *stage_exp, uint16_t *dst_bf16, const int32_t *dst_pages,
                        int32_t n_pages, int32_t n_pools, int64_t dst_pool_stride_pages,
                        int32_t num_kv_heads, int32_t head_dim, int32_t page_size, void *stream)
{
    if (n_pages < 0 || n_pools < 0 || num_kv_heads <= 0)
        return HMA_EINVAL;
    if (head_dim != kSupportedHeadDim || page_size != kSupportedPageSize)
        return HMA_EUNSUPPORTED;
    if (n_pages == 0 || n_pools == 0)
        return HMA_OK;
    if (!host_mant || !host_exp || !stage_mant || !stage_exp || !dst_bf16)
        return HMA_EINVAL;
    if (!aligned(stage_mant, 16) || !aligned(stage_exp, 16) || !aligned(dst_bf16, 16))
        return HMA_EINVAL;
    if (n_pools > 1 && dst_pool_stride_pages < 1)
        return HMA_EINVAL;
    if (dst_pool_stride_pages < 0)
        return HMA_EINVAL;
    const int64_t tiles = (int64_t)n_pools * n_pages * num_kv_heads;
    if (tiles / 4 + 1 > (int64_t)INT_MAX)
        return HMA_EINVAL;
    const size_t mant_bytes = (size_t)tiles * kSupportedPageSize * kSupportedHeadDim;
    const size_t exp_bytes = mant_bytes / 16;
    // the two staging buffers must not overlap each other or start at the
    // destination (the destination's extent depends on device-side page ids)
    if (overlaps(stage_mant, (int64_t)mant_bytes, stage_exp, (int64_t)exp_bytes))
        return HMA_EINVAL;
    if ((const void *)dst_bf16 == (const void *)stage_mant || (const void *)dst_bf16 == (const void *)stage_exp)
        return HMA_EINVAL;
    const int rc = hma::launch_ingress_rebuild(host_mant, host_exp, stage_mant, stage_exp, dst_bf16, dst_pages,
                                               n_pages, n_pools, dst_pool_stride_pages, num_kv_heads,
                                               mant_bytes, exp_bytes, static_cast<hipStream_t>(stream));
    return rc == 0 ? HMA_OK : HMA_EHIP;
}

int64_t hma_tiled_shard_bytes(int32_t n_tokens, int32_t heads_per_shard, int32_t head_dim)
{
    if (n_tokens < 0 || heads_per_shard < 1 || head_dim != kSupportedHeadDim)
        return -1;
    return tiled_shard_bytes(n_tokens, heads_per_shard);
}

int hma_bfp8_rebuild_tiled(const uint8_t *src, int64_t src_pool_stride_bytes, int32_t n_pools,
                           int32_t n_shards, int32_t n_tokens, uint16_t *dst_bf16,
                           const int32_t *dst_pages, int64_t dst_pool_stride_pages,
                           int32_t num_kv_heads, int32_t head_dim, int32_t page_size,
                           int32_t rope_reorder, void *stream)
{
    if (rope_reorder != 0 && rope_reorder != 1)
        return HMA_EINVAL;
    const int st = tiled_check(src, src_pool_stride_bytes, n_pools, n_shards, n_tokens, dst_bf16, dst_bf16,
                               dst_pool_stride_pages, num_kv_heads, head_dim, page_size);
    if (st != HMA_OK || n_pools == 0 || n_tokens == 0)
        return st;
    const int rc = hma::launch_bfp8_rebuild_tiled(src, src_pool_stride_bytes, n_pools, n_shards, n_tokens,
                                                  dst_bf16, dst_pages, dst_pool_stride_pages, num_kv_heads,
                                                  rope_reorder, static_cast<hipStream_t>(stream));
    return rc == 0 ? HMA_OK : HMA_EHIP;
}

int hma_bfp8_pack_tiled(const uint8_t *src, int64_t src_pool_stride_bytes, int32_t n_pools,
                        int32_t n_shards, int32_t n_tokens, uint8_t *dst_mant, uint8_t *dst_exp,
                        const int32_t *dst_pages, int64_t dst_pool_stride_pages, int32_t num_kv_heads,
                        int32_t head_dim, int32_t page_size, void *stream)
{
    const int st = tiled_check(src, src_pool_stride_bytes, n_pools, n_shards, n_tokens, dst_mant, dst_exp,
                               dst_pool_stride_pages, num_kv_heads, head_dim, page_size);
    if (st != HMA_OK || n_pools == 0 || n_tokens == 0)
        return st;
    if (dst_mant == dst_exp)
        return HMA_EINVAL;
    const int rc = hma::launch_bfp8_pack_tiled(src, src_pool_stride_bytes, n_pools, n_shards, n_tokens, dst_mant,
                                               dst_exp, dst_pages, dst_pool_stride_pages, num_kv_heads,
                                               static_cast<hipStream_t>(stream));
    return rc == 0 ? HMA_OK : HMA_EHIP;
}

int32_t hma_decode_attn_tokens_per_split(int32_t batch, int32_t num_q_heads,
                                         int32_t num_kv_heads, int32_t max_context_len)
{
    if (!attn_sizes_ok(batch, num_q_heads, num_kv_heads, max_context_len))
        return 0;
    return auto_tokens_per_split(batch, num_kv_heads, max_context_len);
}

size_t hma_decode_attn_workspace_bytes(int32_t batch, int32_t num_q_heads, int32_t num_kv_heads,
                                       int32_t max_context_len, int32_t tokens_per_split)
{
    if (!attn_sizes_ok(batch, num_q_heads, num_kv_heads, max_context_len))
        return (size_t)-1;
    if (tokens_per_split < 0 || tokens_per_split % kSplitQuantum != 0 ||
        tokens_per_split > hma::kMaxTokensPerSplit)
        return (size_t)-1;
    const AttnPlan pl = attn_plan(batch, num_q_heads, num_kv_heads, max_context_len, tokens_per_split);
    return pl.ticket_bytes + pl.ml_bytes + pl.o_bytes;
}

int hma_decode_attn_bfp8(const uint16_t *q, const uint8_t *k_mant, const uint8_t *k_exp,
                         const uint8_t *v_mant, const uint8_t *v_exp, const uint16_t *k_bf16,
                         const uint16_t *v_bf16, const int32_t *page_table,
                         int32_t max_pages_per_seq, const int32_t *context_lens,
                         int32_t max_context_len, int32_t batch, int32_t num_q_heads,
                         int32_t num_kv_heads, int32_t head_dim, int32_t page_size, float scale,
                         int32_t key_order, int32_t tokens_per_split, uint16_t *out, float *lse,
                         void *workspace, size_t workspace_bytes, void *stream)
{
    const int st = attn_check(q, k_mant, k_exp, v_mant, v_exp, k_bf16, v_bf16, page_table, max_pages_per_seq,
                              context_lens, max_context_len, batch, num_q_heads, num_kv_heads, head_dim,
                              page_size, scale, key_order, tokens_per_split, out, lse);
    if (st != HMA_OK || batch == 0)
        return st;
    const AttnPlan pl = attn_plan(batch, num_q_heads, num_kv_heads, max_context_len, tokens_per_split);
    const size_t need = pl.ticket_bytes + pl.ml_bytes + pl.o_bytes;
    if (need > 0 && (workspace == nullptr || workspace_bytes < need))
        return HMA_EWORKSPACE;
    if (need > 0 && !aligned(workspace, 256))
        return HMA_EINVAL;
    uint8_t *ws = static_cast<uint8_t *>(workspace);
    return attn_launch(q, k_mant, k_exp, v_mant, v_exp, k_bf16, v_bf16, page_table, max_pages_per_seq,
                       context_lens, max_context_len, batch, num_q_heads, num_kv_heads, scale, key_order, pl,
                       out, lse, ws, ws + pl.ticket_bytes, stream);
}

int hma_decode_attn_bfp8_noalloc(const uint16_t *q, const uint8_t *k_mant, const uint8_t *k_exp,
                                 const uint8_t *v_mant, const uint8_t *v_exp, const uint16_t *k_bf16,
                                 const uint16_t *v_bf16, const int32_t *page_table,
                                 int32_t max_pages_per_seq, const int32_t *context_lens,
                                 int32_t max_context_len, int32_t batch, int32_t num_q_heads,
                                 int32_t num_kv_heads, int32_t head_dim, int32_t page_size, float scale,
                                 int32_t key_order, int32_t tokens_per_split, uint16_t *out, float *lse,
                                 void *stream)
{
    const int st = attn_check(q, k_mant, k_exp, v_mant, v_exp, k_bf16, v_bf16, page_table, max_pages_per_seq,
                              context_lens, max_context_len, batch, num_q_heads, num_kv_heads, head_dim,
                              page_size, scale, key_order, tokens_per_split, out, lse);
    if (st != HMA_OK || batch == 0)
        return st;
    const AttnPlan pl = attn_plan(batch, num_q_heads, num_kv_heads, max_context_len, tokens_per_split);
    // tickets sit in a fixed region of the scratch, the partials after it
    if (pl.ticket_bytes > hma::kScratchTicketBytes ||
        pl.ml_bytes + pl.o_bytes > hma::kScratchBytes - hma::kScratchTicketBytes)
        return HMA_ESCRATCH;
    const hipStream_t s = static_cast<hipStream_t>(stream);
    uint8_t *base = nullptr;
    if (pl.slots > 0 && hma::noalloc_scratch(s, &base) != 0)
        return HMA_EHIP;
    return attn_launch(q, k_mant, k_exp, v_mant, v_exp, k_bf16, v_bf16, page_table, max_pages_per_seq,
                       context_lens, max_context_len, batch, num_q_heads, num_kv_heads, scale, key_order, pl,
                       out, lse, base, base ? base + hma::kScratchTicketBytes : nullptr, stream);
}

int hma_validate_page_table(const int32_t *page_table, int32_t batch, int32_t max_pages_per_seq,
                            const int32_t *context_lens, int32_t max_context_len, int64_t num_bfp8_pages,
                            int64_t num_bf16_pages, int32_t page_size, int64_t *first_bad)
{
    if (first_bad)
        *first_bad = -1;
    if (batch < 0 || max_pages_per_seq < 0 || max_context_len < 0 || num_bfp8_pages < 0)
        return HMA_EINVAL;
    if (page_size != kSupportedPageSize)
        return HMA_EUNSUPPORTED;
    if ((int64_t)max_context_len > (int64_t)max_pages_per_seq * page_size)
        return HMA_EINVAL;
    if (batch == 0)
        return HMA_OK;
    if (!page_table || !context_lens)
        return HMA_EINVAL;
    for (int32_t b = 0; b < batch; b++) {
        // the entries the attention kernel reads for this sequence
        const int32_t ctx = std::min(std::max(context_lens[b], 0), max_context_len);
        const int32_t n = (ctx + page_size - 1) / page_size;
        for (int32_t i = 0; i < n; i++) {
            const int64_t at = (int64_t)b * max_pages_per_seq + i;
            const int32_t e = page_table[at];
            const int64_t id = e & HMA_PAGE_ID_MASK;
            const bool tagged = (e & HMA_PAGE_BF16) != 0 && num_bf16_pages >= 0;
            const bool ok = e >= 0 && id < (tagged ? num_bf16_pages : num_bfp8_pages);
            if (!ok) {
                if (first_bad)
                    *first_bad = at;
                return HMA_EINVAL;
            }
        }
    }
    return HMA_OK;
}

int hma_paged_read_probe(const uint8_t *k_mant, const uint8_t *k_exp, const uint8_t *v_mant, const uint8_t *v_exp,
                         const int32_t *page_table, int32_t max_pages_per_seq, const int32_t *context_lens,
                         int32_t max_context_len, int32_t batch, int32_t num_kv_heads,
                         int32_t heads_per_workgroup, int32_t pages_per_split, int32_t n_splits, uint32_t *sink,
                         size_t sink_words, void *stream)
{
    if (batch < 0 || num_kv_heads <= 0 || max_pages_per_seq < 0 || max_context_len < 0)
        return HMA_EINVAL;
    const int32_t hpw = heads_per_workgroup;
    if (!(hpw == 1 || hpw == 2 || hpw == 4 || hpw == 8) || num_kv_heads % hpw != 0)
        return HMA_EINVAL;
    if (pages_per_split < 1 || pages_per_split > hma::kMaxSplitPages || n_splits < 1)
        return HMA_EINVAL;
    if ((int64_t)n_splits * pages_per_split * kSupportedPageSize < max_context_len ||
        (int64_t)max_context_len > (int64_t)max_pages_per_seq * kSupportedPageSize)
        return HMA_EINVAL;
    const int64_t grid = (int64_t)batch * (num_kv_heads / hpw) * n_splits;
    if (grid > INT_MAX)
        return HMA_EINVAL;
    if (batch == 0)
        return HMA_OK;
    if (!k_mant || !k_exp || !v_mant || !v_exp || !page_table || !context_lens || !sink)
        return HMA_EINVAL;
    if (!aligned(k_mant, 16) || !aligned(k_exp, 16) || !aligned(v_mant, 16) || !aligned(v_exp, 16) ||
        !aligned(page_table, 4) || !aligned(context_lens, 4) || !aligned(sink, 4))
        return HMA_EINVAL;
    if (sink_words < (size_t)grid * 8)
        return HMA_EINVAL;
    return hma::launch_paged_read_probe(k_mant, k_exp, v_mant, v_exp, page_table, max_pages_per_seq,
                                        context_lens, max_context_len, batch, num_kv_heads, hpw,
                                        pages_per_split, n_splits, sink, static_cast<hipStream_t>(stream)) == 0
               ? HMA_OK
               : HMA_EHIP;
}

int hma_stream_read_probe(const void *buf, size_t bytes, int32_t n_workgroups, uint32_t *sink, size_t sink_words,
                          void *stream)
{
    if (!buf || !sink || !aligned(buf, 16) || !aligned(sink, 4))
        return HMA_EINVAL;
    if (bytes == 0 || bytes % 16 != 0 || n_workgroups < 1 || n_workgroups > (1 << 20))
        return HMA_EINVAL;
    if (sink_words < (size_t)n_workgroups * 4)
        return HMA_EINVAL;
    return hma::launch_stream_read_probe(buf, bytes, sink, n_workgroups, static_cast<hipStream_t>(stream)) == 0
               ? HMA_OK
               : HMA_EHIP;
}

int hma_issue_probe(int32_t valu_kind, int32_t valu_ops, int32_t with_mfma, int32_t waves_per_simd, int32_t iters,
                    uint64_t *cycles, size_t cycles_words, uint32_t *sink, size_t sink_words, void *stream)
{
    if (valu_kind < 0 || valu_kind > 4 || !(valu_ops == 0 || valu_ops == 8 || valu_ops == 16) ||
        (with_mfma != 0 && with_mfma != 1))
        return HMA_EINVAL;
    if (valu_ops == 0 && with_mfma == 0)
        return HMA_EINVAL;
    if (waves_per_simd < 1 || waves_per_simd > 4 || iters < 1 || iters > (1 << 20))
        return HMA_EINVAL;
    const int64_t n_waves = 4 * kComputeUnits * waves_per_simd;
    if (!cycles || !sink || !aligned(cycles, 8) || !aligned(sink, 4) || cycles_words < (size_t)n_waves ||
        sink_words < (size_t)n_waves * 64)
        return HMA_EINVAL;
    return hma::launch_issue_probe(valu_kind, valu_ops, with_mfma != 0, (int32_t)n_waves, iters, cycles, sink,
                                   static_cast<hipStream_t>(stream)) == 0
               ? HMA_OK
               : HMA_EHIP;
}

size_t hma_decode_attn_valu_workspace_bytes(int32_t batch, int32_t num_q_heads, int32_t num_kv_heads,
                                            int32_t max_context_len, int32_t tokens_per_split)
{
    if (!valu_sizes_ok(batch, num_q_heads, num_kv_heads, max_context_len, tokens_per_split))
        return (size_t)-1;
    if (batch == 0)
        return 0;
    const ValuPlan pl = valu_plan(batch, num_q_heads, num_kv_heads, max_context_len, tokens_per_split);
    return pl.ml_bytes + pl.o_bytes;
}

int hma_decode_attn_bfp8_valu(const uint16_t *q, const uint8_t *k_mant, const uint8_t *k_exp, const uint8_t *v_mant,
                              const uint8_t *v_exp, const int32_t *page_table, int32_t max_pages_per_seq,
                              const int32_t *context_lens, int32_t max_context_len, int32_t batch,
                              int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim, int32_t page_size,
                              float scale, int32_t tokens_per_split, uint16_t *out, float *lse, void *workspace,
                              size_t workspace_bytes, void *stream)
{
    const int st = attn_check(q, k_mant, k_exp, v_mant, v_exp, nullptr, nullptr, page_table, max_pages_per_seq,
                              context_lens, max_context_len, batch, num_q_heads, num_kv_heads, head_dim,
                              page_size, scale, 0, tokens_per_split, out, lse);
    if (st != HMA_OK)
        return st;
    if (num_q_heads / num_kv_heads > kValuMaxGroup)
        return HMA_EUNSUPPORTED;
    if (batch == 0)
        return HMA_OK;
    const ValuPlan pl = valu_plan(batch, num_q_heads, num_kv_heads, max_context_len, tokens_per_split);
    if ((int64_t)batch * num_kv_heads * pl.n_splits > (int64_t)INT_MAX)
        return HMA_EINVAL;
    if (workspace == nullptr || workspace_bytes < pl.ml_bytes + pl.o_bytes)
        return HMA_EWORKSPACE;
    if (!aligned(workspace, 256))
        return HMA_EINVAL;
    uint8_t *ws = static_cast<uint8_t *>(workspace);
    return hma::launch_decode_attn_valu(q, k_mant, k_exp, v_mant, v_exp, page_table, max_pages_per_seq,
                                        context_lens, max_context_len, batch, num_q_heads, num_kv_heads, scale,
                                        pl.tps, pl.n_splits, reinterpret_cast<float *>(ws),
                                        reinterpret_cast<float *>(ws + pl.ml_bytes), out, lse,
                                        static_cast<hipStream_t>(stream)) == 0
               ? HMA_OK
               : HMA_EHIP;
}

}  // extern "C"
