// hma_internal.h -- launchers behind the C ABI (not exported).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace hma {

// Longest split the attention kernel accepts: its page-table slice is staged
// in LDS (4 bytes per 16-token page).
constexpr int32_t kMaxTokensPerSplit = 16384;
constexpr int kMaxSplitPages = kMaxTokensPerSplit / 16;
// Largest batch, and bound on the splits per sequence, that the length-aware
// schedule handles (its tables sit in LDS); beyond them the direct schedule
// runs.
constexpr int kPlanMaxBatch = 1024;

// Returns 0 on a successful launch, -1 if the launch failed.  src_pages or
// dst_pages may be NULL (identity).
int launch_bfp8_dequant_pages(const uint8_t *src_mant, const uint8_t *src_exp, uint16_t *dst,
                              const int32_t *src_pages, const int32_t *dst_pages,
                              int32_t n_pages, int32_t n_pools, int64_t src_stride_pages,
                              int64_t dst_stride_pages, int32_t hkv, hipStream_t stream);

// One thread per element: the comparison baseline (same arguments and result).
int launch_bfp8_dequant_pages_naive(const uint8_t *src_mant, const uint8_t *src_exp, uint16_t *dst,
                                    const int32_t *src_pages, const int32_t *dst_pages,
                                    int32_t n_pages, int32_t n_pools, int64_t src_stride_pages,
                                    int64_t dst_stride_pages, int32_t hkv, hipStream_t stream);

// Tiled per-chip prefill shards -> BF16 pages (see rebuild_tiled.hip).
int launch_bfp8_rebuild_tiled(const uint8_t *src, int64_t src_pool_stride_bytes, int32_t n_pools,
                              int32_t n_shards, int32_t n_tokens, uint16_t *dst, const int32_t *dst_pages,
                              int64_t dst_stride_pages, int32_t hkv, int32_t rope_reorder,
                              hipStream_t stream);

// Tiled per-chip prefill shards -> BFP8 pages, bytes unchanged.
int launch_bfp8_pack_tiled(const uint8_t *src, int64_t src_pool_stride_bytes, int32_t n_pools, int32_t n_shards,
                           int32_t n_tokens, uint8_t *dst_mant, uint8_t *dst_exp, const int32_t *dst_pages,
                           int64_t dst_stride_pages, int32_t hkv, hipStream_t stream);

// Host -> device copy of the staged pages on `stream`, then their rebuild
// (src = staged page i, dst = dst_pages[i] or i when NULL).
int launch_ingress_rebuild(const uint8_t *host_mant, const uint8_t *host_exp, uint8_t *stage_mant,
                           uint8_t *stage_exp, uint16_t *dst, const int32_t *dst_pages, int32_t n_pages,
                           int32_t n_pools, int64_t dst_stride_pages, int32_t hkv, size_t mant_bytes,
                           size_t exp_bytes, hipStream_t stream);

// Largest grid of the page-balanced schedule (two workgroups per CU on the
// 256 CUs of an MI355X) and its waves per workgroup: they bound the page
// ranges per KV head (one per wave), hence the partial slots the host
// reserves.
constexpr int32_t kBalancedGridCap = 512;
constexpr int32_t kBalancedWaves = 4;
// Pages per range of the page-balanced schedule (the device clamps to these).
constexpr int32_t kMaxChunkPages = kMaxSplitPages;

struct AttnLaunch {
    const uint16_t *q;
    const uint8_t *k_mant, *k_exp, *v_mant, *v_exp;
    const uint16_t *k_bf16, *v_bf16;
    const int32_t *page_table;
    const int32_t *ctx_lens;
    uint16_t *out;
    float *lse;
    int32_t *tickets;       // one per (sequence, KV head): zero before the call, left zero
    float2 *part_ml;        // (max, sum) per partial slot and query head
    float *part_o;          // 128 weighted values per partial slot and query head
    int32_t max_pages, batch, hq, hkv, tps, n_splits;
    int32_t max_ctx;        // host bound on the context lengths (longer ones are clamped)
    int32_t waves;          // 4 or 8 waves per workgroup
    int32_t planned;        // persistent schedule built on the device (4 waves, batch <= kPlanMaxBatch)
    int32_t balanced;       // with planned: page-balanced chunks (automatic split length)
    int32_t slots_per_head; // balanced: partial slots per KV head
    int32_t key_interleaved;  // K channels stored as rotary pairs (2i, 2i+1)
    float scale;
};

int launch_decode_attn(const AttnLaunch &a, hipStream_t stream);
// Fixed device scratch of the no-allocation entry point (one per GPU, for the
// life of the process): split-merge tickets in the first kScratchTicketBytes
// (the same place for calls of any shape), partials after them.
constexpr size_t kScratchBytes = size_t(16) << 20;
constexpr size_t kScratchTicketBytes = size_t(64) << 10;

// Device address of the current device's scratch; the first call on a device
// clears its ticket region with a kernel on `stream`.  Returns 0 or -1.
int noalloc_scratch(hipStream_t stream, uint8_t **base);

// Read-only probes (read_probe.hip): the attention's BFP8 bytes in its
// decomposition, and one contiguous buffer; each wave writes an XOR to sink.
int launch_paged_read_probe(const uint8_t *k_mant, const uint8_t *k_exp, const uint8_t *v_mant,
                            const uint8_t *v_exp, const int32_t *page_table, int32_t max_pages,
                            const int32_t *ctx, int32_t max_ctx, int32_t batch, int32_t hkv,
                            int32_t heads_per_wg, int32_t pages_per_split, int32_t n_splits, uint32_t *sink,
                            hipStream_t stream);
int launch_stream_read_probe(const void *buf, uint64_t bytes, uint32_t *sink, int32_t n_workgroups,
                             hipStream_t stream);
// Issue probe (read_probe.hip): n_waves one-wave workgroups; kind 0..4,
// valu_ops in {0, 8, 16}; cycles[w] and sink[w * 64 + lane] written per wave.
int launch_issue_probe(int32_t kind, int32_t valu_ops, bool mfma, int32_t n_waves, int32_t iters, uint64_t *cycles,
                       uint32_t *sink, hipStream_t stream);

// Vector-ALU decode attention (valu_attn.hip): per split a partial kernel
// (grid batch * hkv * n_splits), then a merge kernel (grid batch * hkv).
// part_ml holds batch * hkv * n_splits * g * 2 floats, part_o
// batch * hkv * n_splits * g * 128; every slot is written each call.
int launch_decode_attn_valu(const uint16_t *q, const uint8_t *k_mant, const uint8_t *k_exp, const uint8_t *v_mant,
                            const uint8_t *v_exp, const int32_t *page_table, int32_t max_pages,
                            const int32_t *ctx, int32_t max_ctx, int32_t batch, int32_t hq, int32_t hkv,
                            float scale, int32_t tps, int32_t n_splits, float *part_ml, float *part_o,
                            uint16_t *out, float *lse, hipStream_t stream);

}  // namespace hma
