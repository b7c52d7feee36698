/*
 * hma.h -- C ABI of libhma, the MI355X (gfx950) decode-side hot path of
 * HMA-Serve's deferred dequantization ("HBM Is Not All You Need", arXiv
 * 2606.29986, Sec. 3.3 and Fig. 2).
 *
 * KV-cache pages arrive from the prefill side as raw block-float BFP8 bytes
 * and stay that way in HBM.  Two calls consume them:
 *   hma_bfp8_dequant_pages  lazily rebuilds BFP8 pages into the paged BF16
 *                           cache (Sec. 3.3: whole-request reconstruction);
 *   hma_decode_attn_bfp8    single-token GQA decode attention that decodes
 *                           BFP8 pages in registers inside the paged read
 *                           (Sec. 3.3, Fig. 2), with the context split across
 *                           workgroups and merged by log-sum-exp.
 *
 * BFP8 element format (the paper gives a per-block shared exponent and a
 * 7-bit mantissa; the rest are this library's readings):
 *   block    = 16 consecutive head-dim channels of one token of one KV head
 *   exponent = one byte E per block (bias 127)
 *   element  = one byte: bit 7 sign s, bits 6..0 magnitude m
 *   value    = (-1)^s * m * 2^(E-133)   (exactly representable in BF16;
 *              E = 255 with m >= 64 is +-Inf; m = 0 is a zero with sign s)
 *
 * Page layouts (head_dim D = 128, page_size P = 16, per pool):
 *   mantissa pool  uint8  [pages][Hkv][P][D]      2048 B per (page, head)
 *   exponent pool  uint8  [pages][Hkv][P][D/16]    128 B per (page, head)
 *   BF16 pool      uint16 [pages][Hkv][P][D]      4096 B per (page, head)
 * A page table entry is a page id; with HMA_PAGE_BF16 set the page lives in
 * the BF16 pool, else in the BFP8 pools.  Logical token t of a sequence is
 * slot t % P of the page named by entry t / P.
 *
 * Conventions for every call:
 *   - Pointers are DEVICE pointers unless stated otherwise; the caller owns
 *     every buffer.  The library keeps no pointer to caller memory.  Its
 *     process-wide state is a per-device cache of the attention kernel's
 *     occupancy (queried on first use) and the fixed device scratch of
 *     hma_decode_attn_bfp8_noalloc with its per-device address.  Calls are
 *     reentrant and may run on different streams concurrently, provided they
 *     do not share a workspace (nor, for the no-allocation entry, a GPU).
 *   - Work is enqueued on `stream` (a hipStream_t; NULL = default stream).
 *     No call synchronises or allocates.
 *   - Arguments are validated on the host before any HIP call; a rejected
 *     call enqueues nothing.  Device-resident contents (page ids in range)
 *     are the caller's contract; breaking it is undefined behaviour.  A
 *     caller that wants them checked runs hma_validate_page_table on host
 *     copies first (there is no device-side trap).
 *   - Return value: HMA_OK, or a negative hma_status.  HMA_EHIP means the
 *     launch itself failed.
 */
#ifndef HMA_H
#define HMA_H

#include <stddef.h>
#include <stdint.h>

#if defined(__GNUC__)
#define HMA_API __attribute__((visibility("default")))
#else
#define HMA_API
#endif

#ifdef __cplusplus
extern "C" {
#endif

enum hma_status {
    HMA_OK = 0,
    HMA_EINVAL = -1,        /* NULL pointer, bad size, misalignment, aliasing */
    HMA_EUNSUPPORTED = -2,  /* valid but not implemented: head_dim != 128, page_size != 16, g > 16 */
    HMA_EWORKSPACE = -3,    /* workspace missing or smaller than required */
    HMA_EHIP = -4,          /* kernel launch failed */
    HMA_ESCRATCH = -5       /* larger than the fixed scratch of hma_decode_attn_bfp8_noalloc */
};

#define HMA_PAGE_BF16 0x40000000     /* page-table tag: page lives in the BF16 pool */
#define HMA_PAGE_ID_MASK 0x3FFFFFFF  /* page id bits of a page-table entry */

/*
 * hma_bfp8_dequant_pages -- lazy BFP8 -> BF16 page reconstruction
 * (Sec. 3.3: raw BFP8 pages kept in HBM and rebuilt to BF16 on the decode
 * GPU; the paper reports a fused whole-request rebuild).
 *
 * For every pool p in [0, n_pools) and pair i in [0, n_pages), the whole
 * page src_pages[i] (all KV heads) of BFP8 pool p is decoded into page
 * dst_pages[i] of BF16 pool p.  Pool p of the mantissa / exponent / BF16
 * streams starts p * src_pool_stride_pages (BFP8) or
 * p * dst_pool_stride_pages (BF16) pages after pool 0, so one call can
 * rebuild a request's K and V of every layer when those pools sit at a fixed
 * page stride in one allocation.  The output is bit-exact: every BF16 value
 * is the exact value of its BFP8 element.  Pages not named in dst_pages are
 * not touched.
 *
 *   src_mant   uint8 mantissa pool 0, 16-byte aligned
 *   src_exp    uint8 exponent pool 0, 16-byte aligned
 *   dst_bf16   uint16 BF16 pool 0, 16-byte aligned; must not overlap the
 *              source ranges touched by this call
 *   src_pages, dst_pages  int32 [n_pages] device arrays of page ids (ids in
 *              range of their pools; no two pairs may name the same
 *              destination page); either may be NULL, meaning page i
 *              itself (the identity)
 *   n_pages    number of page pairs (0 is a no-op)
 *   n_pools    number of pools (>= 1 unless n_pages == 0)
 *   num_kv_heads >= 1, head_dim == 128, page_size == 16
 * Errors: HMA_EINVAL (NULL pool pointer with n_pages > 0, negative count,
 * misalignment, pool stride below 1 with n_pools > 1, or a destination that
 * overlaps a source stream over the span the host can bound: pools
 * 0 .. n_pools - 1 at their strides with n_pages pages each, the pages an
 * identity page list touches), HMA_EUNSUPPORTED (head_dim / page_size),
 * HMA_EHIP.
 */
HMA_API int hma_bfp8_dequant_pages(const uint8_t *src_mant, const uint8_t *src_exp, uint16_t *dst_bf16,
                           const int32_t *src_pages, const int32_t *dst_pages, int32_t n_pages,
                           int32_t n_pools, int64_t src_pool_stride_pages,
                           int64_t dst_pool_stride_pages, int32_t num_kv_heads,
                           int32_t head_dim, int32_t page_size, void *stream);

/*
 * hma_bfp8_dequant_pages_naive -- the same rebuild with one thread per
 * element (byte loads, 2-byte stores, the block exponent re-read for every
 * element): the "naive elementwise reconstruction" the paper compares its
 * fused pass against (Sec. 3.3).  Arguments, result and errors are those of
 * hma_bfp8_dequant_pages.  A measurement baseline, not for production use.
 */
HMA_API int hma_bfp8_dequant_pages_naive(const uint8_t *src_mant, const uint8_t *src_exp,
                                 uint16_t *dst_bf16, const int32_t *src_pages,
                                 const int32_t *dst_pages, int32_t n_pages, int32_t n_pools,
                                 int64_t src_pool_stride_pages, int64_t dst_pool_stride_pages,
                                 int32_t num_kv_heads, int32_t head_dim, int32_t page_size,
                                 void *stream);

/*
 * hma_bfp8_rebuild_tiled -- the rest of the decoder's single reconstruction
 * pass (Sec. 3.3): the prefill side's tiled layout to row-major pages, the
 * merge of the per-chip KV shards, and (keys) the post-rotary re-layout from
 * interleaved pairs (2i, 2i+1) to half-split pairs (i, i + 64), together with
 * the BFP8 -> BF16 decode.
 *
 * Source (the paper gives no tile byte order; this is the one fixed here):
 * for each pool (a layer's K or V of one request), n_shards shards back to
 * back; shard t (chip t) holds KV heads [t*Hs, (t+1)*Hs), Hs =
 * num_kv_heads / n_shards, as 32x32-element tiles ordered [local head]
 * [token tile: 32 tokens][channel tile: 32 channels], each tile 1088 bytes:
 * 64 exponent bytes [face][row] then 1024 mantissa bytes [face][row][16];
 * face f covers tile rows 16*(f/2).. and tile channels 16*(f%2)..; the 16
 * channels of a face row (one token) share their exponent.  Rows past
 * n_tokens in the last token tile are padding and are ignored.
 *
 * Output: token p of the request goes to slot p % 16 of page dst_pages[p / 16]
 * of BF16 pool `pool`, KV head t*Hs + h, bit-exact.  With rope_reorder = 1,
 * source channel c is written to channel c/2 (c even) or 64 + c/2 (c odd).
 *
 *   src        device bytes, 16-byte aligned; pool i at + i*src_pool_stride_bytes
 *              (a multiple of 16, at least hma_tiled_shard_bytes() x n_shards)
 *   dst_bf16   BF16 pool 0 [pages][Hkv][16][128], 16-byte aligned; pool i at
 *              + i*dst_pool_stride_pages pages
 *   dst_pages  int32 [ceil(n_tokens / 16)] device page ids, or NULL (page i)
 *   num_kv_heads divisible by n_shards; head_dim 128, page_size 16
 *   rope_reorder 0 (values, or keys already half-split) or 1 (keys)
 * Errors: HMA_EINVAL, HMA_EUNSUPPORTED, HMA_EHIP.
 */
HMA_API int hma_bfp8_rebuild_tiled(const uint8_t *src, int64_t src_pool_stride_bytes, int32_t n_pools,
                           int32_t n_shards, int32_t n_tokens, uint16_t *dst_bf16,
                           const int32_t *dst_pages, int64_t dst_pool_stride_pages,
                           int32_t num_kv_heads, int32_t head_dim, int32_t page_size,
                           int32_t rope_reorder, void *stream);

/*
 * hma_bfp8_pack_tiled -- the layout half of the same pass for a decoder that
 * keeps raw BFP8 pages (Sec. 3.3): the tiled shards (source exactly as for
 * hma_bfp8_rebuild_tiled) become BFP8 pages -- mantissa rows of 128 bytes and
 * exponent rows of 8 -- with every byte unchanged and the shards merged.
 * Keys keep the interleaved rotary order (a 16-channel block cannot be
 * relabelled without re-encoding): read them with hma_decode_attn_bfp8's
 * key_order = 1.
 *   dst_mant  uint8 mantissa pool 0 [pages][Hkv][16][128], 16-byte aligned
 *   dst_exp   uint8 exponent pool 0 [pages][Hkv][16][8], 16-byte aligned
 *   pool i at + i*dst_pool_stride_pages pages of both; other arguments and
 *   errors as hma_bfp8_rebuild_tiled.
 */
HMA_API int hma_bfp8_pack_tiled(const uint8_t *src, int64_t src_pool_stride_bytes, int32_t n_pools,
                        int32_t n_shards, int32_t n_tokens, uint8_t *dst_mant, uint8_t *dst_exp,
                        const int32_t *dst_pages, int64_t dst_pool_stride_pages, int32_t num_kv_heads,
                        int32_t head_dim, int32_t page_size, void *stream);

/* Bytes of one shard of hma_bfp8_rebuild_tiled's source (host only; -1 on
 * invalid sizes): heads_per_shard x ceil(n_tokens / 32) x (head_dim / 32)
 * tiles of 1088 bytes. */
HMA_API int64_t hma_tiled_shard_bytes(int32_t n_tokens, int32_t heads_per_shard, int32_t head_dim);

/*
 * hma_ingress_rebuild -- the decode-side end of the layer-wise transfer
 * pipeline (Sec. 3.2: the decoder overlaps receive, host-to-device copy and
 * dequantization with decode; Sec. 3.3: raw BFP8 bytes arrive verbatim and are
 * rebuilt lazily).  On `stream`, in order:
 *   1. copy n_pools x n_pages raw BFP8 pages (mantissa and exponent streams)
 *      from host memory into the device staging buffers;
 *   2. rebuild them into the BF16 pools: staged page i of pool p goes to page
 *      dst_pages[i] of BF16 pool p (exactly as hma_bfp8_dequant_pages).
 * Nothing is synchronized: callers run this on a side stream, once per layer
 * as the layer's bytes arrive, and gate the decode stream on an event
 * recorded after it.  The staging buffers may be reused by the next call on
 * the same stream.
 *
 *   host_mant  uint8 [n_pools][n_pages][Hkv][16][128]; pinned (page-locked)
 *              host memory for an asynchronous copy
 *   host_exp   uint8 [n_pools][n_pages][Hkv][16][8]; pinned
 *   stage_mant, stage_exp  device buffers of the same sizes, 16-byte aligned
 *   dst_bf16   uint16 BF16 pool 0, 16-byte aligned; pool p starts
 *              p * dst_pool_stride_pages pages after it
 *   dst_pages  int32 [n_pages] device array of destination page ids (NULL:
 *              page i); no two may repeat
 *   num_kv_heads >= 1, head_dim == 128, page_size == 16
 * Errors: HMA_EINVAL (NULL pointer with pages to move, negative count,
 * misalignment, staging overlapping the destination, pool stride below 1
 * with n_pools > 1), HMA_EUNSUPPORTED, HMA_EHIP (copy or launch failed).
 */
HMA_API int hma_ingress_rebuild(const uint8_t *host_mant, const uint8_t *host_exp, uint8_t *stage_mant,
                        uint8_t *stage_exp, uint16_t *dst_bf16, const int32_t *dst_pages,
                        int32_t n_pages, int32_t n_pools, int64_t dst_pool_stride_pages,
                        int32_t num_kv_heads, int32_t head_dim, int32_t page_size, void *stream);

/*
 * hma_decode_attn_bfp8 -- single-token GQA decode attention over the paged,
 * mixed-format KV cache, with BFP8 pages decoded in registers inside the
 * paged read (Sec. 3.3, Fig. 2: reconstruction inline in paged attention).
 *
 * For sequence b and query head h (kv head j = h / (num_q_heads / num_kv_heads)):
 *   s_t = scale * <q[b][h], k_t>  for logical tokens t in [0, context_lens[b])
 *   out[b][h] = sum_t softmax(s)_t v_t           (BF16, round to nearest even)
 *   lse[b][h] = log(sum_t exp(s_t))              (natural log, float32)
 * k_t and v_t are the exact values of the stored BFP8 elements (or the stored
 * BF16 values of tagged pages).  Products and sums use float32; the context
 * is split into ranges handled by separate workgroups whose partial (max,
 * sum, weighted values) are merged exactly by log-sum-exp:
 *   - with tokens_per_split > 0, ranges of tokens_per_split tokens; when they
 *     outnumber what the chip runs at once, the kernel orders them itself
 *     from the device-resident lengths (full splits level by level, then the
 *     shorter last splits);
 *   - with tokens_per_split = 0, when the batch needs more workgroups than
 *     one per compute unit (4-wave shape), the kernel cuts the pages of the
 *     whole batch, per KV head and in sequence order, into equal chunks
 *     built on the device from the lengths, for a grid of min(2, resident
 *     workgroups per CU) x CUs: one chunk per wave when that gives chunks of
 *     at least 64 pages (each wave then attends its pieces alone), else one
 *     per workgroup; a chunk that spans several sequences yields one range
 *     per sequence.  Ragged batches therefore load every compute unit
 *     equally.  Otherwise the ranges are tokens_per_split tokens of the
 *     library's choice.
 * A ragged batch needs no host-side length information, and the schedule
 * depends only on the lengths: repeated calls give the same bits.  (The
 * number of chunks follows the occupancy of the kernel variant that runs --
 * with or without BF16 pools -- so where the two variants' occupancies
 * differ, the same batch read with and without BF16 pools may differ in the
 * last bits; each is deterministic.)
 * context_lens[b] == 0 gives out = 0 and lse = -inf.  Slots at
 * or past the context end in the last page are never used, whatever they
 * hold.
 *
 * Non-finite and extreme inputs: an element with E = 255 and m >= 64 is an
 * infinity.  Attention over a context holding an infinite K or V element is
 * outside this function's contract: the query heads that read it get
 * non-finite results (NaN or +-Inf), where float64 arithmetic would give
 * +-Inf or NaN by its own rules.  Finite elements of every exponent are
 * decoded exactly; scores and sums are float32, so a score beyond the
 * float32 range (|s_t| > ~3.4e38, possible only for block exponents near
 * 254 with large queries) overflows as float32 does.
 *
 *   q          uint16 BF16 [batch][num_q_heads][128], 16-byte aligned
 *   k_mant, v_mant  uint8 mantissa pools, 16-byte aligned
 *   k_exp, v_exp    uint8 exponent pools, 16-byte aligned
 *   k_bf16, v_bf16  uint16 BF16 pools, 16-byte aligned; both NULL or both
 *              set.  When NULL the HMA_PAGE_BF16 bit is ignored and every
 *              page is read from the BFP8 pools.
 *   page_table int32 [batch][max_pages_per_seq]
 *   context_lens  int32 [batch]; a length above max_context_len is read as
 *              max_context_len, a negative one as 0
 *   max_context_len  host-side bound that sizes the launch (no device read
 *              on the host); must be <= max_pages_per_seq * page_size
 *   num_q_heads % num_kv_heads == 0 and num_q_heads / num_kv_heads <= 16;
 *   head_dim == 128, page_size == 16
 *   scale      softmax scale (typically 1/sqrt(128))
 *   key_order  0: K pages hold key channels in the queries' order (half-split
 *              rotary pairs (i, i + 64)); 1: K pages (of both formats) hold
 *              them as the prefill side leaves them, rotary pairs (2i, 2i+1):
 *              stored channel 2i is key channel i and 2i+1 is 64 + i (the
 *              paper's post-RoPE key re-layout, Sec. 3.3, absorbed by
 *              permuting the query once instead of the keys)
 *   tokens_per_split  0 = chosen by the library (see above and
 *              hma_decode_attn_tokens_per_split); else a positive multiple
 *              of page_size (16), at most 16384
 *   out        uint16 BF16 [batch][num_q_heads][128], 16-byte aligned
 *   lse        float32 [batch][num_q_heads], or NULL
 *   workspace  device buffer of at least hma_decode_attn_workspace_bytes()
 *              bytes for the same (batch, heads, max_context_len,
 *              tokens_per_split), 256-byte aligned, zero-filled once by the
 *              caller when allocated.  Its first bytes hold one split-merge
 *              counter per (sequence, KV head) (4 bytes each, the region
 *              padded to 256 bytes) and the partial results follow.  Every
 *              call leaves its counters at zero, so the buffer serves later
 *              calls with the same batch * num_kv_heads without a new zero
 *              fill; a call with another batch * num_kv_heads needs a buffer
 *              zero-filled for it (its counters would otherwise land on
 *              earlier partials).  May be NULL when the required size is 0.
 * The argument order (key_order before tokens_per_split) is this library's.
 * Errors: HMA_EINVAL, HMA_EUNSUPPORTED, HMA_EWORKSPACE, HMA_EHIP.
 */
HMA_API int hma_decode_attn_bfp8(const uint16_t *q, const uint8_t *k_mant, const uint8_t *k_exp,
                         const uint8_t *v_mant, const uint8_t *v_exp, const uint16_t *k_bf16,
                         const uint16_t *v_bf16, const int32_t *page_table,
                         int32_t max_pages_per_seq, const int32_t *context_lens,
                         int32_t max_context_len, int32_t batch, int32_t num_q_heads,
                         int32_t num_kv_heads, int32_t head_dim, int32_t page_size, float scale,
                         int32_t key_order,
                         int32_t tokens_per_split, uint16_t *out, float *lse, void *workspace,
                         size_t workspace_bytes, void *stream);

/*
 * hma_decode_attn_bfp8_noalloc -- hma_decode_attn_bfp8 for callers that
 * cannot allocate (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc): the same arguments, validation and
 * result, without the workspace.  The split-merge counters and partial
 * results live in a fixed device array of HMA_NOALLOC_SCRATCH_BYTES inside
 * the library (one per GPU, held until the process ends); the counters sit
 * in its first 64 KiB whatever the call's shape.  The first call on a GPU
 * clears them with a kernel on `stream`; every call leaves them at zero.
 * Calls whose counters (4 bytes per (sequence, KV head)) exceed 64 KiB or
 * whose partials exceed the rest of the array return HMA_ESCRATCH without
 * launching (hma_decode_attn_workspace_bytes minus the counter region is the
 * partials' size).  The call allocates nothing.  All calls on one GPU share
 * its array: calls that overlap in time on one GPU (other streams, other
 * threads) race and give undefined results -- serialize them.
 * Errors: those of hma_decode_attn_bfp8 except HMA_EWORKSPACE, and
 * HMA_ESCRATCH.
 */
#define HMA_NOALLOC_SCRATCH_BYTES (16u << 20)
HMA_API int hma_decode_attn_bfp8_noalloc(const uint16_t *q, const uint8_t *k_mant, const uint8_t *k_exp,
                                         const uint8_t *v_mant, const uint8_t *v_exp, const uint16_t *k_bf16,
                                         const uint16_t *v_bf16, const int32_t *page_table,
                                         int32_t max_pages_per_seq, const int32_t *context_lens,
                                         int32_t max_context_len, int32_t batch, int32_t num_q_heads,
                                         int32_t num_kv_heads, int32_t head_dim, int32_t page_size,
                                         float scale, int32_t key_order, int32_t tokens_per_split,
                                         uint16_t *out, float *lse, void *stream);

/*
 * Split length the library uses for tokens_per_split = 0 (host only, no HIP
 * call).  Returns a positive multiple of 16, or 0 on invalid sizes.  It
 * decides the workgroup shape; in the 4-wave shape the ranges come from the
 * page-balanced chunking instead.  It assumes the 256 compute units of an
 * MI355X (the library is built for gfx950 only).
 */
HMA_API int32_t hma_decode_attn_tokens_per_split(int32_t batch, int32_t num_q_heads,
                                         int32_t num_kv_heads, int32_t max_context_len);

/*
 * Workspace bytes hma_decode_attn_bfp8 needs for these sizes (host only).
 * tokens_per_split = 0 means the library's choice.  Returns 0 when no
 * workspace is needed (every sequence is handled in one range) and
 * (size_t)-1 on invalid sizes.
 */
HMA_API size_t hma_decode_attn_workspace_bytes(int32_t batch, int32_t num_q_heads, int32_t num_kv_heads,
                                       int32_t max_context_len, int32_t tokens_per_split);

/*
 * hma_validate_page_table -- host-side check of what hma_decode_attn_bfp8
 * leaves to the caller (device-resident page ids in range), on HOST copies
 * of the page table and the context lengths, for callers that want the check
 * (debug builds, tests); the attention call itself never traps.
 *
 * For every sequence b, the entries the attention kernel reads -- the first
 * ceil(min(max(context_lens[b], 0), max_context_len) / page_size) of row b --
 * must be non-negative and name a page in range: an entry tagged
 * HMA_PAGE_BF16 an id below num_bf16_pages, any other an id below
 * num_bfp8_pages.  num_bf16_pages < 0 means the call passes no BF16 pools:
 * the tag is then ignored (as the attention kernel ignores it) and every id
 * is checked against num_bfp8_pages.
 *
 *   page_table   host int32 [batch][max_pages_per_seq]
 *   context_lens host int32 [batch]
 *   first_bad    out: flat index b * max_pages_per_seq + i of the first bad
 *                entry, or -1 (may be NULL)
 * Returns HMA_OK, HMA_EINVAL (a bad entry, NULL arrays with batch > 0, or
 * bad sizes) or HMA_EUNSUPPORTED (page_size != 16).
 */
HMA_API int hma_validate_page_table(const int32_t *page_table, int32_t batch, int32_t max_pages_per_seq,
                                    const int32_t *context_lens, int32_t max_context_len,
                                    int64_t num_bfp8_pages, int64_t num_bf16_pages, int32_t page_size,
                                    int64_t *first_bad);

/*
 * Read probes -- measurement, not part of the method: the HBM read ceiling
 * that the fused attention of Sec. 3.3 (whose cost is its read of the BFP8
 * pages) is compared against.  Both only read and XOR; each wave writes the
 * XOR of every 32-bit word it loaded to `sink`, so the XOR of all sink words
 * equals the XOR of all words of the bytes read, whatever the order.
 *
 * hma_paged_read_probe reads exactly the BFP8 bytes of an attention call
 * over BFP8 pages: for every sequence b and KV head j, the K and V mantissa
 * tiles (2048 B) and exponent tiles (128 B) of the pages named by the first
 * ceil(min(max(context_lens[b], 0), max_context_len) / 16) entries of row b
 * (the HMA_PAGE_BF16 tag is ignored: every entry is read as a BFP8 page).
 * Decomposition: one workgroup of 8 waves per (sequence, group of
 * heads_per_workgroup KV heads, split of pages_per_split pages); wave w reads
 * head w mod heads_per_workgroup of the group and every
 * (8 / heads_per_workgroup)-th page of the split.  heads_per_workgroup = 1 is
 * the attention kernel's decomposition (one KV head per workgroup);
 * heads_per_workgroup = num_kv_heads reads the heads of a page together.
 *   sink        device uint32 [batch * (num_kv_heads / heads_per_workgroup)
 *               * n_splits * 8]; sink_words is its length
 * Returns HMA_EINVAL for NULL or misaligned (16 B) pools, heads_per_workgroup
 * not in {1, 2, 4, 8} or not dividing num_kv_heads, pages_per_split outside
 * [1, 1024], n_splits * pages_per_split * 16 < max_context_len,
 * max_context_len > max_pages_per_seq * 16, or a short sink.
 */
HMA_API int hma_paged_read_probe(const uint8_t *k_mant, const uint8_t *k_exp, const uint8_t *v_mant,
                                 const uint8_t *v_exp, const int32_t *page_table, int32_t max_pages_per_seq,
                                 const int32_t *context_lens, int32_t max_context_len, int32_t batch,
                                 int32_t num_kv_heads, int32_t heads_per_workgroup, int32_t pages_per_split,
                                 int32_t n_splits, uint32_t *sink, size_t sink_words, void *stream);

/*
 * hma_stream_read_probe reads `bytes` contiguous bytes (a positive multiple
 * of 16, `buf` 16-byte aligned) with non-temporal 128-bit loads over
 * n_workgroups workgroups of 4 waves, each reading its own contiguous range.
 *   sink        device uint32 [n_workgroups * 4]; sink_words is its length
 * Returns HMA_EINVAL for a NULL or misaligned buffer, bytes not a positive
 * multiple of 16, n_workgroups outside [1, 1048576] or a short sink.
 */
HMA_API int hma_stream_read_probe(const void *buf, size_t bytes, int32_t n_workgroups, uint32_t *sink,
                                  size_t sink_words, void *stream);

/*
 * hma_issue_probe -- measurement, not part of the method: the SIMD issue rate
 * of matrix and vector instructions of the kinds the fused attention's loop
 * issues.  Launches 4 x 256 x waves_per_simd one-wave workgroups
 * (waves_per_simd waves on each SIMD of the 256 CUs); each wave runs `iters`
 * steps, each step issuing eight times one v_mfma_f32_16x16x32_bf16
 * (with_mfma = 1, eight independent accumulators) and valu_ops VALU
 * instructions of one kind (eight independent chains), and writes the
 * shader-clock cycles (s_memtime) of its loop to cycles[wave];
 * cycles / (iters * 8) is one step's time on a SIMD shared with the other
 * waves.
 *   valu_kind       0 v_add_u32, 1 v_perm_b32, 2 v_cvt_f32_ubyte1,
 *                   3 v_pk_sub_u16 (clamped), 4 v_fma_f32
 *   valu_ops        0, 8 or 16; with_mfma 0 or 1, not both zero
 *   waves_per_simd  1..4; iters 1..1048576
 *   cycles          device uint64 [1024 * waves_per_simd]; cycles_words its length
 *   sink            device uint32 [1024 * waves_per_simd * 64] (results kept live)
 * Errors: HMA_EINVAL, HMA_EHIP.
 */
HMA_API int hma_issue_probe(int32_t valu_kind, int32_t valu_ops, int32_t with_mfma, int32_t waves_per_simd,
                            int32_t iters, uint64_t *cycles, size_t cycles_words, uint32_t *sink, size_t sink_words,
                            void *stream);

/*
 * hma_decode_attn_bfp8_valu -- measurement, not for production: the fused
 * attention of hma_decode_attn_bfp8 over BFP8 pages (Sec. 3.3: the pages
 * decoded exactly in registers inside the paged read) with both products on
 * the vector ALU instead of the matrix cores, the comparison point for that
 * choice.  Same reads, decode routes and split decomposition (one
 * workgroup of 8 waves per (range, sequence, KV head)); QK^T runs on
 * v_dot2c_f32_bf16 (BF16 pairs, float32 sums), PV on float32 FMAs with
 * unrounded weights.  The ranges' partials are merged by log-sum-exp in a
 * second kernel.  The result is the function of hma_decode_attn_bfp8 (same
 * tolerance against exact arithmetic); the bits differ, since the sums run
 * in another order.
 *
 * Arguments as hma_decode_attn_bfp8, with these restrictions: BFP8 pools
 * only (page table entries are read as BFP8 page ids; the HMA_PAGE_BF16 tag
 * is ignored), key_order 0, num_q_heads / num_kv_heads <= 8
 * (HMA_EUNSUPPORTED otherwise).  tokens_per_split = 0 lets the library cut
 * every sequence into ranges of one length, from max_context_len: the
 * length that gives the batch one workgroup per compute unit, rounded up to
 * a multiple of 16 and at most 4096 (a static grid: a ragged batch is not
 * balanced across compute units); else a positive multiple of 16, at most
 * 16384.
 *   workspace  device buffer of at least hma_decode_attn_valu_workspace_bytes()
 *              bytes for the same sizes, 256-byte aligned; every call writes
 *              all of it before reading it (no zero fill needed).
 * Errors: HMA_EINVAL, HMA_EUNSUPPORTED, HMA_EWORKSPACE, HMA_EHIP.
 */
HMA_API int hma_decode_attn_bfp8_valu(const uint16_t *q, const uint8_t *k_mant, const uint8_t *k_exp,
                                      const uint8_t *v_mant, const uint8_t *v_exp, const int32_t *page_table,
                                      int32_t max_pages_per_seq, const int32_t *context_lens,
                                      int32_t max_context_len, int32_t batch, int32_t num_q_heads,
                                      int32_t num_kv_heads, int32_t head_dim, int32_t page_size, float scale,
                                      int32_t tokens_per_split, uint16_t *out, float *lse, void *workspace,
                                      size_t workspace_bytes, void *stream);

/*
 * Workspace bytes of hma_decode_attn_bfp8_valu (host only): (2 + 128)
 * floats per (sequence, query head, range), the (max, sum) pairs first, the
 * region padded to 256 bytes.  Returns (size_t)-1 on invalid or unsupported
 * sizes, 0 for batch 0.
 */
HMA_API size_t hma_decode_attn_valu_workspace_bytes(int32_t batch, int32_t num_q_heads, int32_t num_kv_heads,
                                                    int32_t max_context_len, int32_t tokens_per_split);

/* Static, never-NULL description of a status code. */
HMA_API const char *hma_status_string(int status);

#ifdef __cplusplus
}
#endif

#endif /* HMA_H */
