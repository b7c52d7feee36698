// rebuild_tiled.hip -- tiled per-chip prefill shards -> BF16 pages (gfx950).
//
// The decoder's single reconstruction pass also converts the prefill side's
// tiled layout to the row-major paged layout, merges the per-chip KV shards
// and moves keys from the interleaved rotary order to the half-split order
// (Sec. 3.3).  Tile byte order (the paper gives none; fixed here):
//   shard t (chip t) holds KV heads [t*Hs, (t+1)*Hs);
//   tiles [local head][token tile of 32][channel tile of 32], 1088 bytes each:
//   64 exponent bytes [face][row], then 1024 mantissa bytes [face][row][16];
//   face f covers tile rows 16*(f/2).. and tile channels 16*(f%2)..
// With the rotary re-layout, source channel c goes to c/2 (even c) or
// 64 + c/2 (odd c).
//
// One wave rebuilds one (pool, shard, local head, token tile): the four
// channel tiles of a token tile are 4352 contiguous bytes, the output is 32
// rows of 256 bytes (two page slots ranges).  The wave first copies its 4352
// source bytes into its own LDS region with five coalesced 1 KB loads (each
// byte read once, in whole 64-byte lines), then gathers from LDS.  The work
// is cut into 512 pieces of 8 output channels (16 bytes): piece (row, q)
// writes output channels [8q, 8q + 8) of tile row `row`; lane l takes pieces
// l + 64 s, s = 0..7, so every store instruction writes 1 KB of consecutive
// page bytes.  A piece reads its block exponent and the 8 source bytes it
// needs (half a face row), or with the rotary re-layout the whole 16-byte
// face row whose even (q < 8) or odd (q >= 8) channels it keeps.
#include "hma_device.h"
#include "hma_internal.h"

namespace hma {

constexpr int kTiledWaves = 4;
constexpr int kTileBytes = 64 + 32 * 32;
constexpr int kChanTiles = kHeadDim / 32;
constexpr int kTokenTileBytes = kChanTiles * kTileBytes;     // 4352 = 272 x 16
constexpr int kTokenTileChunks = kTokenTileBytes / 16;

template <bool ROPE>
__global__ __launch_bounds__(64 * kTiledWaves) void bfp8_rebuild_tiled_kernel(
    const uint8_t *__restrict__ src, int64_t src_pool_stride_bytes, int64_t shard_bytes,
    int32_t n_shards, int32_t heads_per_shard, int32_t token_tiles, int32_t n_tokens, int64_t n_units,
    uint16_t *__restrict__ dst, const int32_t *__restrict__ dst_pages, int64_t dst_stride_pages,
    int32_t hkv)
{
    __shared__ __attribute__((aligned(16))) uint8_t sm_tiles[kTiledWaves][kTokenTileBytes];
    // wave-uniform values in scalar registers
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const int64_t unit = (int64_t)blockIdx.x * kTiledWaves + wave;
    if (unit >= n_units)
        return;          // no workgroup barrier below: each wave works alone
    const int lane = threadIdx.x & 63;
    const int tt = (int)(unit % token_tiles);
    int64_t rest = unit / token_tiles;
    const int h = (int)(rest % heads_per_shard);
    rest /= heads_per_shard;
    const int t = (int)(rest % n_shards);
    const int64_t pool = rest / n_shards;
    const uint8_t *tiles = src + pool * src_pool_stride_bytes + t * shard_bytes
                           + ((int64_t)h * token_tiles + tt) * kTokenTileBytes;

    // the tile's 32 tokens fill pages 2 tt and 2 tt + 1 (the second only
    // when the tokens reach it); their ids are read before the tile bytes
    const int32_t pi0 = 2 * tt, pi1 = 2 * tt + 1;
    const bool has1 = 16 * pi1 < n_tokens;
    const int64_t page0 = pool * dst_stride_pages + (dst_pages ? dst_pages[pi0] : pi0);
    const int64_t page1 = pool * dst_stride_pages + (has1 ? (dst_pages ? dst_pages[pi1] : pi1) : 0);

    // the token tile into this wave's LDS region: chunk lane + 64 k
    uint8_t *buf = sm_tiles[wave];
    u32x4_t chunk[5];
#pragma unroll
    for (int k = 0; k < 5; k++)
        if (lane + 64 * k < kTokenTileChunks)
            chunk[k] = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t *>(tiles) + lane + 64 * k);
#pragma unroll
    for (int k = 0; k < 5; k++)
        if (lane + 64 * k < kTokenTileChunks)
            *reinterpret_cast<u32x4_t *>(buf + 16 * (lane + 64 * k)) = chunk[k];
    // the other lanes' bytes are read below: order the wave's LDS writes
    // before its reads
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

    const int q = lane & 15;                       // output channels [8q, 8q + 8)
    // source face row of this piece: channels [16 c16, 16 c16 + 16) of the row
    const int c16 = ROPE ? (q & 7) : (q >> 1);
    const uint8_t *tile = buf + (c16 >> 1) * kTileBytes;
    const int fc = c16 & 1;

    uint32_t w0[8], w1[8], ex[8];
#pragma unroll
    for (int s = 0; s < 8; s++) {
        const int r = 4 * s + (lane >> 4);       // tile row
        const int face = 2 * (r >> 4) + fc;
        const uint8_t *frow = tile + 64 + face * 256 + (r & 15) * 16;
        ex[s] = tile[face * 16 + (r & 15)];
        if constexpr (ROPE) {
            // keep the even (q < 8) or odd (q >= 8) bytes of the face row
            const u32x4_t v = *reinterpret_cast<const u32x4_t *>(frow);
            const uint32_t sel = q < 8 ? 0x06040200u : 0x07050301u;
            w0[s] = __builtin_amdgcn_perm(v.y, v.x, sel);
            w1[s] = __builtin_amdgcn_perm(v.w, v.z, sel);
        } else {
            const u32x2_t v = *reinterpret_cast<const u32x2_t *>(frow + 8 * (q & 1));
            w0[s] = v.x;
            w1[s] = v.y;
        }
    }
#pragma unroll
    for (int s = 0; s < 8; s++) {
        const int r = 4 * s + (lane >> 4);       // rows 0..15 for s < 4, 16..31 after
        const int token = 32 * tt + r;
        if (token < n_tokens) {
            const int es = (int)ex[s] - kExpBias;
            const u32x2_t a = bfp8_word_to_bf16(w0[s], es);
            const u32x2_t c = bfp8_word_to_bf16(w1[s], es);
            const int64_t page = s < 4 ? page0 : page1;
            uint16_t *out = dst + ((page * hkv + (int64_t)t * heads_per_shard + h) * kPageSize + (r & 15))
                                  * kHeadDim + 8 * q;
            __builtin_nontemporal_store(u32x4_t{a.x, a.y, c.x, c.y}, reinterpret_cast<u32x4_t *>(out));
        }
    }
}

// The layout half of the pass, bytes unchanged: tiled shards -> BFP8 pages
// (mantissa rows of 128 bytes, exponent rows of 8), for a decoder that keeps
// raw BFP8 pages and decodes them inside attention.  Keys keep the interleaved
// rotary order (a 16-channel block cannot be relabelled without re-encoding);
// attention absorbs it by permuting the query.  Piece (row, q), q = 0..7, is
// face row (channel tile q/2, face column q%2) of tile row `row`: 16 mantissa
// bytes and the block's exponent byte; lane l takes pieces l + 64 s.
__global__ __launch_bounds__(64 * kTiledWaves) void bfp8_pack_tiled_kernel(
    const uint8_t *__restrict__ src, int64_t src_pool_stride_bytes, int64_t shard_bytes,
    int32_t n_shards, int32_t heads_per_shard, int32_t token_tiles, int32_t n_tokens, int64_t n_units,
    uint8_t *__restrict__ dst_mant, uint8_t *__restrict__ dst_exp, const int32_t *__restrict__ dst_pages,
    int64_t dst_stride_pages, int32_t hkv)
{
    const int64_t unit = (int64_t)blockIdx.x * kTiledWaves + (threadIdx.x >> 6);
    if (unit >= n_units)
        return;
    const int lane = threadIdx.x & 63;
    const int tt = (int)(unit % token_tiles);
    int64_t rest = unit / token_tiles;
    const int h = (int)(rest % heads_per_shard);
    rest /= heads_per_shard;
    const int t = (int)(rest % n_shards);
    const int64_t pool = rest / n_shards;
    const uint8_t *tiles = src + pool * src_pool_stride_bytes + t * shard_bytes
                           + ((int64_t)h * token_tiles + tt) * kChanTiles * kTileBytes;
    const int q = lane & 7;
    const uint8_t *tile = tiles + (q >> 1) * kTileBytes;
    u32x4_t m[4];
    uint32_t e[4];
#pragma unroll
    for (int s = 0; s < 4; s++) {
        const int r = 8 * s + (lane >> 3);
        const int face = 2 * (r >> 4) + (q & 1);
        m[s] = *reinterpret_cast<const u32x4_t *>(tile + 64 + face * 256 + (r & 15) * 16);
        e[s] = tile[face * 16 + (r & 15)];
    }
#pragma unroll
    for (int s = 0; s < 4; s++) {
        const int r = 8 * s + (lane >> 3);
        const int token = 32 * tt + r;
        if (token < n_tokens) {
            const int32_t pidx = token / kPageSize;
            const int64_t page = pool * dst_stride_pages + (dst_pages ? dst_pages[pidx] : pidx);
            const int64_t row = (page * hkv + (int64_t)t * heads_per_shard + h) * kPageSize + token % kPageSize;
            __builtin_nontemporal_store(m[s], reinterpret_cast<u32x4_t *>(dst_mant + row * kHeadDim + 16 * q));
            dst_exp[row * kExpPerRow + q] = (uint8_t)e[s];
        }
    }
}

int launch_bfp8_pack_tiled(const uint8_t *src, int64_t src_pool_stride_bytes, int32_t n_pools, int32_t n_shards,
                           int32_t n_tokens, uint8_t *dst_mant, uint8_t *dst_exp, const int32_t *dst_pages,
                           int64_t dst_stride_pages, int32_t hkv, hipStream_t stream)
{
    const int32_t hs = hkv / n_shards;
    const int32_t token_tiles = (n_tokens + 31) / 32;
    const int64_t shard_bytes = (int64_t)hs * token_tiles * kChanTiles * kTileBytes;
    const int64_t n_units = (int64_t)n_pools * n_shards * hs * token_tiles;
    const int64_t blocks = (n_units + kTiledWaves - 1) / kTiledWaves;
    hipLaunchKernelGGL(bfp8_pack_tiled_kernel, dim3((unsigned)blocks), dim3(64 * kTiledWaves), 0, stream,
                       src, src_pool_stride_bytes, shard_bytes, n_shards, hs, token_tiles, n_tokens, n_units,
                       dst_mant, dst_exp, dst_pages, dst_stride_pages, hkv);
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

int launch_bfp8_rebuild_tiled(const uint8_t *src, int64_t src_pool_stride_bytes, int32_t n_pools,
                              int32_t n_shards, int32_t n_tokens, uint16_t *dst, const int32_t *dst_pages,
                              int64_t dst_stride_pages, int32_t hkv, int32_t rope_reorder,
                              hipStream_t stream)
{
    const int32_t hs = hkv / n_shards;
    const int32_t token_tiles = (n_tokens + 31) / 32;
    const int64_t shard_bytes = (int64_t)hs * token_tiles * kChanTiles * kTileBytes;
    const int64_t n_units = (int64_t)n_pools * n_shards * hs * token_tiles;
    const int64_t blocks = (n_units + kTiledWaves - 1) / kTiledWaves;
    if (rope_reorder)
        hipLaunchKernelGGL(bfp8_rebuild_tiled_kernel<true>, dim3((unsigned)blocks), dim3(64 * kTiledWaves), 0,
                           stream, src, src_pool_stride_bytes, shard_bytes, n_shards, hs, token_tiles, n_tokens,
                           n_units, dst, dst_pages, dst_stride_pages, hkv);
    else
        hipLaunchKernelGGL(bfp8_rebuild_tiled_kernel<false>, dim3((unsigned)blocks), dim3(64 * kTiledWaves), 0,
                           stream, src, src_pool_stride_bytes, shard_bytes, n_shards, hs, token_tiles, n_tokens,
                           n_units, dst, dst_pages, dst_stride_pages, hkv);
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

}  // namespace hma
