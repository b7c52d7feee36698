// bfp8_dequant.hip -- lazy BFP8 -> BF16 page reconstruction (gfx950).
//
// The paper keeps KV pages as raw BFP8 bytes in decoder HBM and rebuilds a
// whole request's KV to BF16 in one fused pass (Sec. 3.3).  Here one wave
// rebuilds one (pool, page pair, KV head) tile: 2048 mantissa bytes and 128
// exponent bytes in, 4096 BF16 bytes out.  The pass is bound by HBM: per
// element it reads 1.0625 B and writes 2 B, against ~3.75 VALU operations.
//
// Lane mapping: a tile is 256 runs of 8 elements; in step s (0..3) lane l
// handles run l + 64 s, so every load instruction of a wave reads 512
// contiguous bytes and every store writes 1024 contiguous bytes.  All four
// steps' loads are issued before any decode to keep 2.1 KB per wave in
// flight.
#include "hma_device.h"
#include "hma_internal.h"

namespace hma {

constexpr int kDequantWaves = 4;   // tiles per workgroup

__global__ __launch_bounds__(64 * kDequantWaves) void bfp8_dequant_pages_kernel(
    const uint8_t *__restrict__ src_mant, const uint8_t *__restrict__ src_exp,
    uint16_t *__restrict__ dst, const int32_t *__restrict__ src_pages,
    const int32_t *__restrict__ dst_pages, int32_t n_pages, int64_t n_tiles, int32_t hkv,
    int64_t src_stride_pages, int64_t dst_stride_pages)
{
    const int64_t tile = (int64_t)blockIdx.x * kDequantWaves + (threadIdx.x >> 6);
    if (tile >= n_tiles)
        return;
    const int lane = threadIdx.x & 63;
    const int head = (int)(tile % hkv);
    const int64_t rest = tile / hkv;
    const int pair = (int)(rest % n_pages);
    const int64_t pool = rest / n_pages;
    const int64_t sp = src_pages ? src_pages[pair] : pair;     // NULL: the identity
    const int64_t dp = dst_pages ? dst_pages[pair] : pair;
    const int64_t src_tile = (pool * src_stride_pages + sp) * hkv + head;
    const int64_t dst_tile = (pool * dst_stride_pages + dp) * hkv + head;
    const uint8_t *m = src_mant + src_tile * kTileMant;
    const uint8_t *e = src_exp + src_tile * kTileExp;
    uint16_t *o = dst + dst_tile * kTileMant;

    u32x2_t w[4];
    uint32_t ex[4];
#pragma unroll
    for (int s = 0; s < 4; s++) {
        const int run = lane + 64 * s;                      // 8 elements: [8 run, 8 run + 8)
        w[s] = *reinterpret_cast<const u32x2_t *>(m + 8 * run);
        ex[s] = e[run >> 1];                                // 2 runs per 16-element block
    }
#pragma unroll
    for (int s = 0; s < 4; s++) {
        const int run = lane + 64 * s;
        const int es = (int)ex[s] - kExpBias;
        const u32x2_t a = bfp8_word_to_bf16(w[s].x, es);
        const u32x2_t c = bfp8_word_to_bf16(w[s].y, es);
        // streaming store: the rebuilt pages are not read again by this pass
        __builtin_nontemporal_store(u32x4_t{a.x, a.y, c.x, c.y}, reinterpret_cast<u32x4_t *>(o + 8 * run));
    }
}

int launch_bfp8_dequant_pages(const uint8_t *src_mant, const uint8_t *src_exp, uint16_t *dst,
                              const int32_t *src_pages, const int32_t *dst_pages,
                              int32_t n_pages, int32_t n_pools, int64_t src_stride_pages,
                              int64_t dst_stride_pages, int32_t hkv, hipStream_t stream)
{
    const int64_t n_tiles = (int64_t)n_pools * n_pages * hkv;
    const int64_t blocks = (n_tiles + kDequantWaves - 1) / kDequantWaves;
    hipLaunchKernelGGL(bfp8_dequant_pages_kernel, dim3((unsigned)blocks), dim3(64 * kDequantWaves),
                       0, stream, src_mant, src_exp, dst, src_pages, dst_pages, n_pages, n_tiles,
                       hkv, src_stride_pages, dst_stride_pages);
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

// Comparison baseline for the rebuild above: one thread per element, byte
// loads and 2-byte stores, no vector access and no sharing of the exponent
// between the elements of a block -- the "naive elementwise reconstruction"
// the paper sets against its fused pass (Sec. 3.3).  Same output.
__global__ __launch_bounds__(256) void bfp8_dequant_pages_naive_kernel(
    const uint8_t *__restrict__ src_mant, const uint8_t *__restrict__ src_exp,
    uint16_t *__restrict__ dst, const int32_t *__restrict__ src_pages,
    const int32_t *__restrict__ dst_pages, int32_t n_pages, int64_t n_elems, int32_t hkv,
    int64_t src_stride_pages, int64_t dst_stride_pages)
{
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= n_elems)
        return;
    const int within = (int)(e % kTileMant);            // token * 128 + channel
    const int64_t tile_idx = e / kTileMant;
    const int head = (int)(tile_idx % hkv);
    const int64_t rest = tile_idx / hkv;
    const int pair = (int)(rest % n_pages);
    const int64_t pool = rest / n_pages;
    const int64_t sp = src_pages ? src_pages[pair] : pair;
    const int64_t dp = dst_pages ? dst_pages[pair] : pair;
    const int64_t src_tile = (pool * src_stride_pages + sp) * hkv + head;
    const int64_t dst_tile = (pool * dst_stride_pages + dp) * hkv + head;
    const uint32_t b = src_mant[src_tile * kTileMant + within];
    const int E = src_exp[src_tile * kTileExp + (within / kHeadDim) * kExpPerRow + (within % kHeadDim) / kBlock];
    const float v = __builtin_amdgcn_ldexpf((float)(b & 0x7Fu), E - kExpBias);
    dst[dst_tile * kTileMant + within] = (uint16_t)((__float_as_uint(v) >> 16) | ((b & 0x80u) << 8));
}

int launch_bfp8_dequant_pages_naive(const uint8_t *src_mant, const uint8_t *src_exp, uint16_t *dst,
                                    const int32_t *src_pages, const int32_t *dst_pages,
                                    int32_t n_pages, int32_t n_pools, int64_t src_stride_pages,
                                    int64_t dst_stride_pages, int32_t hkv, hipStream_t stream)
{
    const int64_t n_elems = (int64_t)n_pools * n_pages * hkv * kTileMant;
    const int64_t blocks = (n_elems + 255) / 256;
    hipLaunchKernelGGL(bfp8_dequant_pages_naive_kernel, dim3((unsigned)blocks), dim3(256), 0, stream,
                       src_mant, src_exp, dst, src_pages, dst_pages, n_pages, n_elems, hkv,
                       src_stride_pages, dst_stride_pages);
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

int launch_ingress_rebuild(const uint8_t *host_mant, const uint8_t *host_exp, uint8_t *stage_mant,
                           uint8_t *stage_exp, uint16_t *dst, const int32_t *dst_pages, int32_t n_pages,
                           int32_t n_pools, int64_t dst_stride_pages, int32_t hkv, size_t mant_bytes,
                           size_t exp_bytes, hipStream_t stream)
{
    if (hipMemcpyAsync(stage_mant, host_mant, mant_bytes, hipMemcpyHostToDevice, stream) != hipSuccess)
        return -1;
    if (hipMemcpyAsync(stage_exp, host_exp, exp_bytes, hipMemcpyHostToDevice, stream) != hipSuccess)
        return -1;
    // staged pool p holds its n_pages pages contiguously: source stride n_pages
    return launch_bfp8_dequant_pages(stage_mant, stage_exp, dst, nullptr, dst_pages, n_pages, n_pools,
                                     n_pages, dst_stride_pages, hkv, stream);
}

}  // namespace hma
