// read_probe.hip -- measurement probes: the HBM read ceiling that the fused
// attention's page loop is measured against, and the SIMD issue rate of
// matrix and vector instructions mixed as in its loop.
//
// The paged probe reads exactly the bytes a decode-attention launch must read
// (the BFP8 mantissa and exponent tiles of every page of every sequence, per
// KV head) in the attention's decomposition -- one workgroup of 8 waves per
// (sequence, group of KV heads, split), the split's page-table slice staged in
// LDS, two pages in flight per wave, non-temporal 128-bit loads -- and does
// nothing with them but an XOR.  The streaming probe reads one contiguous
// buffer.  Each wave writes the XOR of every 32-bit word it loaded to a sink,
// so a host can check that every byte was read exactly once (XOR does not
// depend on the order).
#include "hma_device.h"
#include "hma_internal.h"

namespace hma {
namespace {

constexpr int kProbeWaves = 8;
constexpr int kNonTemporal = 2;

struct PagedProbeParams {
    const uint8_t *k_mant, *k_exp, *v_mant, *v_exp;
    const int32_t *page_table;
    const int32_t *ctx;
    uint32_t *sink;
    int32_t max_pages, max_ctx, hkv, heads_per_wg, pages_per_split, n_splits;
};

struct TileWords {
    u32x4_t k0, k1, v0, v1;
    uint32_t e;
};

__device__ __forceinline__ __amdgpu_buffer_rsrc_t probe_rsrc(const void *base, uint32_t bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), 0, bytes, 0x00020000);
}

// One lane's share of the four tiles of (page entry, KV head j): 16 bytes
// of each half of each mantissa tile (each load instruction reads 1 KB of
// whole 64-byte lines) and one exponent word (lanes 0-31 of K, 32-63 of V;
// the other half's offset is past its resource and reads zero).  A dead slot gets
// empty resources: the loads are issued but read nothing.
__device__ __forceinline__ TileWords load_tiles(const PagedProbeParams &p, uint32_t ent, bool live, int j,
                                                int lane)
{
    const int64_t tile = (int64_t)(ent & kIdMask) * p.hkv + j;
    const uint32_t nm = live ? (uint32_t)kTileMant : 0u;
    const uint32_t ne = live ? (uint32_t)kTileExp : 0u;
    const __amdgpu_buffer_rsrc_t km = probe_rsrc(p.k_mant + tile * kTileMant, nm);
    const __amdgpu_buffer_rsrc_t vm = probe_rsrc(p.v_mant + tile * kTileMant, nm);
    const __amdgpu_buffer_rsrc_t kx = probe_rsrc(p.k_exp + tile * kTileExp, ne);
    const __amdgpu_buffer_rsrc_t vx = probe_rsrc(p.v_exp + tile * kTileExp, ne);
    const uint32_t off = (uint32_t)lane * 16u;
    TileWords t;
    t.k0 = __builtin_amdgcn_raw_buffer_load_b128(km, off, 0, kNonTemporal);
    t.k1 = __builtin_amdgcn_raw_buffer_load_b128(km, off + 1024u, 0, kNonTemporal);
    t.v0 = __builtin_amdgcn_raw_buffer_load_b128(vm, off, 0, kNonTemporal);
    t.v1 = __builtin_amdgcn_raw_buffer_load_b128(vm, off + 1024u, 0, kNonTemporal);
    const uint32_t ek = __builtin_amdgcn_raw_buffer_load_b32(kx, lane < 32 ? (uint32_t)lane * 4u : (uint32_t)kTileExp,
                                                             0, kNonTemporal);
    const uint32_t ev = __builtin_amdgcn_raw_buffer_load_b32(vx, lane >= 32 ? (uint32_t)(lane - 32) * 4u
                                                                            : (uint32_t)kTileExp,
                                                             0, kNonTemporal);
    t.e = ek ^ ev;
    return t;
}

__device__ __forceinline__ uint32_t fold(const TileWords &t)
{
    const u32x4_t x = t.k0 ^ t.k1 ^ t.v0 ^ t.v1;
    return x.x ^ x.y ^ x.z ^ x.w ^ t.e;
}

__device__ __forceinline__ uint32_t wave_xor(uint32_t x)
{
#pragma unroll
    for (int off = 32; off > 0; off >>= 1)
        x ^= (uint32_t)__shfl_xor((int)x, off, 64);
    return x;
}

__global__ __launch_bounds__(64 * kProbeWaves) void paged_read_probe_kernel(PagedProbeParams p)
{
    __shared__ int32_t sm_pt[kMaxSplitPages];
    const int groups = p.hkv / p.heads_per_wg;
    const int s = (int)(blockIdx.x % (uint32_t)p.n_splits);
    const int hg = (int)((blockIdx.x / (uint32_t)p.n_splits) % (uint32_t)groups);
    const int b = (int)(blockIdx.x / (uint32_t)(p.n_splits * groups));
    // wave-uniform values in scalar registers, so the buffer resources are
    // scalar (a per-lane resource would turn every load into a loop)
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const int lane = (int)(threadIdx.x & 63);

    const int ctx = min(max(p.ctx[b], 0), p.max_ctx);
    const int n_pages = (ctx + kPageSize - 1) / kPageSize;
    const int lo = s * p.pages_per_split;
    const int n_local = max(0, min(n_pages - lo, p.pages_per_split));
    for (int i = (int)threadIdx.x; i < n_local; i += (int)blockDim.x)
        sm_pt[i] = p.page_table[(int64_t)b * p.max_pages + lo + i];
    __syncthreads();

    // wave w reads KV head (w mod heads_per_wg) of the group, every
    // (8 / heads_per_wg)-th page of the split
    const int j = hg * p.heads_per_wg + wave % p.heads_per_wg;
    const int step = kProbeWaves / p.heads_per_wg;
    int i = wave / p.heads_per_wg;
    auto load = [&](int k) {
        const bool live = k < n_local;
        const uint32_t ent = live ? (uint32_t)__builtin_amdgcn_readfirstlane(sm_pt[k]) : 0u;
        return load_tiles(p, ent, live, j, lane);
    };
    uint32_t acc = 0;
    TileWords t0 = load(i);
    TileWords t1 = load(i + step);
    for (; i < n_local; i += step) {
        const TileWords t2 = load(i + 2 * step);
        acc ^= fold(t0);
        t0 = t1;
        t1 = t2;
    }
    acc = wave_xor(acc);
    if (lane == 0)
        p.sink[(int64_t)blockIdx.x * kProbeWaves + wave] = acc;
}

constexpr int kStreamThreads = 256;

__global__ __launch_bounds__(kStreamThreads) void stream_read_probe_kernel(const u32x4_t *buf, uint64_t n16,
                                                                           uint32_t *sink)
{
    // workgroup w reads its own contiguous range of 16-byte chunks, 4 KB per
    // load instruction of the workgroup and four of them in flight
    const uint64_t per = (n16 + gridDim.x - 1) / gridDim.x;
    const uint64_t lo = (uint64_t)blockIdx.x * per;
    const uint64_t hi = lo + per < n16 ? lo + per : n16;
    u32x4_t acc = {0u, 0u, 0u, 0u};
    uint64_t i = lo + threadIdx.x;
    for (; i + 3 * kStreamThreads < hi; i += 4 * kStreamThreads) {
        const u32x4_t a = __builtin_nontemporal_load(buf + i);
        const u32x4_t b = __builtin_nontemporal_load(buf + i + kStreamThreads);
        const u32x4_t c = __builtin_nontemporal_load(buf + i + 2 * kStreamThreads);
        const u32x4_t d = __builtin_nontemporal_load(buf + i + 3 * kStreamThreads);
        acc ^= a ^ b ^ c ^ d;
    }
    for (; i < hi; i += kStreamThreads)
        acc ^= __builtin_nontemporal_load(buf + i);
    const uint32_t x = wave_xor(acc.x ^ acc.y ^ acc.z ^ acc.w);
    if ((threadIdx.x & 63) == 0)
        sink[(uint64_t)blockIdx.x * (kStreamThreads / 64) + (threadIdx.x >> 6)] = x;
}

// Issue probe: one wave per workgroup, waves_per_simd of them on every SIMD;
// each step of a wave issues, eight times over, one 16x16x32 BF16 matrix
// instruction (eight independent accumulators) and/or VALU instructions of
// one kind (eight independent chains), written as inline assembly so that
// the compiler neither drops nor reorders them.  Kinds: 0 v_add_u32,
// 1 v_perm_b32, 2 v_cvt_f32_ubyte1, 3 v_pk_sub_u16 (clamped), 4 v_fma_f32
// (the first and last are plain ALU operations, the middle three are the
// block-float decode's).  A wave reports the shader-clock cycles (s_memtime)
// of its whole loop; cycles / (iters * 8) is the time of one step on a SIMD
// shared with the other waves.
template <int KIND, int VALU, bool MFMA>
__global__ __launch_bounds__(64) void issue_probe_kernel(uint64_t *cycles, uint32_t *sink, int32_t iters)
{
    const uint32_t lane = threadIdx.x;
    f32x4_t c0 = {0.f, 0.f, 0.f, 0.f}, c1 = c0, c2 = c0, c3 = c0, c4 = c0, c5 = c0, c6 = c0, c7 = c0;
    const u32x4_t a = {lane, lane * 3u, 7u, 9u};
    const uint32_t k1 = lane ^ 0x5A5A5A5Au, k2 = lane * 7u + 3u;
    uint32_t x[8];
    float f[8];
#pragma unroll
    for (int k = 0; k < 8; k++) {
        x[k] = lane * (2u * k + 1u);
        f[k] = (float)(lane + k);
    }
#define HMA_PROBE_MFMA(c)                                                                                       \
    do {                                                                                                        \
        if (MFMA)                                                                                               \
            asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+v"(c) : "v"(a), "v"(a));                \
    } while (0)
#define HMA_PROBE_VALU()                                                                                        \
    do {                                                                                                        \
        _Pragma("unroll") for (int k_ = 0; k_ < VALU; k_++) {                                                   \
            if (KIND == 0)                                                                                      \
                asm volatile("v_add_u32 %0, %0, %1" : "+v"(x[k_ & 7]) : "v"(k1));                              \
            if (KIND == 1)                                                                                      \
                asm volatile("v_perm_b32 %0, %0, %1, %2" : "+v"(x[k_ & 7]) : "v"(k1), "v"(k2));                \
            if (KIND == 2)                                                                                      \
                asm volatile("v_cvt_f32_ubyte1 %0, %1" : "=v"(f[k_ & 7]) : "v"(x[k_ & 7]));                    \
            if (KIND == 3)                                                                                      \
                asm volatile("v_pk_sub_u16 %0, %0, %1 clamp" : "+v"(x[k_ & 7]) : "v"(k1));                     \
            if (KIND == 4)                                                                                      \
                asm volatile("v_fma_f32 %0, %0, %1, %0" : "+v"(f[k_ & 7]) : "v"(k1));                          \
        }                                                                                                       \
    } while (0)
    const uint64_t t0 = __builtin_amdgcn_s_memtime();
    for (int it = 0; it < iters; it++) {
        HMA_PROBE_MFMA(c0);
        HMA_PROBE_VALU();
        HMA_PROBE_MFMA(c1);
        HMA_PROBE_VALU();
        HMA_PROBE_MFMA(c2);
        HMA_PROBE_VALU();
        HMA_PROBE_MFMA(c3);
        HMA_PROBE_VALU();
        HMA_PROBE_MFMA(c4);
        HMA_PROBE_VALU();
        HMA_PROBE_MFMA(c5);
        HMA_PROBE_VALU();
        HMA_PROBE_MFMA(c6);
        HMA_PROBE_VALU();
        HMA_PROBE_MFMA(c7);
        HMA_PROBE_VALU();
    }
    const uint64_t t1 = __builtin_amdgcn_s_memtime();
#undef HMA_PROBE_MFMA
#undef HMA_PROBE_VALU
    const f32x4_t c = c0 + c1 + c2 + c3 + c4 + c5 + c6 + c7;
    uint32_t xs = 0;
#pragma unroll
    for (int k = 0; k < 8; k++)
        xs ^= x[k] ^ __float_as_uint(f[k]);
    sink[(uint64_t)blockIdx.x * 64 + lane] = __float_as_uint(c.x + c.y + c.z + c.w) ^ xs;
    if (lane == 0)
        cycles[blockIdx.x] = t1 - t0;
}

}  // namespace

template <int KIND>
static void launch_issue_kind(int32_t valu_ops, bool mfma, dim3 grid, dim3 block, int32_t iters, uint64_t *cycles,
                              uint32_t *sink, hipStream_t stream)
{
#define HMA_PROBE_LAUNCH(V)                                                                                     \
    do {                                                                                                        \
        if (mfma)                                                                                               \
            hipLaunchKernelGGL((issue_probe_kernel<KIND, V, true>), grid, block, 0, stream, cycles, sink, iters); \
        else                                                                                                    \
            hipLaunchKernelGGL((issue_probe_kernel<KIND, V, false>), grid, block, 0, stream, cycles, sink, iters); \
    } while (0)
    if (valu_ops == 0)
        HMA_PROBE_LAUNCH(0);
    else if (valu_ops == 8)
        HMA_PROBE_LAUNCH(8);
    else
        HMA_PROBE_LAUNCH(16);
#undef HMA_PROBE_LAUNCH
}

int launch_issue_probe(int32_t kind, int32_t valu_ops, bool mfma, int32_t n_waves, int32_t iters, uint64_t *cycles,
                       uint32_t *sink, hipStream_t stream)
{
    const dim3 grid((uint32_t)n_waves), block(64);
    if (valu_ops != 0 && valu_ops != 8 && valu_ops != 16)
        return -1;
    switch (kind) {
    case 0: launch_issue_kind<0>(valu_ops, mfma, grid, block, iters, cycles, sink, stream); break;
    case 1: launch_issue_kind<1>(valu_ops, mfma, grid, block, iters, cycles, sink, stream); break;
    case 2: launch_issue_kind<2>(valu_ops, mfma, grid, block, iters, cycles, sink, stream); break;
    case 3: launch_issue_kind<3>(valu_ops, mfma, grid, block, iters, cycles, sink, stream); break;
    case 4: launch_issue_kind<4>(valu_ops, mfma, grid, block, iters, cycles, sink, stream); break;
    default: return -1;
    }
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

int launch_paged_read_probe(const uint8_t *k_mant, const uint8_t *k_exp, const uint8_t *v_mant,
                            const uint8_t *v_exp, const int32_t *page_table, int32_t max_pages,
                            const int32_t *ctx, int32_t max_ctx, int32_t batch, int32_t hkv,
                            int32_t heads_per_wg, int32_t pages_per_split, int32_t n_splits, uint32_t *sink,
                            hipStream_t stream)
{
    PagedProbeParams p;
    p.k_mant = k_mant;
    p.k_exp = k_exp;
    p.v_mant = v_mant;
    p.v_exp = v_exp;
    p.page_table = page_table;
    p.ctx = ctx;
    p.sink = sink;
    p.max_pages = max_pages;
    p.max_ctx = max_ctx;
    p.hkv = hkv;
    p.heads_per_wg = heads_per_wg;
    p.pages_per_split = pages_per_split;
    p.n_splits = n_splits;
    const int64_t grid = (int64_t)batch * (hkv / heads_per_wg) * n_splits;
    hipLaunchKernelGGL(paged_read_probe_kernel, dim3((uint32_t)grid), dim3(64 * kProbeWaves), 0, stream, p);
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

int launch_stream_read_probe(const void *buf, uint64_t bytes, uint32_t *sink, int32_t n_workgroups,
                             hipStream_t stream)
{
    hipLaunchKernelGGL(stream_read_probe_kernel, dim3((uint32_t)n_workgroups), dim3(kStreamThreads), 0, stream,
                       static_cast<const u32x4_t *>(buf), bytes / 16, sink);
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

}  // namespace hma
