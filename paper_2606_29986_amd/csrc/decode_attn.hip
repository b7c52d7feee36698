// decode_attn.hip -- fused BFP8 paged single-token GQA decode attention (gfx950).
//
// The paper reconstructs BFP8 pages to BF16 inline, inside the paged-attention
// read (Sec. 3.3, Fig. 2).  This kernel does the same on CDNA4: mantissa and
// exponent bytes are streamed from HBM once, decoded to exact BF16 in
// registers on the VALU, and fed to the matrix cores.
//
// Work decomposition.  One workgroup (4 waves) owns one (sequence b, KV head
// j, split s): the tokens [s*tps, min(ctx_b, (s+1)*tps)).  The split's slice
// of the page table is staged in LDS once.  A wave walks the split one
// 16-token page at a time, page c going to wave c % 4.  For pure-BFP8 page
// tables each page's four tiles are copied into LDS by direct-to-LDS loads,
// the next page's loads in flight while the current page is decoded and
// multiplied; when BF16 pages may appear, pages are loaded into registers.
//
// Per page, with g = Hq/Hkv query heads padded to 16:
//   QK : S[16 tok][16 heads] = K_page[16 tok][128] . Q^T[128][16]
//        four v_mfma_f32_16x16x32_bf16.  Lane (G = lane/16, r = lane%16)
//        feeds token r with channels {16G..16G+15} and {64+16G..64+16G+15}
//        (two 16-channel blocks, one exponent each) and Q^T's column r (head
//        j*g + r) with the same channels; the order of the contraction index
//        is free as long as both operands agree.
//   softmax : online, in the log2 domain; the C layout leaves lane (G, r)
//        with head r and tokens 4G..4G+3.
//   PV : O^T[128][16 heads] += V^T[128][16 tok] . P^T[16 tok][16 heads]
//        eight v_mfma_f32_16x16x16_bf16 pairs (n = 0..7; P^T as BF16 high +
//        low parts, so the softmax weights keep ~16 bits); row r of MFMA n is
//        channel 8r + n, so lane (G, r) needs 8 consecutive bytes (channels
//        8r..8r+7, one exponent block) of each of its tokens 4G..4G+3, and
//        P^T is exactly the lane's own softmax output.  The accumulator
//        leaves lane (G, r) with head r, channels 32G..32G+31 -- the same head
//        as its softmax state, so the online rescale needs no data movement.
//
// Split merge.  The four waves are merged through LDS.  With more than one
// split, each workgroup publishes (max, sum, weighted values) with
// device-coherent (sc1) stores, waits for them to complete, and takes a ticket
// with a device-scope atomic; the last workgroup of (b, j) folds all the
// splits' partials, in split order, with device-coherent loads (log-sum-exp).
// No cache-wide writeback or invalidate is involved (on this multi-XCD part
// an agent-scope fence writes back and invalidates the whole L2).
#include "hma_device.h"
#include "hma_internal.h"

// No implicit multiply-add contraction: both kernel variants (pure BFP8 and
// mixed formats) must evaluate the same operation sequence, so that a page's
// result does not depend on the variant that read it; the fused operations
// below are written out with fmaf.
#pragma clang fp contract(off)

namespace hma {

constexpr int kAttnWaves = 4;
constexpr float kLn2 = 0.69314718055994531f;
constexpr float kLog2e = 1.44269504088896341f;
constexpr int kCoherent = 16;                // buffer cache policy: sc1 (device-coherent)

struct AttnParams {
    const uint16_t *q;
    const uint8_t *k_mant, *k_exp, *v_mant, *v_exp;
    const uint16_t *k_bf16, *v_bf16;
    const int32_t *page_table;
    const int32_t *ctx_lens;
    uint16_t *out;
    float *lse;
    int32_t *tickets;
    float2 *part_ml;
    float *part_o;
    int32_t max_pages, batch, hq, hkv, g, tps, n_splits;
    float scale_log2;
};

typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));

// 16 x 16 x 32 tile (QK: contraction over 32 channels)
__device__ __forceinline__ f32x4_t mfma_k32(u32x4_t a, u32x4_t b, f32x4_t c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                   __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}

// 16 x 16 x 16 tile (PV: contraction over the 16 tokens of a page)
__device__ __forceinline__ f32x4_t mfma_k16(u32x2_t a, u32x2_t b, f32x4_t c)
{
    return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(bf16x4_t, a),
                                                     __builtin_bit_cast(bf16x4_t, b), c, 0, 0, 0);
}

// float -> BF16 bits, round to nearest even (v_cvt_pk_bf16_f32 on gfx950)
__device__ __forceinline__ uint32_t pack_bf16_rne(float lo, float hi)
{
    typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
    typedef float f32x2_t __attribute__((ext_vector_type(2)));
    f32x2_t f = {lo, hi};
    bf16x2_t h = __builtin_convertvector(f, bf16x2_t);
    return __builtin_bit_cast(uint32_t, h);
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t raw_rsrc(const void *base)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), 0, 0x7FFFFFFF, 0x00020000);
}

// Channel of the k-th 8-element group of lane group G in the QK contraction.
__device__ __forceinline__ int qk_channel(int G, int kk)
{
    return (kk >> 1) * 64 + 16 * G + (kk & 1) * 8;
}

// Write 32 channels of one head as BF16: o[n][i] is channel 32G + 8i + n.
__device__ __forceinline__ void store_out_row(uint16_t *dst, const f32x4_t (&o)[8], float inv)
{
#pragma unroll
    for (int i = 0; i < 4; i++) {
        u32x4_t v;
        v.x = pack_bf16_rne(o[0][i] * inv, o[1][i] * inv);
        v.y = pack_bf16_rne(o[2][i] * inv, o[3][i] * inv);
        v.z = pack_bf16_rne(o[4][i] * inv, o[5][i] * inv);
        v.w = pack_bf16_rne(o[6][i] * inv, o[7][i] * inv);
        *reinterpret_cast<u32x4_t *>(dst + 8 * i) = v;
    }
}

// ------------------------------------------------------------ page loads

// Uniform description of one page step: its page-table entry and the number
// of valid tokens (1..16).
struct PageInfo {
    uint32_t ent;
    int nval;
};

__device__ __forceinline__ PageInfo page_info(const uint32_t *sm_pt, int pi, int n_tok)
{
    PageInfo c;
    c.nval = min(kPageSize, n_tok - pi * kPageSize);
    c.ent = __builtin_amdgcn_readfirstlane(sm_pt[pi]);
    return c;
}

// Raw bytes of one page held by one lane.
template <bool MIXED>
struct PageRaw;

template <>
struct PageRaw<false> {
    u32x4_t km0, km1;     // K mantissa: blocks G and 4 + G of token r
    u32x2_t ke;           // K exponent row of token r
    u32x2_t vm[4];        // V mantissa: channels 8r..8r+7 of tokens 4G + i
    uint32_t ve[4];       // V exponent byte (block r/2) of those tokens
};

template <>
struct PageRaw<true> {
    u32x4_t k[4];         // BFP8: [0..1] mantissa, [2].xy exponent row; BF16: 4 x 8 values
    u32x4_t v[4];         // BFP8: .xy mantissa, .z exponent byte; BF16: 8 values
};

// Register loads of one page (the mixed-format path).
__device__ __forceinline__ void load_page_regs(PageRaw<true> &c, const PageInfo &inf, const AttnParams &p,
                                               int j, int G, int r)
{
    const int64_t tile = (int64_t)(inf.ent & kIdMask) * p.hkv + j;
    const uint32_t off_vm = 4 * G * kHeadDim + 8 * r;
    if (inf.ent & kTagBf16) {
        const char *kt = reinterpret_cast<const char *>(p.k_bf16 + tile * kTileMant);
        const char *vt = reinterpret_cast<const char *>(p.v_bf16 + tile * kTileMant);
#pragma unroll
        for (int kk = 0; kk < 4; kk++)
            c.k[kk] = *reinterpret_cast<const u32x4_t *>(kt + 2 * (r * kHeadDim + qk_channel(G, kk)));
#pragma unroll
        for (int i = 0; i < 4; i++)
            c.v[i] = *reinterpret_cast<const u32x4_t *>(vt + 2 * (off_vm + i * kHeadDim));
    } else {
        const uint8_t *kt = p.k_mant + tile * kTileMant;
        const uint8_t *vt = p.v_mant + tile * kTileMant;
        const uint8_t *vx = p.v_exp + tile * kTileExp;
        c.k[0] = *reinterpret_cast<const u32x4_t *>(kt + r * kHeadDim + 16 * G);
        c.k[1] = *reinterpret_cast<const u32x4_t *>(kt + r * kHeadDim + 64 + 16 * G);
        const u32x2_t ke = *reinterpret_cast<const u32x2_t *>(p.k_exp + tile * kTileExp + r * kExpPerRow);
        c.k[2] = u32x4_t{ke.x, ke.y, 0u, 0u};
#pragma unroll
        for (int i = 0; i < 4; i++) {
            const u32x2_t vm = *reinterpret_cast<const u32x2_t *>(vt + off_vm + i * kHeadDim);
            c.v[i] = u32x4_t{vm.x, vm.y, (uint32_t)vx[(4 * G + i) * kExpPerRow + (r >> 1)], 0u};
        }
    }
}

// ----------------------------------------------- LDS staging (BFP8 pages)
//
// A staging buffer holds one page (4352 bytes):
//   [0, 2048)     K mantissa tile, 16-byte units XOR-swizzled: unit 8*row + u
//                 holds bytes [16*(u ^ (row & 7)), +16) of token row `row`, so
//                 the lanes' 128-bit operand reads hit distinct banks
//   [2048, 2176)  K exponent tile [token][8]
//   [2176, 4224)  V mantissa tile [token][128]
//   [4224, 4352)  V exponent tile [token][8]
// It is filled with direct-to-LDS loads (global_load_lds_dwordx4): each of
// the 6 load instructions of a page moves a contiguous 1 KB (or 128 B) of one
// tile, and no VGPR holds data in flight.
constexpr int kPageBytes = 2 * (kTileMant + kTileExp);
constexpr int kDmaPerPage = 6;

// Wait until at most N vector-memory instructions of this wave are in flight
// (they retire in order); also a compiler memory barrier.
template <int N>
__device__ __forceinline__ void wait_vmem()
{
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// One direct-to-LDS load: every active lane copies 16 bytes from `src` to LDS
// address lds + 16 * lane.  Written as assembly so that the compiler does not
// track it as an LDS write (it would otherwise drain every such load before
// any LDS read): the explicit wait_vmem calls order it against the reads of
// the buffer it fills.  M0 is named as clobbered; nothing else in these
// kernels keeps a value in M0 (LDS instructions on gfx9+ do not use it).
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void dma16(const void *src, uint32_t lds)
{
    asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
                 :: "v"(src), "s"(lds) : "memory", "m0");
}
#pragma clang diagnostic pop

__device__ __forceinline__ uint32_t lds_addr(const void *ptr)
{
    typedef const __attribute__((address_space(3))) uint8_t *lds_ptr_t;
    return __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(lds_ptr_t)ptr);
}

__device__ __forceinline__ void dma_page(uint32_t dst, const AttnParams &p, const PageInfo &inf, int j,
                                         int lane)
{
    const int64_t tile = (int64_t)(inf.ent & kIdMask) * p.hkv + j;
    const uint8_t *km = p.k_mant + tile * kTileMant;
    const uint8_t *vm = p.v_mant + tile * kTileMant;
#pragma unroll
    for (int h = 0; h < 2; h++) {
        const int row = 8 * h + (lane >> 3);
        const int unit = (lane & 7) ^ (row & 7);
        dma16(km + row * kHeadDim + 16 * unit, dst + 1024 * h);
    }
#pragma unroll
    for (int h = 0; h < 2; h++)
        dma16(vm + 1024 * h + 16 * lane, dst + kTileMant + kTileExp + 1024 * h);
    if (lane < 8) {
        dma16(p.k_exp + tile * kTileExp + 16 * lane, dst + kTileMant);
        dma16(p.v_exp + tile * kTileExp + 16 * lane, dst + 2 * kTileMant + kTileExp);
    }
}

// The lane's operand bytes of a staged page.
__device__ __forceinline__ void lds_read_page(const uint8_t *b, PageRaw<false> &c, int G, int r)
{
    c.km0 = *reinterpret_cast<const u32x4_t *>(b + 16 * (8 * r + (G ^ (r & 7))));
    c.km1 = *reinterpret_cast<const u32x4_t *>(b + 16 * (8 * r + ((4 + G) ^ (r & 7))));
    c.ke = *reinterpret_cast<const u32x2_t *>(b + kTileMant + kExpPerRow * r);
    const uint8_t *v = b + kTileMant + kTileExp;
    const uint8_t *ve = v + kTileMant;
#pragma unroll
    for (int i = 0; i < 4; i++) {
        c.vm[i] = *reinterpret_cast<const u32x2_t *>(v + (4 * G + i) * kHeadDim + 8 * r);
        c.ve[i] = ve[(4 * G + i) * kExpPerRow + (r >> 1)];
    }
}

// ------------------------------------------------------- page compute

// K operands of one BFP8 page: decode the lane's two blocks to exact BF16.
__device__ __forceinline__ void k_operands_bfp8(u32x4_t km0, u32x4_t km1, u32x2_t ke, int G,
                                                u32x4_t (&A)[4])
{
    const int esa = (int)((ke.x >> (8 * G)) & 0xFFu) - kExpBias;
    const int esb = (int)((ke.y >> (8 * G)) & 0xFFu) - kExpBias;
    bfp8_block_to_bf16(km0, esa, A[0], A[1]);
    bfp8_block_to_bf16(km1, esb, A[2], A[3]);
}

// V^T operand pairs of two token slots (a, b) of one BFP8 page:
// pr[n] = {channel 8r+n of slot b : of slot a} as exact BF16.
__device__ __forceinline__ void v_pairs_bfp8(u32x2_t va, uint32_t ea, u32x2_t vb, uint32_t eb,
                                             uint32_t (&pr)[8])
{
    const int esa = (int)ea - kExpBias;
    const int esb = (int)eb - kExpBias;
#pragma unroll
    for (int d = 0; d < 2; d++) {
        const uint32_t wa = d ? va.y : va.x;
        const uint32_t wb = d ? vb.y : vb.x;
        const uint32_t ma = magnitudes(wa);
        const uint32_t mb = magnitudes(wb);
#pragma unroll
        for (int n4 = 0; n4 < 4; n4++)
            pr[4 * d + n4] = pack_bf16_signed(bfp8_mag_f32(ma, n4, esa), bfp8_mag_f32(mb, n4, esb),
                                              wa, n4, wb, n4);
    }
}

// Same for two slots of a BF16 page (8 values each: channels 8r..8r+7).
__device__ __forceinline__ void v_pairs_bf16(u32x4_t va, u32x4_t vb, uint32_t (&pr)[8])
{
#pragma unroll
    for (int n = 0; n < 8; n++) {
        const int w = n >> 1;
        const uint32_t a = w == 0 ? va.x : w == 1 ? va.y : w == 2 ? va.z : va.w;
        const uint32_t b = w == 0 ? vb.x : w == 1 ? vb.y : w == 2 ? vb.z : vb.w;
        pr[n] = __builtin_amdgcn_perm(b, a, (n & 1) ? kPermHiHalves : kPermLoHalves);
    }
}

// Max over the four lane groups holding the same head (lanes l, l^16, l^32,
// l^48): two gfx950 lane swaps, no LDS round trip.
__device__ __forceinline__ float max_over_groups(float x)
{
    const uint32_t u = __float_as_uint(x);
    const auto a = __builtin_amdgcn_permlane32_swap(u, u, false, false);
    const float y = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
    const uint32_t v = __float_as_uint(y);
    const auto c = __builtin_amdgcn_permlane16_swap(v, v, false, false);
    return fmaxf(__uint_as_float(c[0]), __uint_as_float(c[1]));
}

struct SoftmaxState {
    float m;       // running max of scaled scores (log2 units), head r
    float l;       // this lane's share of the running sum of weights, head r
};

// One page: QK on the matrix cores, V decode (independent of the softmax, so
// it fills the matrix-core latency), online softmax, PV on the matrix cores.
template <bool MIXED>
__device__ __forceinline__ void process_page(const PageRaw<MIXED> &c, const PageInfo &inf,
                                             const u32x4_t (&qB)[4], float scale_log2, int G,
                                             SoftmaxState &st, f32x4_t (&O)[8])
{
    // ---- QK^T
    u32x4_t A[4];
    if constexpr (MIXED) {
        if (inf.ent & kTagBf16) {
#pragma unroll
            for (int kk = 0; kk < 4; kk++)
                A[kk] = c.k[kk];
        } else {
            k_operands_bfp8(c.k[0], c.k[1], u32x2_t{c.k[2].x, c.k[2].y}, G, A);
        }
    } else {
        k_operands_bfp8(c.km0, c.km1, c.ke, G, A);
    }
    f32x4_t S = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < 4; kk++)
        S = mfma_k32(A[kk], qB[kk], S);

    // ---- V^T operands: Av[n] = channel 8r + n of tokens 4G..4G+3
    u32x2_t Av[8];
#pragma unroll
    for (int k2 = 0; k2 < 2; k2++) {
        uint32_t pr[8];
        if constexpr (MIXED) {
            const u32x4_t va = c.v[2 * k2];
            const u32x4_t vb = c.v[2 * k2 + 1];
            if (inf.ent & kTagBf16)
                v_pairs_bf16(va, vb, pr);
            else
                v_pairs_bfp8(u32x2_t{va.x, va.y}, va.z, u32x2_t{vb.x, vb.y}, vb.z, pr);
        } else {
            v_pairs_bfp8(c.vm[2 * k2], c.ve[2 * k2], c.vm[2 * k2 + 1], c.ve[2 * k2 + 1], pr);
        }
#pragma unroll
        for (int n = 0; n < 8; n++) {
            if (k2 == 0)
                Av[n].x = pr[n];
            else
                Av[n].y = pr[n];
        }
    }

    // ---- online softmax (head r, tokens 4G + i)
    float x[4];
#pragma unroll
    for (int i = 0; i < 4; i++)
        x[i] = S[i] * scale_log2;
    if (inf.nval < kPageSize) {
        // tokens past the context: no weight, and their V (which may hold
        // anything) is zeroed so that 0 * V stays 0
        const uint32_t m0 = (4 * G + 0 < inf.nval ? 0x0000FFFFu : 0u) | (4 * G + 1 < inf.nval ? 0xFFFF0000u : 0u);
        const uint32_t m1 = (4 * G + 2 < inf.nval ? 0x0000FFFFu : 0u) | (4 * G + 3 < inf.nval ? 0xFFFF0000u : 0u);
#pragma unroll
        for (int n = 0; n < 8; n++) {
            Av[n].x &= m0;
            Av[n].y &= m1;
        }
#pragma unroll
        for (int i = 0; i < 4; i++)
            if (4 * G + i >= inf.nval)
                x[i] = -INFINITY;
    }
    const float cmax = max_over_groups(fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3])));
    const float m_new = fmaxf(st.m, cmax);
    const float alpha = __builtin_amdgcn_exp2f(st.m - m_new);
    st.m = m_new;
    // P^T split into BF16 high and low parts (p = hi + lo to ~2^-17 relative)
    u32x2_t Phi, Plo;
    float psum = 0.0f;
#pragma unroll
    for (int k = 0; k < 2; k++) {
        const float p0 = __builtin_amdgcn_exp2f(x[2 * k] - m_new);
        const float p1 = __builtin_amdgcn_exp2f(x[2 * k + 1] - m_new);
        const uint32_t hi = pack_bf16_rne(p0, p1);
        const float h0 = __uint_as_float(hi << 16);
        const float h1 = __uint_as_float(hi & 0xFFFF0000u);
        const uint32_t lo = pack_bf16_rne(p0 - h0, p1 - h1);
        psum += p0 + p1;   // (p0 + p1) + (p2 + p3) for k = 1
        if (k == 0) {
            Phi.x = hi;
            Plo.x = lo;
        } else {
            Phi.y = hi;
            Plo.y = lo;
        }
    }
    st.l = fmaf(st.l, alpha, psum);
    // The running max rarely grows after the first pages: the rescale path
    // carries its own copy of the PV products so that the common path leaves
    // the accumulators where they are (no register copies at the join).
    if (__any(alpha != 1.0f)) {
#pragma unroll
        for (int n = 0; n < 8; n++) {
            O[n] *= alpha;
            O[n] = mfma_k16(Av[n], Phi, O[n]);
            O[n] = mfma_k16(Av[n], Plo, O[n]);
        }
    } else {
#pragma unroll
        for (int n = 0; n < 8; n++) {
            O[n] = mfma_k16(Av[n], Phi, O[n]);
            O[n] = mfma_k16(Av[n], Plo, O[n]);
        }
    }
}

// ------------------------------------------------------------------ kernel

constexpr int kMergeBytes = ((kAttnWaves - 1) * 32 * 64 + 2 * kAttnWaves * 16) * 4;
constexpr int kStageBytes = 2 * kAttnWaves * kPageBytes;
static_assert(kMergeBytes <= kStageBytes, "wave merge must fit in the staging buffers");

template <bool MIXED>
__global__ __launch_bounds__(64 * kAttnWaves, 2) void decode_attn_bfp8_kernel(AttnParams p)
{
    const int id = blockIdx.x;
    const int j = id % p.hkv;
    const int b = (id / p.hkv) % p.batch;
    const int s = id / (p.hkv * p.batch);
    const int ctx = p.ctx_lens[b];
    // the wave index is uniform: page bookkeeping stays in scalar registers
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    const int G = lane >> 4;
    const int r = lane & 15;
    const bool head_ok = r < p.g;
    const int head = j * p.g + (head_ok ? r : 0);
    const int64_t out_row = (int64_t)b * p.hq + head;

    const int t_begin = s * p.tps;
    if (t_begin >= ctx) {
        // empty split; split 0 of an empty sequence owns its (zero) output
        if (s == 0 && wave == 0 && head_ok) {
            u32x4_t z = {0u, 0u, 0u, 0u};
            uint16_t *o = p.out + out_row * kHeadDim + 32 * G;
#pragma unroll
            for (int i = 0; i < 4; i++)
                *reinterpret_cast<u32x4_t *>(o + 8 * i) = z;
            if (p.lse && G == 0)
                p.lse[out_row] = -INFINITY;
        }
        return;
    }
    const int n_tok = min(ctx, t_begin + p.tps) - t_begin;
    const int n_split_b = (ctx + p.tps - 1) / p.tps;
    const int n_pages = (n_tok + kPageSize - 1) / kPageSize;

    // LDS: page staging buffers [2][wave] (pure-BFP8 path), reused for the wave merge
    __shared__ __attribute__((aligned(16))) uint8_t sm_buf[MIXED ? kMergeBytes : kStageBytes];
    __shared__ uint32_t sm_pt[kMaxSplitPages];

    // stage this split's page-table slice in LDS
    {
        const int32_t *pt = p.page_table + (int64_t)b * p.max_pages + t_begin / kPageSize;
        for (int i = threadIdx.x; i < n_pages; i += 64 * kAttnWaves)
            sm_pt[i] = (uint32_t)pt[i];
    }

    // Q^T operand (column r = head j*g + r; zero for padded heads)
    u32x4_t qB[4];
    {
        const uint16_t *qrow = p.q + out_row * kHeadDim;
#pragma unroll
        for (int kk = 0; kk < 4; kk++) {
            u32x4_t v = *reinterpret_cast<const u32x4_t *>(qrow + qk_channel(G, kk));
            qB[kk] = head_ok ? v : u32x4_t{0u, 0u, 0u, 0u};
        }
    }
    __syncthreads();

    SoftmaxState st = {-INFINITY, 0.0f};
    f32x4_t O[8];
#pragma unroll
    for (int n = 0; n < 8; n++)
        O[n] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    if constexpr (MIXED) {
        // mixed page formats: register loads, one page at a time
        for (int pi = wave; pi < n_pages; pi += kAttnWaves) {
            PageRaw<true> rc;
            const PageInfo ic = page_info(sm_pt, pi, n_tok);
            load_page_regs(rc, ic, p, j, G, r);
            process_page<true>(rc, ic, qB, p.scale_log2, G, st, O);
        }
    } else {
        // staged pipeline: page k of this wave lives in buffer k % 2; the next
        // page's direct-to-LDS loads are issued before the current page is read
        // and computed.  The prefetch is issued unconditionally (past the last
        // page it re-requests the current page into the idle buffer, served by
        // the cache), so no branch separates a load from its wait and the wait
        // before each read covers exactly the page being read.
        const int my_pages = n_pages > wave ? (n_pages - wave + kAttnWaves - 1) / kAttnWaves : 0;
        if (my_pages > 0) {
            const uint8_t *buf0 = sm_buf + wave * kPageBytes;
            const uint8_t *buf1 = sm_buf + (kAttnWaves + wave) * kPageBytes;
            const uint32_t lds0 = lds_addr(buf0), lds1 = lds_addr(buf1);
            PageInfo c0 = page_info(sm_pt, wave, n_tok), c1;
            dma_page(lds0, p, c0, j, lane);
            for (int k = 0; k < my_pages; k += 2) {
                c1 = k + 1 < my_pages ? page_info(sm_pt, wave + (k + 1) * kAttnWaves, n_tok) : c0;
                dma_page(lds1, p, c1, j, lane);
                wait_vmem<kDmaPerPage>();
                {
                    PageRaw<false> rc;
                    lds_read_page(buf0, rc, G, r);
                    process_page<false>(rc, c0, qB, p.scale_log2, G, st, O);
                }
                if (k + 1 >= my_pages)
                    break;
                c0 = k + 2 < my_pages ? page_info(sm_pt, wave + (k + 2) * kAttnWaves, n_tok) : c1;
                dma_page(lds0, p, c0, j, lane);
                wait_vmem<kDmaPerPage>();
                {
                    PageRaw<false> rc;
                    lds_read_page(buf1, rc, G, r);
                    process_page<false>(rc, c1, qB, p.scale_log2, G, st, O);
                }
            }
            wait_vmem<0>();     // the last prefetch has landed before the buffers are reused
        }
    }
    // every wave is done with its staging buffers before they are reused
    __syncthreads();

    // ---- merge the four waves of the workgroup through LDS
    float l_run = st.l;
    l_run += __shfl_xor(l_run, 16);
    l_run += __shfl_xor(l_run, 32);
    float(*sm_o)[32][64] = reinterpret_cast<float(*)[32][64]>(sm_buf);
    float(*sm_m)[16] = reinterpret_cast<float(*)[16]>(sm_buf + (kAttnWaves - 1) * 32 * 64 * 4);
    float(*sm_l)[16] = reinterpret_cast<float(*)[16]>(sm_buf + ((kAttnWaves - 1) * 32 * 64 + kAttnWaves * 16) * 4);
    if (wave > 0) {
        if (G == 0) {
            sm_m[wave][r] = st.m;
            sm_l[wave][r] = l_run;
        }
#pragma unroll
        for (int n = 0; n < 8; n++)
#pragma unroll
            for (int i = 0; i < 4; i++)
                sm_o[wave - 1][8 * i + n][lane] = O[n][i];
    }
    __syncthreads();
    if (wave > 0)
        return;

    float M = st.m;
#pragma unroll
    for (int w = 1; w < kAttnWaves; w++)
        M = fmaxf(M, sm_m[w][r]);
    float L;
    {
        const float a0 = __builtin_amdgcn_exp2f(st.m - M);
        L = l_run * a0;
#pragma unroll
        for (int n = 0; n < 8; n++)
            O[n] *= a0;
#pragma unroll
        for (int w = 1; w < kAttnWaves; w++) {
            const float aw = __builtin_amdgcn_exp2f(sm_m[w][r] - M);
            L = fmaf(aw, sm_l[w][r], L);
#pragma unroll
            for (int n = 0; n < 8; n++)
#pragma unroll
                for (int i = 0; i < 4; i++)
                    O[n][i] = fmaf(aw, sm_o[w - 1][8 * i + n][lane], O[n][i]);
        }
    }

    if (n_split_b == 1) {
        if (head_ok) {
            store_out_row(p.out + out_row * kHeadDim + 32 * G, O, 1.0f / L);
            if (p.lse && G == 0)
                p.lse[out_row] = (M + log2f(L)) * kLn2;
        }
        return;
    }

    // ---- several splits: publish this split's partial (device-coherent),
    //      then the last workgroup of (b, j) to arrive merges all of them
    const int64_t pair_id = (int64_t)b * p.hkv + j;
    const __amdgpu_buffer_rsrc_t rs_o = raw_rsrc(p.part_o + pair_id * p.n_splits * p.g * kHeadDim);
    const __amdgpu_buffer_rsrc_t rs_ml = raw_rsrc(p.part_ml + pair_id * p.n_splits * p.g);
    if (head_ok) {
        const uint32_t ob = (uint32_t)(((s * p.g + r) * kHeadDim + 32 * G) * 4);
#pragma unroll
        for (int i = 0; i < 4; i++) {
            const f32x4_t a = {O[0][i], O[1][i], O[2][i], O[3][i]};
            const f32x4_t c = {O[4][i], O[5][i], O[6][i], O[7][i]};
            __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4_t, a), rs_o, ob + 32 * i, 0,
                                                   kCoherent);
            __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4_t, c), rs_o, ob + 32 * i + 16,
                                                   0, kCoherent);
        }
        if (G == 0) {
            const u32x2_t ml = {__float_as_uint(M), __float_as_uint(L)};
            __builtin_amdgcn_raw_buffer_store_b64(ml, rs_ml, (uint32_t)((s * p.g + r) * 8), 0, kCoherent);
        }
    }
    // every store of this wave has completed (device-coherent) before the ticket
    __builtin_amdgcn_s_waitcnt(0);
    int last = 0;
    if (lane == 0)
        last = __hip_atomic_fetch_add(&p.tickets[pair_id], 1, __ATOMIC_RELAXED,
                                      __HIP_MEMORY_SCOPE_AGENT) == n_split_b - 1;
    last = __shfl(last, 0);
    if (!last)
        return;

    if (head_ok) {
        // log-sum-exp merge of every split's partial: the maximum over the
        // splits first, then the weighted sums in split order (the result
        // must not depend on which workgroup arrived last).  Loads are issued
        // a batch ahead of their use, so the merge pays about one
        // device-coherent load latency per pass instead of one per split.
        constexpr int kMlBatch = 8;
        M = -INFINITY;
        for (int t0 = 0; t0 < n_split_b; t0 += kMlBatch) {
            float mt[kMlBatch];
#pragma unroll
            for (int u = 0; u < kMlBatch; u++) {
                const int t = min(t0 + u, n_split_b - 1);
                mt[u] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(
                    rs_ml, (uint32_t)((t * p.g + r) * 8), 0, kCoherent));
            }
#pragma unroll
            for (int u = 0; u < kMlBatch; u++)
                M = fmaxf(M, mt[u]);     // clamped repeats of the last split change nothing
        }
        L = 0.0f;
#pragma unroll
        for (int n = 0; n < 8; n++)
            O[n] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        f32x4_t cur[8];
        u32x2_t cur_ml;
        auto load_split = [&](int t, f32x4_t(&dst)[8], u32x2_t &ml) {
            const uint32_t ob = (uint32_t)(((t * p.g + r) * kHeadDim + 32 * G) * 4);
#pragma unroll
            for (int i = 0; i < 4; i++) {
                dst[i] = __builtin_bit_cast(
                    f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rs_o, ob + 32 * i, 0, kCoherent));
                dst[4 + i] = __builtin_bit_cast(
                    f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rs_o, ob + 32 * i + 16, 0, kCoherent));
            }
            ml = __builtin_amdgcn_raw_buffer_load_b64(rs_ml, (uint32_t)((t * p.g + r) * 8), 0, kCoherent);
        };
        load_split(0, cur, cur_ml);
        for (int t = 0; t < n_split_b; t++) {
            // the next split's loads go out before this one is folded (past
            // the end the last split is re-read and not used)
            f32x4_t nxt[8];
            u32x2_t nxt_ml;
            load_split(min(t + 1, n_split_b - 1), nxt, nxt_ml);
            const float c = __builtin_amdgcn_exp2f(__uint_as_float(cur_ml.x) - M);
            L = fmaf(__uint_as_float(cur_ml.y), c, L);
#pragma unroll
            for (int i = 0; i < 4; i++)
#pragma unroll
                for (int n = 0; n < 4; n++) {
                    O[n][i] = fmaf(cur[i][n], c, O[n][i]);
                    O[4 + n][i] = fmaf(cur[4 + i][n], c, O[4 + n][i]);
                }
#pragma unroll
            for (int k = 0; k < 8; k++)
                cur[k] = nxt[k];
            cur_ml = nxt_ml;
        }
        store_out_row(p.out + out_row * kHeadDim + 32 * G, O, 1.0f / L);
        if (p.lse && G == 0)
            p.lse[out_row] = (M + log2f(L)) * kLn2;
    }
    if (lane == 0)     // ready for the next call
        __hip_atomic_store(&p.tickets[pair_id], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

size_t attn_workspace_bytes(int32_t batch, int32_t hq, int32_t hkv, int32_t n_splits)
{
    if (n_splits <= 1)
        return 0;
    const size_t pairs = (size_t)batch * hkv;
    const size_t g = (size_t)(hq / hkv);
    const size_t tickets = (pairs * sizeof(int32_t) + 255) & ~(size_t)255;
    const size_t ml = (pairs * n_splits * g * sizeof(float2) + 255) & ~(size_t)255;
    const size_t o = pairs * n_splits * g * kHeadDim * sizeof(float);
    return tickets + ml + o;
}

int launch_decode_attn(const AttnLaunch &a, hipStream_t stream)
{
    AttnParams p;
    p.q = a.q;
    p.k_mant = a.k_mant;
    p.k_exp = a.k_exp;
    p.v_mant = a.v_mant;
    p.v_exp = a.v_exp;
    p.k_bf16 = a.k_bf16;
    p.v_bf16 = a.v_bf16;
    p.page_table = a.page_table;
    p.ctx_lens = a.ctx_lens;
    p.out = a.out;
    p.lse = a.lse;
    p.max_pages = a.max_pages;
    p.batch = a.batch;
    p.hq = a.hq;
    p.hkv = a.hkv;
    p.g = a.hq / a.hkv;
    p.tps = a.tps;
    p.n_splits = a.n_splits;
    p.scale_log2 = a.scale * kLog2e;
    p.tickets = nullptr;
    p.part_ml = nullptr;
    p.part_o = nullptr;
    if (a.n_splits > 1) {
        const size_t pairs = (size_t)a.batch * a.hkv;
        const size_t g = (size_t)p.g;
        char *ws = static_cast<char *>(a.workspace);
        const size_t tickets = (pairs * sizeof(int32_t) + 255) & ~(size_t)255;
        const size_t ml = (pairs * a.n_splits * g * sizeof(float2) + 255) & ~(size_t)255;
        p.tickets = reinterpret_cast<int32_t *>(ws);
        p.part_ml = reinterpret_cast<float2 *>(ws + tickets);
        p.part_o = reinterpret_cast<float *>(ws + tickets + ml);
    }
    const int64_t blocks = (int64_t)a.batch * a.hkv * a.n_splits;
    const bool mixed = a.k_bf16 != nullptr && a.v_bf16 != nullptr;
    if (mixed)
        hipLaunchKernelGGL(decode_attn_bfp8_kernel<true>, dim3((unsigned)blocks), dim3(64 * kAttnWaves), 0,
                           stream, p);
    else
        hipLaunchKernelGGL(decode_attn_bfp8_kernel<false>, dim3((unsigned)blocks), dim3(64 * kAttnWaves), 0,
                           stream, p);
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

}  // namespace hma
