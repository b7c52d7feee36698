// decode_attn.hip -- fused BFP8 paged single-token GQA decode attention (gfx950).
//
// The paper reconstructs BFP8 pages to BF16 inline, inside the paged-attention
// read (Sec. 3.3, Fig. 2).  This kernel does the same on CDNA4: mantissa and
// exponent bytes are streamed from HBM once, decoded to exact BF16 in
// registers on the VALU, and fed to the matrix cores.
//
// Work decomposition.  A workgroup of 8 waves (one per CU, when every split
// fits in one pass over the CUs) or 4 waves (three per CU) handles one
// (sequence b, KV head j, split s) at a time: the tokens
// [s*tps, min(ctx_b, (s+1)*tps)).  Which workgroup takes which split is the
// split schedule (below the kernel body).  The split's slice of the page
// table is staged in LDS once.  A wave walks the split one 16-token page at a
// time, every fourth page of its group's share.  A page's bytes are
// loaded straight into registers in the lane layout of the matrix-core
// operands (no LDS round trip: for this scattered-page access pattern plain
// vector loads sustain a higher HBM rate than direct-to-LDS copies), and the
// loads of the wave's next page are in flight while the current page is
// decoded and multiplied.
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
// Split merge.  The waves leave their partials in LDS and each wave combines
// one (or two) of the eight accumulator columns of all of them.  With more
// than one split, every wave publishes its columns of the workgroup's
// (max, sum, weighted values) with device-coherent (sc1) stores, the stores
// complete, and one device-scope atomic takes a ticket; in the last workgroup
// of (b, j) each wave folds its columns of all the splits' partials, in split
// order, with device-coherent loads (log-sum-exp).
// No cache-wide writeback or invalidate is involved (on this multi-XCD part
// an agent-scope fence writes back and invalidates the whole L2).
#include <algorithm>
#include <atomic>
#include <mutex>

#include "hma_device.h"
#include "hma_internal.h"

// No implicit multiply-add contraction: both kernel variants (pure BFP8 and
// mixed formats) must evaluate the same operation sequence, so that a page's
// result does not depend on the variant that read it; the fused operations
// below are written out with fmaf.
#pragma clang fp contract(off)

namespace hma {

constexpr float kLn2 = 0.69314718055994531f;
constexpr float kLog2e = 1.44269504088896341f;
constexpr int kCoherent = 16;                // buffer cache policy: sc1 (device-coherent)
constexpr int kStream = 2;                   // buffer cache policy: nt (read once, streamed)

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
    int32_t max_ctx;          // context lengths are clamped to [0, max_ctx]
    int32_t planned;          // 1: persistent schedule built on the device (4-wave shape)
    int32_t balanced;         // with planned: page-balanced chunks instead of tps-token splits
    int32_t slots_per_head;   // balanced: partial slots per KV head
    int32_t key_interleaved;
    float scale_log2;
};

// One contiguous token range [t_begin, t_begin + n_tok) of (sequence b, KV
// head j) and where its partial goes: the partials of (b, j) occupy slots
// base .. base + n_parts - 1 of the partial arrays, this range's is slot
// base + idx.  n_parts == 1: the range is the whole context and its result
// is the output (no partial, no ticket).
struct Piece {
    int t_begin, n_tok;
    int idx, n_parts;
    int64_t base;
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

// ------------------------------------------------------------ page loads

// Uniform description of one page step: its page-table entry and the number
// of valid tokens (1..16).
struct PageInfo {
    uint32_t ent;
    int nval;
    bool live;      // false: a prefetch past the wave's last page (loads fetch nothing)
};

__device__ __forceinline__ PageInfo page_info(const uint32_t *sm_pt, int pi, int n_tok)
{
    PageInfo c;
    c.nval = min(kPageSize, n_tok - pi * kPageSize);
    c.ent = __builtin_amdgcn_readfirstlane(sm_pt[pi]);
    c.live = true;
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
// Byte offsets of one lane's operand pieces inside a (page, head) tile; the
// tile base is uniform, so each load is a scalar base plus a 32-bit lane
// offset (no per-page 64-bit address arithmetic on the VALU).
struct LaneOffsets {
    uint32_t k0, k1, ke;       // K mantissa pieces (blocks G, 4 + G of token r), K exponent row
    uint32_t vm[4], ve[4];     // V mantissa (channels 8r.. of token 4G + i) and its exponent byte
    uint32_t kb[4];            // BF16 K pieces (8 channels each) of a BF16 page
};

__device__ __forceinline__ LaneOffsets lane_offsets(int G, int r)
{
    LaneOffsets o;
    o.k0 = (uint32_t)(r * kHeadDim + 16 * G);
    o.k1 = o.k0 + 64;
    o.ke = (uint32_t)(r * kExpPerRow);
#pragma unroll
    for (int i = 0; i < 4; i++) {
        o.vm[i] = (uint32_t)((4 * G + i) * kHeadDim + 8 * r);
        o.ve[i] = (uint32_t)((4 * G + i) * kExpPerRow + (r >> 1));
        o.kb[i] = (uint32_t)(2 * (r * kHeadDim + qk_channel(G, i)));
    }
    return o;
}

// Buffer resource over one tile: the base is uniform, so building it is
// scalar work, and each load is resource + 32-bit lane offset (no 64-bit
// address arithmetic on the VALU).  The record count is the tile size, so a
// lane offset outside the tile would read zeros instead of a neighbour.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t tile_rsrc(const void *base, uint32_t bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), 0, bytes, 0x00020000);
}

// Register loads of one BFP8 page (the pure-BFP8 path), in the lane layout
// of the matrix-core operands: 11 loads per wave and page.
__device__ __forceinline__ void load_page_regs(PageRaw<false> &c, const PageInfo &inf, const AttnParams &p,
                                               int j, const LaneOffsets &o)
{
    const int64_t tile = (int64_t)(inf.ent & kIdMask) * p.hkv + j;
    // a prefetch past the wave's last page gets empty resources: its loads
    // are issued (so the wait counts stay uniform) but read no memory
    const uint32_t mant_bytes = inf.live ? kTileMant : 0u;
    const uint32_t exp_bytes = inf.live ? kTileExp : 0u;
    const __amdgpu_buffer_rsrc_t kt = tile_rsrc(p.k_mant + tile * kTileMant, mant_bytes);
    const __amdgpu_buffer_rsrc_t kx = tile_rsrc(p.k_exp + tile * kTileExp, exp_bytes);
    const __amdgpu_buffer_rsrc_t vt = tile_rsrc(p.v_mant + tile * kTileMant, mant_bytes);
    const __amdgpu_buffer_rsrc_t vx = tile_rsrc(p.v_exp + tile * kTileExp, exp_bytes);
    c.km0 = __builtin_amdgcn_raw_buffer_load_b128(kt, o.k0, 0, kStream);
    c.km1 = __builtin_amdgcn_raw_buffer_load_b128(kt, o.k1, 0, kStream);
    c.ke = __builtin_amdgcn_raw_buffer_load_b64(kx, o.ke, 0, kStream);
#pragma unroll
    for (int i = 0; i < 4; i++) {
        c.vm[i] = __builtin_amdgcn_raw_buffer_load_b64(vt, o.vm[i], 0, kStream);
        c.ve[i] = __builtin_amdgcn_raw_buffer_load_b8(vx, o.ve[i], 0, kStream);
    }
}

// Register loads of one page of either format (the mixed-format path).
__device__ __forceinline__ void load_page_regs(PageRaw<true> &c, const PageInfo &inf, const AttnParams &p,
                                               int j, const LaneOffsets &o)
{
    const int64_t tile = (int64_t)(inf.ent & kIdMask) * p.hkv + j;
    if (inf.ent & kTagBf16) {
        const char *kt = reinterpret_cast<const char *>(p.k_bf16 + tile * kTileMant);
        const char *vt = reinterpret_cast<const char *>(p.v_bf16 + tile * kTileMant);
#pragma unroll
        for (int kk = 0; kk < 4; kk++)
            c.k[kk] = *reinterpret_cast<const u32x4_t *>(kt + o.kb[kk]);
#pragma unroll
        for (int i = 0; i < 4; i++)
            c.v[i] = *reinterpret_cast<const u32x4_t *>(vt + 2 * o.vm[i]);
    } else {
        const uint8_t *kt = p.k_mant + tile * kTileMant;
        const uint8_t *kx = p.k_exp + tile * kTileExp;
        const uint8_t *vt = p.v_mant + tile * kTileMant;
        const uint8_t *vx = p.v_exp + tile * kTileExp;
        c.k[0] = *reinterpret_cast<const u32x4_t *>(kt + o.k0);
        c.k[1] = *reinterpret_cast<const u32x4_t *>(kt + o.k1);
        const u32x2_t ke = *reinterpret_cast<const u32x2_t *>(kx + o.ke);
        c.k[2] = u32x4_t{ke.x, ke.y, 0u, 0u};
#pragma unroll
        for (int i = 0; i < 4; i++) {
            const u32x2_t vm = *reinterpret_cast<const u32x2_t *>(vt + o.vm[i]);
            c.v[i] = u32x4_t{vm.x, vm.y, (uint32_t)vx[o.ve[i]], 0u};
        }
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

// Block exponents of one BFP8 page as one lane uses them, as 133 - E in
// 16-bit halves: k = {block G, block 4 + G} of token r; v01, v23 = {token 4G,
// 4G + 1} and {4G + 2, 4G + 3} of channel block r / 2.
struct ExpHalves {
    uint32_t k, v01, v23;
};

__device__ __forceinline__ ExpHalves exp_halves(u32x2_t ke, uint32_t e0, uint32_t e1, uint32_t e2,
                                                uint32_t e3, int G)
{
    const uint32_t bias = 0x00850085u;     // 133 in each half
    ExpHalves h;
    h.k = pk_sub_u16(bias, __builtin_amdgcn_perm(ke.y, ke.x, 0x0C000C00u | ((uint32_t)(4 + G) << 16) | (uint32_t)G));
    h.v01 = pk_sub_u16(bias, __builtin_amdgcn_perm(e1, e0, 0x0C040C00u));
    h.v23 = pk_sub_u16(bias, __builtin_amdgcn_perm(e3, e2, 0x0C040C00u));
    return h;
}

// True (for the whole wave) when every block of the page has 7 <= E <= 133,
// i.e. 133 - E <= 126 as an unsigned 16-bit value, so the packed route is exact.
__device__ __forceinline__ bool fast_route(const ExpHalves &h)
{
    const uint32_t mx = pk_max_u16(pk_max_u16(h.k, h.v01), h.v23);
    const bool out_of_range = (pk_add_sat_u16(mx, 0x7F817F81u) & 0x80008000u) != 0;   // a half >= 127
    return __builtin_amdgcn_ballot_w64(out_of_range) == 0;
}

// K operands on the packed route.
__device__ __forceinline__ void k_operands_fast(u32x4_t km0, u32x4_t km1, uint32_t hk, u32x4_t (&A)[4])
{
    const uint32_t d = pk_shl7_u16(hk);
    bfp8_block_to_bf16_fast(km0, __builtin_amdgcn_perm(d, d, 0x01000100u), A[0], A[1]);
    bfp8_block_to_bf16_fast(km1, __builtin_amdgcn_perm(d, d, 0x03020302u), A[2], A[3]);
}

// V^T operand pairs on the packed route (hab: slot a in the low half, b high).
__device__ __forceinline__ void v_pairs_fast(u32x2_t va, u32x2_t vb, uint32_t hab, uint32_t (&pr)[8])
{
    const uint32_t d = pk_shl7_u16(hab);
#pragma unroll
    for (int dd = 0; dd < 2; dd++) {
        const uint32_t wa = dd ? va.y : va.x;
        const uint32_t wb = dd ? vb.y : vb.x;
        const uint32_t ma = magnitudes(wa);
        const uint32_t mb = magnitudes(wb);
#pragma unroll
        for (int n4 = 0; n4 < 4; n4++)
            pr[4 * dd + n4] = pack_bf16_scaled_signed(mag_byte(ma, n4), mag_byte(mb, n4), d, wa, n4, wb, n4);
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

// Sum over the same four lane groups: (x_l + x_l^16) + (the same at l^32),
// identical in all four lanes.
__device__ __forceinline__ float sum_over_groups(float x)
{
    const uint32_t u = __float_as_uint(x);
    const auto a = __builtin_amdgcn_permlane16_swap(u, u, false, false);
    const float y = __uint_as_float(a[0]) + __uint_as_float(a[1]);
    const uint32_t v = __float_as_uint(y);
    const auto c = __builtin_amdgcn_permlane32_swap(v, v, false, false);
    return __uint_as_float(c[0]) + __uint_as_float(c[1]);
}

// threadIdx.x through an opaque move.  In the persistent schedule the split
// body runs in a loop; without this the compiler hoists lane-derived
// addresses and constants out of the loop and keeps them live across it,
// which costs the registers of a third workgroup per CU.
__device__ __forceinline__ int thread_index()
{
    int t;
    asm volatile("v_mov_b32 %0, %1" : "=v"(t) : "v"((int)threadIdx.x));
    return t;
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
    // ---- decode route of a BFP8 page (uniform over the wave)
    ExpHalves eh;
    bool fast = false;
    if constexpr (MIXED) {
        if (!(inf.ent & kTagBf16)) {
            eh = exp_halves(u32x2_t{c.k[2].x, c.k[2].y}, c.v[0].z, c.v[1].z, c.v[2].z, c.v[3].z, G);
            fast = fast_route(eh);
        }
    } else {
        eh = exp_halves(c.ke, c.ve[0], c.ve[1], c.ve[2], c.ve[3], G);
        fast = fast_route(eh);
    }

    // ---- QK^T
    u32x4_t A[4];
    if constexpr (MIXED) {
        if (inf.ent & kTagBf16) {
#pragma unroll
            for (int kk = 0; kk < 4; kk++)
                A[kk] = c.k[kk];
        } else if (fast) {
            k_operands_fast(c.k[0], c.k[1], eh.k, A);
        } else {
            k_operands_bfp8(c.k[0], c.k[1], u32x2_t{c.k[2].x, c.k[2].y}, G, A);
        }
    } else {
        if (fast)
            k_operands_fast(c.km0, c.km1, eh.k, A);
        else
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
        const uint32_t hab = k2 ? eh.v23 : eh.v01;
        if constexpr (MIXED) {
            const u32x4_t va = c.v[2 * k2];
            const u32x4_t vb = c.v[2 * k2 + 1];
            if (inf.ent & kTagBf16)
                v_pairs_bf16(va, vb, pr);
            else if (fast)
                v_pairs_fast(u32x2_t{va.x, va.y}, u32x2_t{vb.x, vb.y}, hab, pr);
            else
                v_pairs_bfp8(u32x2_t{va.x, va.y}, va.z, u32x2_t{vb.x, vb.y}, vb.z, pr);
        } else {
            if (fast)
                v_pairs_fast(c.vm[2 * k2], c.vm[2 * k2 + 1], hab, pr);
            else
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

// LDS bytes of the wave merge: one slot of accumulators per wave, then their
// (max, sum) per head, then the ticket flag.
constexpr int kMergeSlotBytes = 8 * 64 * 16;     // one wave's accumulators: 8 x f32x4 per lane

template <int WAVES>
constexpr int merge_bytes()
{
    return WAVES * (kMergeSlotBytes + 16 * 8) + 16;
}

// Write accumulator column n (channels 32G + 8i + n, i = 0..3, of one head)
// as BF16, scaled by inv.
__device__ __forceinline__ void store_out_col(uint16_t *dst, int n, f32x4_t c, float inv)
{
#pragma unroll
    for (int i = 0; i < 4; i++)
        dst[8 * i + n] = (uint16_t)(pack_bf16_rne(c[i] * inv, 0.0f) & 0xFFFFu);
}

// With 8 waves per workgroup (one workgroup per CU), waves 0..3 are issued
// ahead of waves 4..7 on every SIMD (the instruction arbiter favours older
// waves), so an even split leaves waves 4..7 finishing last.  Waves 0..3 take
// the first kLeadShare/64 of the split's pages and waves 4..7 the rest
// (measured on Qwen3-32B 8K: 40/64 is 4% faster than an even split).  Any
// share gives the same result up to rounding; the share is fixed, so the
// result does not depend on timing.
constexpr int kLeadShare = 40;

// Pages [first, first + stride * count) of the split belong to `wave`.
struct WavePages {
    int first, count;
};

template <int WAVES>
__device__ __forceinline__ WavePages wave_pages(int n_pages, int wave)
{
    static_assert(WAVES == 4 || WAVES == 8, "4 or 8 waves per workgroup");
    int begin = 0, end = n_pages;
    if constexpr (WAVES == 8) {
        const int n_lead = min(n_pages, (n_pages * kLeadShare + 63) / 64);
        begin = wave < 4 ? 0 : n_lead;
        end = wave < 4 ? n_lead : n_pages;
    }
    const int first = begin + (wave & 3);
    return WavePages{first, end > first ? (end - first + 3) / 4 : 0};
}

// Context length of sequence b as the kernel uses it: clamped to the host
// bound, and a negative length read as an empty sequence.
__device__ __forceinline__ int context_len(const AttnParams &p, int b)
{
    return max(0, min(p.ctx_lens[b], p.max_ctx));
}

// Zero output (and lse = -inf) for the query heads of KV head j of an empty
// sequence b; one wave.
__device__ __forceinline__ void zero_pair_output(const AttnParams &p, int b, int j)
{
    const int lane = threadIdx.x & 63;
    const int G = lane >> 4;
    const int r = lane & 15;
    if (r >= p.g)
        return;
    const int64_t out_row = (int64_t)b * p.hq + j * p.g + r;
    const u32x4_t z = {0u, 0u, 0u, 0u};
    uint16_t *o = p.out + out_row * kHeadDim + 32 * G;
#pragma unroll
    for (int i = 0; i < 4; i++)
        *reinterpret_cast<u32x4_t *>(o + 8 * i) = z;
    if (p.lse && G == 0)
        p.lse[out_row] = -INFINITY;
}

// Q^T operand of lane (G, r): column r = query head j*g + r of row out_row
// (zero for padded heads).  Keys kept in the interleaved rotary order (stored
// channel 2i = key channel i, 2i + 1 = 64 + i) are met by permuting q the
// same way once, here: stored channels c0..c0+7 take q[c0/2 ..] and
// q[64 + c0/2 ..] in turn.
__device__ __forceinline__ void q_operand(const AttnParams &p, int64_t out_row, int G, bool head_ok,
                                          u32x4_t (&qB)[4])
{
    const uint16_t *qrow = p.q + out_row * kHeadDim;
#pragma unroll
    for (int kk = 0; kk < 4; kk++) {
        const int c0 = qk_channel(G, kk);
        u32x4_t v;
        if (p.key_interleaved) {
            const u32x2_t a = *reinterpret_cast<const u32x2_t *>(qrow + c0 / 2);
            const u32x2_t b = *reinterpret_cast<const u32x2_t *>(qrow + kHeadDim / 2 + c0 / 2);
            v = u32x4_t{__builtin_amdgcn_perm(b.x, a.x, kPermLoHalves), __builtin_amdgcn_perm(b.x, a.x, kPermHiHalves),
                        __builtin_amdgcn_perm(b.y, a.y, kPermLoHalves), __builtin_amdgcn_perm(b.y, a.y, kPermHiHalves)};
        } else {
            v = *reinterpret_cast<const u32x4_t *>(qrow + c0);
        }
        qB[kk] = head_ok ? v : u32x4_t{0u, 0u, 0u, 0u};
    }
}

// Online log-sum-exp fold of the n_parts published partials of one (b, j),
// in piece order (the result must not depend on which workgroup or wave
// arrived last), for accumulator columns col0 + q * step, q < NC; the next
// piece's device-coherent loads are in flight while one is folded.  Partial
// of piece t: columns [8][G 4][head g] of f32x4 at rs_o, (max, sum) per head
// at rs_ml.
template <int NC>
__device__ __forceinline__ void fold_partials(__amdgpu_buffer_rsrc_t rs_o, __amdgpu_buffer_rsrc_t rs_ml, int n_parts,
                                              int g, int G, int r, int col0, int step, f32x4_t (&F)[NC], float &Mf,
                                              float &Lf)
{
    auto col_offset = [&](int t, int n) { return (uint32_t)((((t * 8 + n) * 4 + G) * g + r) * 16); };
    Mf = -INFINITY;
    Lf = 0.0f;
#pragma unroll
    for (int q = 0; q < NC; q++)
        F[q] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    auto load_split = [&](int t, f32x4_t(&dst)[NC], u32x2_t &ml) {
#pragma unroll
        for (int q = 0; q < NC; q++)
            dst[q] = __builtin_bit_cast(
                f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rs_o, col_offset(t, col0 + q * step), 0, kCoherent));
        ml = __builtin_amdgcn_raw_buffer_load_b64(rs_ml, (uint32_t)((t * g + r) * 8), 0, kCoherent);
    };
    auto fold = [&](const f32x4_t(&v)[NC], u32x2_t ml) {
        const float mt = __uint_as_float(ml.x);
        const float Mn = fmaxf(Mf, mt);
        const float a = __builtin_amdgcn_exp2f(Mf - Mn);     // 0 for the first split
        const float c = __builtin_amdgcn_exp2f(mt - Mn);
        Lf = fmaf(Lf, a, __uint_as_float(ml.y) * c);
        Mf = Mn;
#pragma unroll
        for (int q = 0; q < NC; q++)
#pragma unroll
            for (int i = 0; i < 4; i++)
                F[q][i] = fmaf(F[q][i], a, v[q][i] * c);
    };
    // two register sets, alternating; past the end the last piece is
    // re-read and not used
    f32x4_t va[NC], vb[NC];
    u32x2_t ma, mb;
    load_split(0, va, ma);
    for (int t = 0; t < n_parts; t += 2) {
        load_split(min(t + 1, n_parts - 1), vb, mb);
        fold(va, ma);
        if (t + 1 >= n_parts)
            break;
        load_split(min(t + 2, n_parts - 1), va, ma);
        fold(vb, mb);
    }
}

// One piece of (sequence b, KV head j) (non-empty).  Every wave of the
// workgroup calls it, and every wave meets the same barriers.
template <bool MIXED, int WAVES>
__device__ __forceinline__ void attend_split(const AttnParams &p, int b, int j, const Piece &pc,
                                             uint8_t *sm_buf, uint32_t *sm_pt)
{
    const int tid = thread_index();
    // the wave index is uniform: page bookkeeping stays in scalar registers
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lane = tid & 63;
    const int G = lane >> 4;
    const int r = lane & 15;
    const bool head_ok = r < p.g;
    const int head = j * p.g + (head_ok ? r : 0);
    const int64_t out_row = (int64_t)b * p.hq + head;

    const int t_begin = pc.t_begin;
    const int n_tok = pc.n_tok;
    const int n_parts = pc.n_parts;
    const int n_pages = (n_tok + kPageSize - 1) / kPageSize;

    // stage this split's page-table slice in LDS
    {
        const int32_t *pt = p.page_table + (int64_t)b * p.max_pages + t_begin / kPageSize;
        for (int i = tid; i < n_pages; i += 64 * WAVES)
            sm_pt[i] = (uint32_t)pt[i];
    }

    u32x4_t qB[4];
    q_operand(p, out_row, G, head_ok, qB);
    __syncthreads();

    SoftmaxState st = {-INFINITY, 0.0f};
    f32x4_t O[8];
#pragma unroll
    for (int n = 0; n < 8; n++)
        O[n] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    // Register pipeline: the loads of the wave's next page are issued before
    // the current page is decoded and multiplied, so one page per wave is in
    // flight behind the computation (two register sets, alternating).  Past
    // the wave's last page the prefetch is still issued (over empty buffer
    // resources on the pure-BFP8 path; re-requesting the last page on the
    // mixed path), so the loop has no branch between a load and its use.
    const WavePages wp = wave_pages<WAVES>(n_pages, wave);
    const int my_pages = wp.count;
    if (my_pages > 0) {
        auto page_at = [&](int k) {
            PageInfo c = page_info(sm_pt, wp.first + min(k, my_pages - 1) * 4, n_tok);
            c.live = k < my_pages;
            return c;
        };
        const LaneOffsets lo = lane_offsets(G, r);
        PageRaw<MIXED> c0, c1;
        PageInfo i0 = page_at(0), i1;
        load_page_regs(c0, i0, p, j, lo);
        for (int k = 0; k < my_pages; k += 2) {
            i1 = page_at(k + 1);
            load_page_regs(c1, i1, p, j, lo);
            process_page<MIXED>(c0, i0, qB, p.scale_log2, G, st, O);
            if (k + 1 >= my_pages)
                break;
            i0 = page_at(k + 2);
            load_page_regs(c0, i0, p, j, lo);
            process_page<MIXED>(c1, i1, qB, p.scale_log2, G, st, O);
        }
    }
    // ---- merge the waves of the workgroup: every wave leaves its partial in
    //      LDS, then wave w combines accumulator column n = w (and w + WAVES)
    //      of all of them, in wave order, by log-sum-exp; the work is spread
    //      over the waves and the result does not depend on timing
    constexpr int kCols = 8 / WAVES;     // accumulator columns per wave
    f32x4_t *sm_o = reinterpret_cast<f32x4_t *>(sm_buf);
    float2 *sm_ml = reinterpret_cast<float2 *>(sm_buf + WAVES * kMergeSlotBytes);
    int32_t *sm_flag = reinterpret_cast<int32_t *>(sm_buf + WAVES * (kMergeSlotBytes + 16 * 8));
    {
        const float lw = sum_over_groups(st.l);
#pragma unroll
        for (int n = 0; n < 8; n++)
            sm_o[(wave * 8 + n) * 64 + lane] = O[n];
        if (G == 0)
            sm_ml[wave * 16 + r] = float2{st.m, lw};
    }
    __syncthreads();
    float M = -INFINITY;
    float2 wml[WAVES];
#pragma unroll
    for (int k = 0; k < WAVES; k++) {
        wml[k] = sm_ml[k * 16 + r];
        M = fmaxf(M, wml[k].x);
    }
    const float Ms = M == -INFINITY ? 0.0f : M;     // a head whose partials are all empty stays empty
    float L = 0.0f;
    f32x4_t C[kCols];
#pragma unroll
    for (int q = 0; q < kCols; q++)
        C[q] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int k = 0; k < WAVES; k++) {
        const float ck = __builtin_amdgcn_exp2f(wml[k].x - Ms);
        L = fmaf(wml[k].y, ck, L);
#pragma unroll
        for (int q = 0; q < kCols; q++) {
            const f32x4_t ok = sm_o[(k * 8 + wave + q * WAVES) * 64 + lane];
#pragma unroll
            for (int i = 0; i < 4; i++)
                C[q][i] = fmaf(ok[i], ck, C[q][i]);
        }
    }
    uint16_t *orow = p.out + out_row * kHeadDim + 32 * G;

    if (n_parts == 1) {
        if (head_ok) {
            const float inv = 1.0f / L;
#pragma unroll
            for (int q = 0; q < kCols; q++)
                store_out_col(orow, wave + q * WAVES, C[q], inv);
            if (p.lse && wave == 0 && G == 0)
                p.lse[out_row] = (M + log2f(L)) * kLn2;
        }
        return;
    }

    // ---- several pieces: publish this piece's partial (device-coherent),
    //      then the last workgroup of (b, j) to arrive merges all of them.
    //      Partial of piece t: columns [8][G 4][head g] of f32x4, and
    //      (max, sum) per head.
    const int s = pc.idx;
    const int64_t pair_id = (int64_t)b * p.hkv + j;
    const __amdgpu_buffer_rsrc_t rs_o = raw_rsrc(p.part_o + pc.base * p.g * kHeadDim);
    const __amdgpu_buffer_rsrc_t rs_ml = raw_rsrc(p.part_ml + pc.base * p.g);
    auto col_offset = [&](int t, int n) { return (uint32_t)((((t * 8 + n) * 4 + G) * p.g + r) * 16); };
    if (head_ok) {
#pragma unroll
        for (int q = 0; q < kCols; q++)
            __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4_t, C[q]), rs_o,
                                                   col_offset(s, wave + q * WAVES), 0, kCoherent);
        if (wave == 0 && G == 0) {
            const u32x2_t ml = {__float_as_uint(M), __float_as_uint(L)};
            __builtin_amdgcn_raw_buffer_store_b64(ml, rs_ml, (uint32_t)((s * p.g + r) * 8), 0, kCoherent);
        }
    }
    // every store of the workgroup has completed (device-coherent) before the ticket
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (wave == 0) {
        int last = 0;
        if (lane == 0)
            last = __hip_atomic_fetch_add(&p.tickets[pair_id], 1, __ATOMIC_RELAXED,
                                          __HIP_MEMORY_SCOPE_AGENT) == n_parts - 1;
        if (lane == 0)
            *sm_flag = last;
    }
    __syncthreads();
    if (!__builtin_amdgcn_readfirstlane(*sm_flag))
        return;

    if (head_ok) {
        float Mf, Lf;
        f32x4_t F[kCols];
        fold_partials<kCols>(rs_o, rs_ml, n_parts, p.g, G, r, wave, WAVES, F, Mf, Lf);
        const float inv = 1.0f / Lf;
#pragma unroll
        for (int q = 0; q < kCols; q++)
            store_out_col(orow, wave + q * WAVES, F[q], inv);
        if (p.lse && wave == 0 && G == 0)
            p.lse[out_row] = (Mf + log2f(Lf)) * kLn2;
    }
    if (wave == 0 && lane == 0)     // ready for the next call
        __hip_atomic_store(&p.tickets[pair_id], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// One piece of (sequence b, KV head j) (non-empty) attended by one wave
// alone (the page-balanced schedule): wpt holds the page-table entries of its
// pages.  No barrier: a piece that is the whole context writes the output;
// otherwise the wave publishes its partial (device-coherent) and the last
// wave to arrive among the pieces of (b, j) folds all of them.
template <bool MIXED>
__device__ __forceinline__ void attend_wave_piece(const AttnParams &p, int b, int j, const Piece &pc,
                                                  const uint32_t *wpt)
{
    const int lane = thread_index() & 63;
    const int G = lane >> 4;
    const int r = lane & 15;
    const bool head_ok = r < p.g;
    const int head = j * p.g + (head_ok ? r : 0);
    const int64_t out_row = (int64_t)b * p.hq + head;
    u32x4_t qB[4];
    q_operand(p, out_row, G, head_ok, qB);

    SoftmaxState st = {-INFINITY, 0.0f};
    f32x4_t O[8];
#pragma unroll
    for (int n = 0; n < 8; n++)
        O[n] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    // the register pipeline of attend_split, over every page of the piece
    const int n_pages = (pc.n_tok + kPageSize - 1) / kPageSize;
    auto page_at = [&](int k) {
        const int kk = min(k, n_pages - 1);
        PageInfo c;
        c.nval = min(kPageSize, pc.n_tok - kk * kPageSize);
        c.ent = __builtin_amdgcn_readfirstlane(wpt[kk]);
        c.live = k < n_pages;
        return c;
    };
    {
        const LaneOffsets lo = lane_offsets(G, r);
        PageRaw<MIXED> c0, c1;
        PageInfo i0 = page_at(0), i1;
        load_page_regs(c0, i0, p, j, lo);
        for (int k = 0; k < n_pages; k += 2) {
            i1 = page_at(k + 1);
            load_page_regs(c1, i1, p, j, lo);
            process_page<MIXED>(c0, i0, qB, p.scale_log2, G, st, O);
            if (k + 1 >= n_pages)
                break;
            i0 = page_at(k + 2);
            load_page_regs(c0, i0, p, j, lo);
            process_page<MIXED>(c1, i1, qB, p.scale_log2, G, st, O);
        }
    }
    const float L = sum_over_groups(st.l);
    const float M = st.m;
    uint16_t *orow = p.out + out_row * kHeadDim + 32 * G;
    if (pc.n_parts == 1) {
        if (head_ok) {
            const float inv = 1.0f / L;
#pragma unroll
            for (int n = 0; n < 8; n++)
                store_out_col(orow, n, O[n], inv);
            if (p.lse && G == 0)
                p.lse[out_row] = (M + log2f(L)) * kLn2;
        }
        return;
    }
    const int s = pc.idx;
    const int64_t pair_id = (int64_t)b * p.hkv + j;
    const __amdgpu_buffer_rsrc_t rs_o = raw_rsrc(p.part_o + pc.base * p.g * kHeadDim);
    const __amdgpu_buffer_rsrc_t rs_ml = raw_rsrc(p.part_ml + pc.base * p.g);
    if (head_ok) {
#pragma unroll
        for (int n = 0; n < 8; n++)
            __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4_t, O[n]), rs_o,
                                                   (uint32_t)((((s * 8 + n) * 4 + G) * p.g + r) * 16), 0, kCoherent);
        if (G == 0) {
            const u32x2_t ml = {__float_as_uint(M), __float_as_uint(L)};
            __builtin_amdgcn_raw_buffer_store_b64(ml, rs_ml, (uint32_t)((s * p.g + r) * 8), 0, kCoherent);
        }
    }
    // every store of the wave has completed (device-coherent) before the ticket
    __builtin_amdgcn_s_waitcnt(0);
    int last = 0;
    if (lane == 0)
        last = __hip_atomic_fetch_add(&p.tickets[pair_id], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
               pc.n_parts - 1;
    if (!__builtin_amdgcn_readfirstlane(last))
        return;
    if (head_ok) {
        float Mf, Lf;
        f32x4_t F[8];
        fold_partials<8>(rs_o, rs_ml, pc.n_parts, p.g, G, r, 0, 1, F, Mf, Lf);
        const float inv = 1.0f / Lf;
#pragma unroll
        for (int n = 0; n < 8; n++)
            store_out_col(orow, n, F[n], inv);
        if (p.lse && G == 0)
            p.lse[out_row] = (Mf + log2f(Lf)) * kLn2;
    }
    if (lane == 0)     // ready for the next call
        __hip_atomic_store(&p.tickets[pair_id], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Split s of (b, j) under tokens_per_split splits: tokens [s*tps, min(ctx,
// (s+1)*tps)); its partial is slot s of the pair's n_splits slots.
__device__ __forceinline__ Piece split_piece(const AttnParams &p, int b, int j, int s, int ctx)
{
    Piece pc;
    pc.t_begin = s * p.tps;
    pc.n_tok = min(ctx, pc.t_begin + p.tps) - pc.t_begin;
    pc.idx = s;
    pc.n_parts = (ctx + p.tps - 1) / p.tps;
    pc.base = ((int64_t)b * p.hkv + j) * p.n_splits;
    return pc;
}

// ------------------------------------------------------- the split schedule
//
// Direct: workgroup id = (s * batch + b) * hkv + j owns split s of (b, j);
// the grid covers every split the longest possible sequence could have, and
// workgroups past their sequence's end leave at once.
//
// Planned (4-wave shape, for batches whose lengths the host does not know):
// the grid is twice the workgroups the chip holds at once, and every
// workgroup derives the same list of splits from the context lengths:
//   1. the full splits (tps tokens) level by level: level s holds split s of
//      every sequence with more than s full splits, in sequence order;
//   2. every sequence's shorter last split, in sequence order;
// each entry for all KV heads (KV head fastest).  Workgroup w takes entries
// w, w + grid, ...  No workgroup is spent on a split that does not exist,
// the short pieces come last, and the splits of one (sequence, KV head)
// pair lie far apart in the list, so they do not all finish (and take their
// tickets) at once.  A split's arithmetic does not depend on which workgroup
// runs it, so both schedules give the same bits.

// Count of n < limit with pre[n + 1] <= k, for a nondecreasing table pre:
// the row whose range [pre[n], pre[n + 1]) holds k.
__device__ __forceinline__ int row_of(const int32_t *pre, int limit, int k)
{
    int n = 0;
    for (int n0 = 0; n0 < limit; n0 += 64) {
        const int i = n0 + (thread_index() & 63);
        const uint64_t le = __ballot(i < limit && pre[i + 1] <= k);
        n += __popcll(le);
        if (le != ~0ull)
            break;
    }
    return __builtin_amdgcn_readfirstlane(n);
}

// The i-th (from 0) sequence, in sequence order, with more than s full splits
// (a context of at least (s + 1) * tps tokens).
__device__ __forceinline__ int nth_longer(const int32_t *sm_ctx, int batch, int tps, int s, int i)
{
    const int lane = thread_index() & 63;
    const int need = (s + 1) * tps;
    for (int b0 = 0; b0 < batch; b0 += 64) {
        const int b = b0 + lane;
        const uint64_t m = __ballot(b < batch && sm_ctx[b] >= need);
        const int cnt = __popcll(m);
        if (i < cnt) {
            const int below = __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                                         __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
            const uint64_t hit = __ballot(((m >> lane) & 1) && below == i);
            return __builtin_amdgcn_readfirstlane(b0 + __builtin_ctzll(hit));
        }
        i -= cnt;
    }
    return 0;     // not reached for an entry of the list
}

// Inclusive prefix sum over the 64 lanes of a wave (row shifts within each
// 16-lane row, then the row totals broadcast to the rows above).
__device__ __forceinline__ int wave_inclusive_scan(int x)
{
    x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xf, 0xf, true);     // row_shr:1
    x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xf, 0xf, true);     // row_shr:2
    x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xf, 0xf, true);     // row_shr:4
    x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xf, 0xf, true);     // row_shr:8
    x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xa, 0xf, false);    // row_bcast:15
    x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xc, 0xf, false);    // row_bcast:31
    return x;
}

struct Plan {
    int n_full;     // full splits over all sequences
    int n_last;     // shorter last splits
};

// True when every sequence has the context length c0 (each wave decides for
// itself; all waves reach the same answer).
__device__ __forceinline__ bool all_lengths_equal(const AttnParams &p, int c0)
{
    const int lane = thread_index() & 63;
    for (int b0 = 0; b0 < p.batch; b0 += 64) {
        const int b = b0 + lane;
        const int c = b < p.batch ? context_len(p, b) : c0;
        if (__ballot(c != c0))
            return false;
    }
    return true;
}

// The list's tables, from the context lengths; wave 0 of every workgroup
// builds its own copy in LDS, 64 entries at a time:
//   sm_ctx[b]    context length of sequence b (clamped to the host bound);
//   sm_last[b]   shorter last splits of the sequences before b (b <= batch);
//   sm_level[s]  full splits in the levels before s (s <= n_splits).  Level s
//                has C(s) = #{b : nfull_b > s} entries, taken from the
//                histogram of nfull: C(s) = #{nfull >= 1} - #{1 <= nfull <= s}.
__device__ __forceinline__ Plan build_plan(const AttnParams &p, int32_t *sm_ctx, int32_t *sm_last,
                                           int32_t *sm_level)
{
    const int n_lv = p.n_splits;     // nfull_b <= n_splits < kPlanMaxBatch (host)
    if (threadIdx.x < 64) {
        const int lane = threadIdx.x;
        for (int s0 = 0; s0 <= n_lv; s0 += 64)
            if (s0 + lane <= n_lv)
                sm_level[s0 + lane] = 0;
        __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "workgroup");
        int n_last = 0, n_long = 0;
        for (int b0 = 0; b0 < p.batch; b0 += 64) {
            const int b = b0 + lane;
            const int c = b < p.batch ? context_len(p, b) : 0;
            const int f = c / p.tps;
            const uint64_t has_last = __ballot(c - f * p.tps > 0);
            if (b < p.batch) {
                sm_ctx[b] = c;
                sm_last[b] = n_last + (int)__builtin_amdgcn_mbcnt_hi(
                                          (uint32_t)(has_last >> 32),
                                          __builtin_amdgcn_mbcnt_lo((uint32_t)has_last, 0u));
            }
            if (f > 0)
                atomicAdd(&sm_level[f], 1);
            n_last += __popcll(has_last);
            n_long += __popcll(__ballot(f > 0));
        }
        if (lane == 0)
            sm_last[p.batch] = n_last;
        __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "workgroup");
        int below = 0, acc = 0;
        for (int s0 = 0; s0 <= n_lv; s0 += 64) {
            const int s = s0 + lane;
            const int h = s <= n_lv ? sm_level[s] : 0;
            const int hs = wave_inclusive_scan(h);
            const int cnt = n_long - (below + hs);          // C(s)
            const int cs = wave_inclusive_scan(cnt);
            if (s <= n_lv)
                sm_level[s] = acc + cs - cnt;
            below += __builtin_amdgcn_readlane(hs, 63);
            acc += __builtin_amdgcn_readlane(cs, 63);
        }
    }
    __syncthreads();
    Plan plan;
    plan.n_full = __builtin_amdgcn_readfirstlane(sm_level[n_lv]);
    plan.n_last = __builtin_amdgcn_readfirstlane(sm_last[p.batch]);
    return plan;
}

// Page-balanced schedule (4-wave shape, automatic split length): the pages
// of each KV head's sequences, taken in sequence order, form one list of T
// pages, cut into equal ranges on the device from the lengths, so every
// compute unit gets the same number of pages whatever the length mix.  A
// range that covers parts of several sequences yields one piece per
// sequence; the pieces of (b, j) come from ranges k_first(b) .. k_last(b), and
// piece k of sequence b is partial slot k + b of KV head j (unique: for two
// pieces (k, b) and (k', b') with k + b = k' + b' the ranges and sequences
// would have to overlap in opposite orders).  Two granularities:
//   - one range per wave (items (range, KV head), KV head fastest; wave w of
//     workgroup x takes items x * WAVES + w, + grid * WAVES, ...): no wave
//     waits for another, and every piece is published by the wave alone.
//     Taken when a wave's range is at least kWaveRangePages long, so that
//     the pieces (one publish each, and a fold over them) are few against
//     the pages;
//   - otherwise one range (chunk) per workgroup, whose waves share each
//     piece's pages and merge them in LDS (shorter ranges would cut most
//     sequences into many published pieces).
// The ranges depend only on the lengths, so the result does not depend on
// timing.
constexpr int kMinChunkPages = 16;
constexpr int kMinWavePages = 4;
constexpr int kWaveRangePages = 64;

__device__ __forceinline__ void balanced_schedule_table(const AttnParams &p, int32_t *sm_pre)
{
    // sm_pre[b] = pages of the sequences before b (clamped lengths), b <= batch
    if (threadIdx.x < 64) {
        const int lane = threadIdx.x;
        int carry = 0;
        for (int b0 = 0; b0 < p.batch; b0 += 64) {
            const int b = b0 + lane;
            const int pages = b < p.batch ? (context_len(p, b) + kPageSize - 1) / kPageSize : 0;
            const int incl = wave_inclusive_scan(pages);
            if (b < p.batch)
                sm_pre[b] = carry + incl - pages;
            carry += __builtin_amdgcn_readlane(incl, 63);
        }
        if (lane == 0)
            sm_pre[p.batch] = carry;
    }
    __syncthreads();
}

// Piece (range k of W pages, sequence b) of KV head j, for a range [g0, g1)
// of the list that overlaps sequence b's pages [pb0, pb1) (non-empty).
__device__ __forceinline__ Piece range_piece(const AttnParams &p, int b, int j, int k, int W, int g0, int g1,
                                             int pb0, int pb1)
{
    const int lo = max(g0, pb0) - pb0;     // local pages [lo, hi)
    const int hi = min(g1, pb1) - pb0;
    const int k_first = pb0 / W;
    const int k_last = (pb1 - 1) / W;
    Piece pc;
    pc.t_begin = lo * kPageSize;
    pc.n_tok = min(context_len(p, b), hi * kPageSize) - pc.t_begin;
    pc.idx = k - k_first;
    pc.n_parts = k_last - k_first + 1;
    pc.base = (int64_t)j * p.slots_per_head + k_first + b;
    return pc;
}

// One range per wave.  wpt: LDS for WAVES x kMaxChunkPages page-table
// entries (one slice per wave).
template <bool MIXED, int WAVES>
__device__ __forceinline__ void balanced_waves(const AttnParams &p, const int32_t *sm_pre, int T, int W,
                                               uint32_t *sm_wpt)
{
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int n_ranges = min((T + W - 1) / W, p.slots_per_head - p.batch);     // host bound holds it
    uint32_t *wpt = sm_wpt + wave * kMaxChunkPages;
    const int n_items = n_ranges * p.hkv;
    for (int it = (int)blockIdx.x * WAVES + wave; it < n_items; it += (int)gridDim.x * WAVES) {
        const int k = it / p.hkv;
        const int j = it - k * p.hkv;
        const int g0 = k * W;
        const int g1 = min(g0 + W, T);
        const int b_first = row_of(sm_pre, p.batch, g0);
        // this range's page-table entries: list page g0 + i at wpt[i]
        const int lane = thread_index() & 63;     // not hoisted out of the item loop
        for (int b = b_first; b < p.batch; b++) {
            const int pb0 = __builtin_amdgcn_readfirstlane(sm_pre[b]);
            if (pb0 >= g1)
                break;
            const int pb1 = __builtin_amdgcn_readfirstlane(sm_pre[b + 1]);
            const int lo = max(g0, pb0);
            const int hi = min(g1, pb1);
            const int32_t *pt = p.page_table + (int64_t)b * p.max_pages + (lo - pb0);
            for (int i = lane; i < hi - lo; i += 64)
                wpt[lo - g0 + i] = (uint32_t)pt[i];
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        for (int b = b_first; b < p.batch; b++) {
            const int pb0 = __builtin_amdgcn_readfirstlane(sm_pre[b]);
            const int pb1 = __builtin_amdgcn_readfirstlane(sm_pre[b + 1]);
            if (pb0 >= g1)
                break;
            if (pb1 <= g0 || pb1 == pb0)
                continue;     // an empty sequence has no piece (its zero output is written by the caller)
            const Piece pc = range_piece(p, b, j, k, W, g0, g1, pb0, pb1);
            attend_wave_piece<MIXED>(p, b, j, pc, wpt + (max(g0, pb0) - g0));
        }
        // the next item rewrites this wave's slice
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
}

// One range (chunk of C pages) per workgroup: items (chunk, KV head), KV head
// fastest; workgroup x takes items x, x + grid, ...
template <bool MIXED, int WAVES>
__device__ __forceinline__ void balanced_chunks(const AttnParams &p, const int32_t *sm_pre, int T, int C,
                                                uint8_t *sm_buf, uint32_t *sm_pt)
{
    const int n_chunks = min((T + C - 1) / C, p.slots_per_head - p.batch);     // host bound holds it
    const int n_items = n_chunks * p.hkv;
    for (int it = blockIdx.x; it < n_items; it += gridDim.x) {
        const int c = it / p.hkv;
        const int j = it - c * p.hkv;
        const int g0 = c * C;
        const int g1 = min(g0 + C, T);
        for (int b = row_of(sm_pre, p.batch, g0); b < p.batch; b++) {
            const int pb0 = __builtin_amdgcn_readfirstlane(sm_pre[b]);
            const int pb1 = __builtin_amdgcn_readfirstlane(sm_pre[b + 1]);
            if (pb0 >= g1)
                break;
            if (pb1 <= g0 || pb1 == pb0)
                continue;     // an empty sequence has no piece (its zero output is written by the caller)
            const Piece pc = range_piece(p, b, j, c, C, g0, g1, pb0, pb1);
            attend_split<MIXED, WAVES>(p, b, j, pc, sm_buf, sm_pt);
        }
    }
}

template <bool MIXED, int WAVES>
__device__ __forceinline__ void balanced_schedule(const AttnParams &p, int32_t *sm_pre, uint8_t *sm_buf,
                                                  uint32_t *sm_pt)
{
    balanced_schedule_table(p, sm_pre);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int T = __builtin_amdgcn_readfirstlane(sm_pre[p.batch]);
    // empty sequences own a zero output
    for (int b = blockIdx.x; b < p.batch; b += gridDim.x)
        if (__builtin_amdgcn_readfirstlane(sm_pre[b + 1] - sm_pre[b]) == 0)
            for (int j = wave; j < p.hkv; j += WAVES)
                zero_pair_output(p, b, j);
    // range lengths: one item per wave (or per workgroup), at least a few
    // pages, at most the page-table slice staged in LDS
    const int n_wg = max(1, (int)gridDim.x / p.hkv);
    const int W = min(kMaxChunkPages, max(kMinWavePages, (T + n_wg * WAVES - 1) / (n_wg * WAVES)));
    if (W >= kWaveRangePages) {
        static_assert(WAVES * kMaxChunkPages * 4 <= merge_bytes<WAVES>(), "page-table slices fit the merge LDS");
        balanced_waves<MIXED, WAVES>(p, sm_pre, T, W, reinterpret_cast<uint32_t *>(sm_buf));
    } else {
        const int C = min(kMaxChunkPages, max(kMinChunkPages, (T + n_wg - 1) / n_wg));
        balanced_chunks<MIXED, WAVES>(p, sm_pre, T, C, sm_buf, sm_pt);
    }
}

// Occupancy: the 4-wave pure-BFP8 kernel is built for three workgroups per CU
// (at most 168 registers per lane); the others for two waves per SIMD.
template <bool MIXED, int WAVES>
__global__ __launch_bounds__(64 * WAVES, (WAVES == 4 && !MIXED) ? 3 : 2) void decode_attn_bfp8_kernel(
    AttnParams p)
{
    // LDS: the wave merge, and the current split's slice of the page table
    __shared__ __attribute__((aligned(16))) uint8_t sm_buf[merge_bytes<WAVES>()];
    __shared__ uint32_t sm_pt[kMaxSplitPages];
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);

    if constexpr (WAVES == 4) {
        if (p.planned) {
            __shared__ int32_t sm_ctx[kPlanMaxBatch], sm_last[kPlanMaxBatch + 1];
            __shared__ int32_t sm_level[kPlanMaxBatch];
            if (p.balanced) {
                balanced_schedule<MIXED, WAVES>(p, sm_last, sm_buf, sm_pt);
                return;
            }
            // equal lengths need no tables: the list is then split-major,
            // entry k = split k / batch of sequence k % batch
            const int c0 = context_len(p, 0);
            const bool uniform = all_lengths_equal(p, c0);
            const int nf0 = c0 / p.tps;
            Plan plan;
            if (uniform) {
                plan.n_full = nf0 * p.batch;
                plan.n_last = c0 > nf0 * p.tps ? p.batch : 0;
            } else {
                plan = build_plan(p, sm_ctx, sm_last, sm_level);
            }
            const int n_items = (plan.n_full + plan.n_last) * p.hkv;
            // empty sequences own a zero output
            for (int b = blockIdx.x; b < p.batch; b += gridDim.x)
                if ((uniform ? c0 : __builtin_amdgcn_readfirstlane(sm_ctx[b])) == 0)
                    for (int j = wave; j < p.hkv; j += WAVES)
                        zero_pair_output(p, b, j);
            for (int it = blockIdx.x; it < n_items; it += gridDim.x) {
                const int k = it / p.hkv;
                const int j = it - k * p.hkv;
                int b, s, ctx;
                if (uniform) {
                    s = k < plan.n_full ? k / p.batch : nf0;
                    b = k < plan.n_full ? k - s * p.batch : k - plan.n_full;
                    ctx = c0;
                } else {
                    if (k < plan.n_full) {
                        s = row_of(sm_level, p.n_splits, k);
                        b = nth_longer(sm_ctx, p.batch, p.tps, s,
                                       k - __builtin_amdgcn_readfirstlane(sm_level[s]));
                    } else {
                        b = row_of(sm_last, p.batch, k - plan.n_full);
                    }
                    ctx = __builtin_amdgcn_readfirstlane(sm_ctx[b]);
                    if (k >= plan.n_full)
                        s = ctx / p.tps;
                }
                attend_split<MIXED, WAVES>(p, b, j, split_piece(p, b, j, s, ctx), sm_buf, sm_pt);
            }
            return;
        }
    }

    const int id = blockIdx.x;
    const int j = id % p.hkv;
    const int b = (id / p.hkv) % p.batch;
    const int s = id / (p.hkv * p.batch);
    const int ctx = context_len(p, b);
    if (s * p.tps >= ctx) {
        // empty split; split 0 of an empty sequence owns its (zero) output
        if (s == 0 && wave == 0)
            zero_pair_output(p, b, j);
        return;
    }
    attend_split<MIXED, WAVES>(p, b, j, split_piece(p, b, j, s, ctx), sm_buf, sm_pt);
}

// Occupancy of the 4-wave kernel: workgroups per CU and CUs, queried once
// per device and variant (0 workgroups on failure).
struct Residency {
    int per_cu, cus;
};

Residency resident_workgroups(bool mixed)
{
    constexpr int kMaxDevices = 64;
    static std::atomic<int> cache[kMaxDevices][2][2];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices)
        return Residency{0, 0};
    Residency r{cache[dev][mixed][0].load(std::memory_order_relaxed),
                cache[dev][mixed][1].load(std::memory_order_relaxed)};
    if (r.per_cu > 0 && r.cus > 0)
        return r;
    const hipError_t e =
        mixed ? hipOccupancyMaxActiveBlocksPerMultiprocessor(&r.per_cu, decode_attn_bfp8_kernel<true, 4>, 256, 0)
              : hipOccupancyMaxActiveBlocksPerMultiprocessor(&r.per_cu, decode_attn_bfp8_kernel<false, 4>, 256, 0);
    if (e != hipSuccess ||
        hipDeviceGetAttribute(&r.cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
        return Residency{0, 0};
    cache[dev][mixed][0].store(r.per_cu, std::memory_order_relaxed);
    cache[dev][mixed][1].store(r.cus, std::memory_order_relaxed);
    return r;
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
    p.max_ctx = a.max_ctx;
    p.planned = a.planned;
    p.balanced = a.balanced;
    p.slots_per_head = a.slots_per_head;
    p.key_interleaved = a.key_interleaved;
    p.scale_log2 = a.scale * kLog2e;
    p.tickets = a.tickets;
    p.part_ml = a.part_ml;
    p.part_o = a.part_o;
    const int64_t blocks = (int64_t)a.batch * a.hkv * a.n_splits;
    const bool mixed = a.k_bf16 != nullptr && a.v_bf16 != nullptr;
    dim3 grid((unsigned)blocks);
    if (a.planned) {
        const Residency r = resident_workgroups(mixed);
        const int64_t resident = (int64_t)r.per_cu * r.cus;
        if (resident < 1)
            return -1;
        // balanced: one chunk per workgroup, at most two workgroups per CU
        // (a third per CU means shorter chunks, so more sequences cut into
        // pieces that each pay a merge; measured slower), and a whole number
        // of workgroups per CU; split schedule: two rounds of the resident
        // workgroups over the split list
        const int64_t balanced_grid = (int64_t)std::min(r.per_cu, 2) * r.cus;
        grid = a.balanced ? dim3((unsigned)std::min<int64_t>(balanced_grid, kBalancedGridCap))
                          : dim3((unsigned)std::min(blocks, 2 * resident));
    }
    if (a.waves == 8) {
        if (mixed)
            hipLaunchKernelGGL((decode_attn_bfp8_kernel<true, 8>), grid, dim3(512), 0, stream, p);
        else
            hipLaunchKernelGGL((decode_attn_bfp8_kernel<false, 8>), grid, dim3(512), 0, stream, p);
    } else {
        if (mixed)
            hipLaunchKernelGGL((decode_attn_bfp8_kernel<true, 4>), grid, dim3(256), 0, stream, p);
        else
            hipLaunchKernelGGL((decode_attn_bfp8_kernel<false, 4>), grid, dim3(256), 0, stream, p);
    }
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

// ------------------------------------------- scratch of the no-alloc entry

static __device__ __align__(256) uint8_t scratch[kScratchBytes];

__global__ void clear_words_kernel(uint32_t *p, int n)
{
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x)
        p[i] = 0u;
}

int noalloc_scratch(hipStream_t stream, uint8_t **base)
{
    constexpr int kMaxDevices = 64;
    static std::atomic<uint8_t *> ptrs[kMaxDevices];
    static std::mutex init_lock;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices)
        return -1;
    uint8_t *ptr = ptrs[dev].load(std::memory_order_acquire);
    if (ptr == nullptr) {
        std::lock_guard<std::mutex> guard(init_lock);
        ptr = ptrs[dev].load(std::memory_order_acquire);
        if (ptr == nullptr) {
            // the array's name is a host-side stand-in: take this device's
            // address of it once, with the device current, and use only that
            void *addr = nullptr;
            if (hipGetSymbolAddress(&addr, HIP_SYMBOL(scratch)) != hipSuccess || addr == nullptr)
                return -1;
            ptr = static_cast<uint8_t *>(addr);
            // the tickets must start at zero (every call leaves its own at zero)
            hipLaunchKernelGGL(clear_words_kernel, dim3(64), dim3(256), 0, stream,
                               reinterpret_cast<uint32_t *>(ptr), (int)(kScratchTicketBytes / 4));
            if (hipGetLastError() != hipSuccess)
                return -1;
            ptrs[dev].store(ptr, std::memory_order_release);
        }
    }
    *base = ptr;
    return 0;
}

}  // namespace hma
