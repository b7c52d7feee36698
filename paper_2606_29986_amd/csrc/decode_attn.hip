// decode_attn.hip -- fused BFP8 paged single-token GQA decode attention (gfx950).
//
// The paper reconstructs BFP8 pages to BF16 inline, inside the paged-attention
// read (Sec. 3.3, Fig. 2).  This kernel does the same on CDNA4: mantissa and
// exponent bytes are streamed from HBM once, decoded to exact BF16 in
// registers on the VALU, and fed to the matrix cores.
//
// Work decomposition.  One workgroup (4 waves) owns one (sequence b, KV head
// j, split s): the tokens [s*tps, min(ctx_b, (s+1)*tps)).  A wave walks the
// split in chunks of 32 tokens (two pages), chunk c going to wave c % 4.
//
// Per chunk, with g = Hq/Hkv query heads padded to 16:
//   QK : S[16 tok][16 heads] = K_page[16 tok][128] . Q^T[128][16]
//        four v_mfma_f32_16x16x32_bf16 per page.  Lane (G = lane/16, r =
//        lane%16) feeds token r of the page with channels {16G..16G+15} and
//        {64+16G..64+16G+15} (two 16-channel blocks, one exponent each) and
//        Q^T's column r (head j*g + r) with the same channels; the order of
//        the contraction index is free as long as both operands agree.
//   softmax : online, in the log2 domain; the C layout leaves lane (G, r)
//        with head r and tokens {4G..4G+3} of each page.
//   PV : O^T[128][16 heads] += V^T[128][32 tok] . P^T[32 tok][16 heads]
//        eight MFMA pairs (n = 0..7; P^T as BF16 high + low parts, so the
//        softmax weights keep ~16 bits); row r of MFMA n is channel 8r + n, so lane
//        (G, r) needs 8 consecutive bytes (channels 8r..8r+7, one exponent
//        block) of each of its 8 tokens, and P^T is exactly the lane's own
//        softmax output.  The accumulator leaves lane (G, r) with head r,
//        channels 32G..32G+31 -- the same head as its softmax state, so the
//        online rescale needs no data movement.
// The four waves are merged through LDS; with more than one split, each
// workgroup writes (max, sum, weighted values) to the workspace and the last
// workgroup of (b, j) to arrive (atomic ticket) merges them by log-sum-exp
// and writes the BF16 output.  A BF16-tagged page is read from the BF16 pool
// and enters the same MFMAs.
#include "hma_device.h"
#include "hma_internal.h"

namespace hma {

constexpr int kAttnWaves = 4;
constexpr int kChunk = 2 * kPageSize;        // tokens per step
constexpr float kLn2 = 0.69314718055994531f;
constexpr float kLog2e = 1.44269504088896341f;

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

__device__ __forceinline__ bf16x8_t as_bf16x8(u32x4_t v)
{
    return __builtin_bit_cast(bf16x8_t, v);
}

__device__ __forceinline__ f32x4_t mfma_bf16(u32x4_t a, u32x4_t b, f32x4_t c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(a), as_bf16x8(b), c, 0, 0, 0);
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

// In-chunk token index of lane group G's token slot q (0..7).
__device__ __forceinline__ int slot_token(int G, int q)
{
    return kPageSize * (q >> 2) + 4 * G + (q & 3);
}

// Channel of the k-th 8-element group of lane group G in the QK contraction.
__device__ __forceinline__ int qk_channel(int G, int kk)
{
    return (kk >> 1) * 64 + 16 * G + (kk & 1) * 8;
}

// Write 32 channels of one head as BF16: o_acc[n][i] is channel 32G + 8i + n.
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

__global__ __launch_bounds__(64 * kAttnWaves, 2) void decode_attn_bfp8_kernel(AttnParams p)
{
    const int id = blockIdx.x;
    const int j = id % p.hkv;
    const int b = (id / p.hkv) % p.batch;
    const int s = id / (p.hkv * p.batch);
    const int ctx = p.ctx_lens[b];
    // the wave index is uniform: page-table reads and page-type branches then
    // compile to scalar loads and scalar branches
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
    const int t_end = min(ctx, t_begin + p.tps);
    const int n_split_b = (ctx + p.tps - 1) / p.tps;
    const bool bf16_pools = p.k_bf16 != nullptr && p.v_bf16 != nullptr;

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

    float m_run = -INFINITY;     // running max of scaled scores (log2 units), head r
    float l_run = 0.0f;          // this lane's share of the running sum, head r
    f32x4_t O[8];
#pragma unroll
    for (int n = 0; n < 8; n++)
        O[n] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    const int32_t *pt = p.page_table + (int64_t)b * p.max_pages;
    const int n_chunks = (t_end - t_begin + kChunk - 1) / kChunk;

    // per-lane byte offsets inside a (page, head) tile; the tile base is uniform,
    // so every load is a scalar base + 32-bit lane offset
    const uint32_t off_km0 = r * kHeadDim + 16 * G;          // K mantissa, block G
    const uint32_t off_km1 = off_km0 + 64;                     // K mantissa, block 4 + G
    const uint32_t off_ke = r * kExpPerRow;                    // K exponent row of token r
    const uint32_t off_vm = 4 * G * kHeadDim + 8 * r;          // V mantissa, token 4G (+i rows)
    const uint32_t off_ve = 4 * G * kExpPerRow + (r >> 1);     // V exponent, token 4G (+i rows)

    for (int ci = wave; ci < n_chunks; ci += kAttnWaves) {
        const int tok0 = t_begin + ci * kChunk;
        const int nval = min(kChunk, t_end - tok0);
        const int lp0 = tok0 / kPageSize;
        uint32_t ent[2];
        ent[0] = (uint32_t)pt[lp0];
        // page 1 of a chunk holding <= 16 tokens does not exist: reuse page 0 (fully masked)
        const uint32_t ent1 = (uint32_t)pt[min(lp0 + 1, p.max_pages - 1)];
        ent[1] = nval > kPageSize ? ent1 : ent[0];
        bool tag[2];
#pragma unroll
        for (int pg = 0; pg < 2; pg++)
            tag[pg] = bf16_pools && (ent[pg] & kTagBf16);

        // ---- issue every load of the chunk
        u32x4_t kraw[2][4];      // BFP8: [0..1] mantissa words, [2].xy exponent row; BF16: 4 x 8 values
        u32x4_t vraw[2][4];      // per slot: BFP8: .xy mantissa, .z exponent byte; BF16: 8 values
#pragma unroll
        for (int pg = 0; pg < 2; pg++) {
            const int64_t tile = (int64_t)(ent[pg] & kIdMask) * p.hkv + j;
            if (tag[pg]) {
                const char *kt = reinterpret_cast<const char *>(p.k_bf16 + tile * kTileMant);
                const char *vt = reinterpret_cast<const char *>(p.v_bf16 + tile * kTileMant);
#pragma unroll
                for (int kk = 0; kk < 4; kk++)
                    kraw[pg][kk] = *reinterpret_cast<const u32x4_t *>(
                        kt + 2 * (r * kHeadDim + qk_channel(G, kk)));
#pragma unroll
                for (int i = 0; i < 4; i++)
                    vraw[pg][i] = *reinterpret_cast<const u32x4_t *>(vt + 2 * (off_vm + i * kHeadDim));
            } else {
                const uint8_t *kt = p.k_mant + tile * kTileMant;
                const uint8_t *ke = p.k_exp + tile * kTileExp;
                const uint8_t *vt = p.v_mant + tile * kTileMant;
                const uint8_t *ve = p.v_exp + tile * kTileExp;
                kraw[pg][0] = *reinterpret_cast<const u32x4_t *>(kt + off_km0);
                kraw[pg][1] = *reinterpret_cast<const u32x4_t *>(kt + off_km1);
                const u32x2_t kex = *reinterpret_cast<const u32x2_t *>(ke + off_ke);
                kraw[pg][2] = u32x4_t{kex.x, kex.y, 0u, 0u};
#pragma unroll
                for (int i = 0; i < 4; i++) {
                    const u32x2_t vm = *reinterpret_cast<const u32x2_t *>(vt + off_vm + i * kHeadDim);
                    const uint32_t vx = ve[off_ve + i * kExpPerRow];
                    vraw[pg][i] = u32x4_t{vm.x, vm.y, vx, 0u};
                }
            }
        }

        // ---- QK^T on the matrix cores
        f32x4_t S[2];
#pragma unroll
        for (int pg = 0; pg < 2; pg++) {
            u32x4_t A[4];
            if (tag[pg]) {
#pragma unroll
                for (int kk = 0; kk < 4; kk++)
                    A[kk] = kraw[pg][kk];
            } else {
                const int esa = (int)((kraw[pg][2].x >> (8 * G)) & 0xFFu) - kExpBias;
                const int esb = (int)((kraw[pg][2].y >> (8 * G)) & 0xFFu) - kExpBias;
                bfp8_block_to_bf16(kraw[pg][0], esa, A[0], A[1]);
                bfp8_block_to_bf16(kraw[pg][1], esb, A[2], A[3]);
            }
            f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kk = 0; kk < 4; kk++)
                acc = mfma_bf16(A[kk], qB[kk], acc);
            S[pg] = acc;
        }

        // ---- online softmax over the chunk (head r, slots q = 4 pg + i)
        float x[8];
#pragma unroll
        for (int q = 0; q < 8; q++)
            x[q] = S[q >> 2][q & 3] * p.scale_log2;
        if (nval < kChunk) {
#pragma unroll
            for (int q = 0; q < 8; q++)
                if (slot_token(G, q) >= nval)
                    x[q] = -INFINITY;
        }
        float cmax = x[0];
#pragma unroll
        for (int q = 1; q < 8; q++)
            cmax = fmaxf(cmax, x[q]);
        cmax = fmaxf(cmax, __shfl_xor(cmax, 16));
        cmax = fmaxf(cmax, __shfl_xor(cmax, 32));
        const float m_new = fmaxf(m_run, cmax);
        const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
        m_run = m_new;
        // P^T operand split into BF16 high and low parts (p = hi + lo to ~2^-17
        // relative): two MFMAs keep the weights at near-FP32 precision
        u32x4_t Phi, Plo;
        float psum = 0.0f;
        {
            uint32_t hi[4], lo[4];
#pragma unroll
            for (int k = 0; k < 4; k++) {
                const float p0 = __builtin_amdgcn_exp2f(x[2 * k] - m_new);
                const float p1 = __builtin_amdgcn_exp2f(x[2 * k + 1] - m_new);
                hi[k] = pack_bf16_rne(p0, p1);
                const float h0 = __uint_as_float(hi[k] << 16);
                const float h1 = __uint_as_float(hi[k] & 0xFFFF0000u);
                lo[k] = pack_bf16_rne(p0 - h0, p1 - h1);
                psum += p0 + p1;
            }
            Phi = u32x4_t{hi[0], hi[1], hi[2], hi[3]};
            Plo = u32x4_t{lo[0], lo[1], lo[2], lo[3]};
        }
        l_run = l_run * alpha + psum;
        if (__any(alpha != 1.0f)) {
#pragma unroll
            for (int n = 0; n < 8; n++)
                O[n] *= alpha;
        }

        // ---- V^T operands: Av[n] = channel 8r + n of slots 0..7, decoded
        u32x4_t Av[8];
#pragma unroll
        for (int pg = 0; pg < 2; pg++) {
#pragma unroll
            for (int k2 = 0; k2 < 2; k2++) {
                const u32x4_t va = vraw[pg][2 * k2];
                const u32x4_t vb = vraw[pg][2 * k2 + 1];
                uint32_t pr[8];
                if (tag[pg]) {
#pragma unroll
                    for (int n = 0; n < 8; n++) {
                        const uint32_t wa = (n >> 1) == 0 ? va.x : (n >> 1) == 1 ? va.y : (n >> 1) == 2 ? va.z : va.w;
                        const uint32_t wb = (n >> 1) == 0 ? vb.x : (n >> 1) == 1 ? vb.y : (n >> 1) == 2 ? vb.z : vb.w;
                        pr[n] = __builtin_amdgcn_perm(wb, wa, (n & 1) ? kPermHiHalves : kPermLoHalves);
                    }
                } else {
                    const int esa = (int)va.z - kExpBias;
                    const int esb = (int)vb.z - kExpBias;
#pragma unroll
                    for (int d = 0; d < 2; d++) {
                        const uint32_t wa = d ? va.y : va.x;
                        const uint32_t wb = d ? vb.y : vb.x;
                        const uint32_t ma = magnitudes(wa);
                        const uint32_t mb = magnitudes(wb);
#pragma unroll
                        for (int n4 = 0; n4 < 4; n4++)
                            pr[4 * d + n4] = pack_bf16_signed(bfp8_mag_f32(ma, n4, esa),
                                                              bfp8_mag_f32(mb, n4, esb),
                                                              wa, n4, wb, n4);
                    }
                }
                // slots 4 pg + 2 k2 (low half) and 4 pg + 2 k2 + 1 (high half)
                const int pair = 2 * pg + k2;
#pragma unroll
                for (int n = 0; n < 8; n++) {
                    if (pair == 0) Av[n].x = pr[n];
                    else if (pair == 1) Av[n].y = pr[n];
                    else if (pair == 2) Av[n].z = pr[n];
                    else Av[n].w = pr[n];
                }
            }
        }
        if (nval < kChunk) {
            // slots past the context may hold anything: zero them (p is 0 there)
            u32x4_t msk;
#pragma unroll
            for (int k = 0; k < 4; k++) {
                const uint32_t lo = slot_token(G, 2 * k) < nval ? 0x0000FFFFu : 0u;
                const uint32_t hi = slot_token(G, 2 * k + 1) < nval ? 0xFFFF0000u : 0u;
                msk[k] = lo | hi;
            }
#pragma unroll
            for (int n = 0; n < 8; n++)
                Av[n] &= msk;
        }
#pragma unroll
        for (int n = 0; n < 8; n++) {
            O[n] = mfma_bf16(Av[n], Phi, O[n]);
            O[n] = mfma_bf16(Av[n], Plo, O[n]);
        }
    }

    // ---- merge the four waves of the workgroup through LDS
    l_run += __shfl_xor(l_run, 16);
    l_run += __shfl_xor(l_run, 32);
    __shared__ float sm_m[kAttnWaves][16];
    __shared__ float sm_l[kAttnWaves][16];
    __shared__ float sm_o[kAttnWaves - 1][32][64];
    if (wave > 0) {
        if (G == 0) {
            sm_m[wave][r] = m_run;
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

    float M = m_run;
#pragma unroll
    for (int w = 1; w < kAttnWaves; w++)
        M = fmaxf(M, sm_m[w][r]);
    float L;
    {
        const float a0 = __builtin_amdgcn_exp2f(m_run - M);
        L = l_run * a0;
#pragma unroll
        for (int n = 0; n < 8; n++)
            O[n] *= a0;
#pragma unroll
        for (int w = 1; w < kAttnWaves; w++) {
            const float aw = __builtin_amdgcn_exp2f(sm_m[w][r] - M);
            L += aw * sm_l[w][r];
#pragma unroll
            for (int n = 0; n < 8; n++)
#pragma unroll
                for (int i = 0; i < 4; i++)
                    O[n][i] += aw * sm_o[w - 1][8 * i + n][lane];
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

    // ---- several splits: publish this split's partial, last arrival merges
    const int64_t pair_id = (int64_t)b * p.hkv + j;
    if (head_ok) {
        float *po = p.part_o + ((pair_id * p.n_splits + s) * p.g + r) * kHeadDim + 32 * G;
#pragma unroll
        for (int i = 0; i < 4; i++) {
            *reinterpret_cast<f32x4_t *>(po + 8 * i) = f32x4_t{O[0][i], O[1][i], O[2][i], O[3][i]};
            *reinterpret_cast<f32x4_t *>(po + 8 * i + 4) = f32x4_t{O[4][i], O[5][i], O[6][i], O[7][i]};
        }
        if (G == 0)
            p.part_ml[(pair_id * p.n_splits + s) * p.g + r] = make_float2(M, L);
    }
    __threadfence();
    int last = 0;
    if (lane == 0)
        last = atomicAdd(&p.tickets[pair_id], 1) == n_split_b - 1;
    last = __shfl(last, 0);
    if (!last)
        return;
    __threadfence();

    if (head_ok) {
        const float2 *ml = p.part_ml + pair_id * p.n_splits * p.g + r;
        float Mx = -INFINITY;
        for (int t = 0; t < n_split_b; t++)
            Mx = fmaxf(Mx, ml[t * p.g].x);
        float Lt = 0.0f;
        f32x4_t acc[8];
#pragma unroll
        for (int n = 0; n < 8; n++)
            acc[n] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        for (int t = 0; t < n_split_b; t++) {
            const float2 v = ml[t * p.g];
            const float a = __builtin_amdgcn_exp2f(v.x - Mx);
            Lt += a * v.y;
            const float *po = p.part_o + ((pair_id * p.n_splits + t) * p.g + r) * kHeadDim + 32 * G;
#pragma unroll
            for (int i = 0; i < 4; i++) {
                const f32x4_t lo = *reinterpret_cast<const f32x4_t *>(po + 8 * i);
                const f32x4_t hi = *reinterpret_cast<const f32x4_t *>(po + 8 * i + 4);
                acc[0][i] += a * lo[0];
                acc[1][i] += a * lo[1];
                acc[2][i] += a * lo[2];
                acc[3][i] += a * lo[3];
                acc[4][i] += a * hi[0];
                acc[5][i] += a * hi[1];
                acc[6][i] += a * hi[2];
                acc[7][i] += a * hi[3];
            }
        }
        store_out_row(p.out + out_row * kHeadDim + 32 * G, acc, 1.0f / Lt);
        if (p.lse && G == 0)
            p.lse[out_row] = (Mx + log2f(Lt)) * kLn2;
    }
    if (lane == 0)
        p.tickets[pair_id] = 0;     // ready for the next call
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
    hipLaunchKernelGGL(decode_attn_bfp8_kernel, dim3((unsigned)blocks), dim3(64 * kAttnWaves), 0,
                       stream, p);
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

}  // namespace hma
