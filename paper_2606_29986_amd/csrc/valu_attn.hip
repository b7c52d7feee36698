// valu_attn.hip -- the fused BFP8 decode attention with QK^T and PV on the
// vector ALU instead of the matrix cores: the measured comparison point of
// the choice of matrix cores (a baseline, not for production use).
//
// It computes what hma_decode_attn_bfp8 computes over BFP8 pages (Sec. 3.3:
// the pages decoded exactly in registers inside the paged read, online
// softmax, split-K partials merged by log-sum-exp), with the same decode
// routes, the same split grid (one workgroup of 8 waves per (split, sequence,
// KV head)) and the same byte traffic.  What changes is where the products
// run.  Lane layout per page: lane (token t = lane / 4, quarter q = lane % 4)
// holds token t's K and V for channels [32 q, 32 q + 32).
//   QK: the query slices of the group's (at most 8) heads for the lane's
//       channels stay in registers as BF16 pairs; 16 v_dot2c_f32_bf16 per
//       head, then a sum over the four quarter lanes;
//   softmax: per-page maximum over the 16 token lanes, log2 domain;
//   PV: the wave writes the decoded V page and the page's weights to LDS;
//       lane l accumulates channels 2l, 2l + 1 of every head over the 16
//       tokens (16 FMAs per token).
// The waves' partials are merged in LDS; a second small kernel merges the
// splits.
#include "hma_device.h"
#include "hma_internal.h"

namespace hma {
namespace {

constexpr int kVWaves = 8;
constexpr int kVMaxGroup = 8;
constexpr float kVLn2 = 0.69314718055994531f;

struct ValuParams {
    const uint16_t *q;
    const uint8_t *k_mant, *k_exp, *v_mant, *v_exp;
    const int32_t *page_table;
    const int32_t *ctx;
    float *part_ml;       // [pair][split][g][2]: (max, sum), log2 domain
    float *part_o;        // [pair][split][g][128]: weighted values
    uint16_t *out;
    float *lse;
    int32_t max_pages, max_ctx, batch, hq, hkv, g, tps, n_splits;
    float scale_log2;
};

__device__ __forceinline__ uint32_t rne_bf16(float x)
{
    typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
    typedef float f32x2_t __attribute__((ext_vector_type(2)));
    const bf16x2_t h = __builtin_convertvector(f32x2_t{x, 0.0f}, bf16x2_t);
    return __builtin_bit_cast(uint32_t, h) & 0xFFFFu;
}

__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float acc)
{
    typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a), __builtin_bit_cast(bf16x2_t, b), acc,
                                           false);
}

// Cross-lane steps on DPP and the gfx950 lane swaps (no LDS round trip).
// quad_sum: the sum over the four lanes of a quad, the same in all four.
__device__ __forceinline__ float quad_sum(float x)
{
    x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0xB1, 0xf, 0xf, false));  // [1,0,3,2]
    x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x4E, 0xf, 0xf, false));  // [2,3,0,1]
    return x;
}

// Maximum (or sum) over the 16 quads of the wave, for a value that is the
// same in the four lanes of each quad: lane i of each 8 against lane 7 - i,
// lane i of each 16 against lane 15 - i, then the 16- and 32-lane swaps.
template <bool SUM>
__device__ __forceinline__ float over_quads(float x)
{
    auto op = [](float a, float b) { return SUM ? a + b : fmaxf(a, b); };
    x = op(x, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x141, 0xf, 0xf, false)));
    x = op(x, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x140, 0xf, 0xf, false)));
    const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    x = op(__uint_as_float(a[0]), __uint_as_float(a[1]));
    const auto c = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return op(__uint_as_float(c[0]), __uint_as_float(c[1]));
}

// 32 BFP8 elements of one token (two blocks: words 0-3 block e0, 4-7 e1) to
// 16 BF16 pairs in channel order, on the route the page takes.
__device__ __forceinline__ void decode_row(u32x4_t a, u32x4_t b, uint32_t e0, uint32_t e1, bool fast,
                                           uint32_t (&out)[16])
{
#pragma unroll
    for (int w = 0; w < 8; w++) {
        const uint32_t word = w < 4 ? a[w] : b[w - 4];
        const uint32_t e = w < 4 ? e0 : e1;
        u32x2_t d;
        if (fast)
            d = bfp8_word_to_bf16_fast(word, ((uint32_t)(kExpBias - (int)e) << 7) * 0x00010001u);
        else
            d = bfp8_word_to_bf16(word, (int)e - kExpBias);
        out[2 * w] = d.x;
        out[2 * w + 1] = d.y;
    }
}

// G: query heads held per KV head (1, 2, 4 or 8; the call's group size
// rounded up, the heads past it have zero queries and are not stored).
template <int G>
__global__ __launch_bounds__(64 * kVWaves, 1) void valu_attn_partial_kernel(ValuParams p)
{
    __shared__ uint32_t sm_pt[kMaxSplitPages];
    __shared__ __attribute__((aligned(16))) uint32_t sm_v[kVWaves][kPageSize * kHeadDim / 2];   // BF16 pairs
    __shared__ __attribute__((aligned(16))) float sm_p[kVWaves][kPageSize * kVMaxGroup];
    __shared__ __attribute__((aligned(16))) float sm_o[kVWaves][kVMaxGroup * kHeadDim];
    __shared__ float sm_ml[kVWaves][2 * kVMaxGroup];

    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const int lane = (int)(threadIdx.x & 63);
    const int tq = lane >> 2;     // token slot of the page
    const int qq = lane & 3;      // channel quarter [32 qq, 32 qq + 32)
    const int id = (int)blockIdx.x;
    const int j = id % p.hkv;
    const int b = (id / p.hkv) % p.batch;
    const int s = id / (p.hkv * p.batch);
    const int ctx = min(max(p.ctx[b], 0), p.max_ctx);
    const int t0 = s * p.tps;
    const int n_tok = max(0, min(ctx, t0 + p.tps) - t0);
    const int n_pages = (n_tok + kPageSize - 1) / kPageSize;
    for (int i = (int)threadIdx.x; i < n_pages; i += 64 * kVWaves)
        sm_pt[i] = (uint32_t)p.page_table[(int64_t)b * p.max_pages + t0 / kPageSize + i];

    // query slices: head h of the group, channels [32 qq, 32 qq + 32)
    uint32_t qv[G][16];
#pragma unroll
    for (int h = 0; h < G; h++) {
        // heads past the group read the group's last row and are zeroed
        const u32x4_t *row = reinterpret_cast<const u32x4_t *>(
            p.q + ((int64_t)b * p.hq + j * p.g + min(h, p.g - 1)) * kHeadDim + 32 * qq);
        const uint32_t live = h < p.g ? 0xFFFFFFFFu : 0u;
#pragma unroll
        for (int k = 0; k < 4; k++) {
            const u32x4_t v = row[k];
#pragma unroll
            for (int e = 0; e < 4; e++)
                qv[h][4 * k + e] = v[e] & live;
        }
    }
    __syncthreads();

    float m_run[G], l_lane[G], O[G][2];
#pragma unroll
    for (int h = 0; h < G; h++) {
        m_run[h] = -INFINITY;
        l_lane[h] = 0.0f;
        O[h][0] = 0.0f;
        O[h][1] = 0.0f;
    }

    for (int i = wave; i < n_pages; i += kVWaves) {
        const uint32_t ent = (uint32_t)__builtin_amdgcn_readfirstlane((int)sm_pt[i]) & kIdMask;
        const int64_t tile = (int64_t)ent * p.hkv + j;
        const int nval = min(kPageSize, n_tok - i * kPageSize);     // tokens of this page in the context
        const uint8_t *km = p.k_mant + tile * kTileMant + tq * kHeadDim + 32 * qq;
        const uint8_t *vm = p.v_mant + tile * kTileMant + tq * kHeadDim + 32 * qq;
        const uint8_t *kx = p.k_exp + tile * kTileExp + tq * kExpPerRow + 2 * qq;
        const uint8_t *vx = p.v_exp + tile * kTileExp + tq * kExpPerRow + 2 * qq;
        const u32x4_t ka = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t *>(km));
        const u32x4_t kb = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t *>(km + 16));
        const u32x4_t va = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t *>(vm));
        const u32x4_t vb = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t *>(vm + 16));
        const uint32_t ke0 = kx[0], ke1 = kx[1], ve0 = vx[0], ve1 = vx[1];
        // the page's route, uniform over the wave: the packed route when every
        // block exponent of its K and V lies in [7, 133]
        const bool in_range = ke0 >= 7 && ke0 <= 133 && ke1 >= 7 && ke1 <= 133 && ve0 >= 7 && ve0 <= 133 &&
                              ve1 >= 7 && ve1 <= 133;
        const bool fast = __builtin_amdgcn_ballot_w64(!in_range) == 0;

        // ---- QK^T: token tq, every head, the lane's 32 channels
        uint32_t kp[16];
        decode_row(ka, kb, ke0, ke1, fast, kp);
        float sc[G];
#pragma unroll
        for (int h = 0; h < G; h++) {
            float acc = 0.0f;
#pragma unroll
            for (int d = 0; d < 16; d++)
                acc = dot2_bf16(kp[d], qv[h][d], acc);
            sc[h] = tq < nval ? quad_sum(acc) * p.scale_log2 : -INFINITY;
        }
        // ---- online softmax: page maximum over the 16 token lanes (finite:
        //      the page holds at least one token of the context; on the
        //      first page alpha = 2^-inf = 0 clears the empty state)
        float pw[G], alpha[G];
#pragma unroll
        for (int h = 0; h < G; h++) {
            const float m_new = fmaxf(m_run[h], over_quads<false>(sc[h]));
            alpha[h] = __builtin_amdgcn_exp2f(m_run[h] - m_new);
            pw[h] = __builtin_amdgcn_exp2f(sc[h] - m_new);
            m_run[h] = m_new;
            l_lane[h] = fmaf(l_lane[h], alpha[h], pw[h]);
        }
        // ---- the page's weights and decoded V to LDS (slots past the
        //      context hold anything: their V is zeroed, so 0 * V stays 0)
        uint32_t vp[16];
        decode_row(va, vb, ve0, ve1, fast, vp);
        const uint32_t keep = tq < nval ? 0xFFFFFFFFu : 0u;
#pragma unroll
        for (int d = 0; d < 16; d++)
            vp[d] &= keep;
        uint32_t *vrow = sm_v[wave] + tq * (kHeadDim / 2) + 16 * qq;
#pragma unroll
        for (int k = 0; k < 4; k++)
            reinterpret_cast<u32x4_t *>(vrow)[k] = u32x4_t{vp[4 * k], vp[4 * k + 1], vp[4 * k + 2], vp[4 * k + 3]};
        if (qq == 0) {
#pragma unroll
            for (int h = 0; h < G; h++)
                sm_p[wave][tq * kVMaxGroup + h] = pw[h];
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        // ---- PV: channels 2 lane, 2 lane + 1 of every head
#pragma unroll
        for (int h = 0; h < G; h++) {
            O[h][0] *= alpha[h];
            O[h][1] *= alpha[h];
        }
#pragma unroll 4
        for (int t = 0; t < kPageSize; t++) {
            const uint32_t v2 = sm_v[wave][t * (kHeadDim / 2) + lane];
            const float v0 = __uint_as_float(v2 << 16);
            const float v1 = __uint_as_float(v2 & 0xFFFF0000u);
#pragma unroll
            for (int h = 0; h < G; h++) {
                const float ph = sm_p[wave][t * kVMaxGroup + h];     // same address in every lane
                O[h][0] = fmaf(ph, v0, O[h][0]);
                O[h][1] = fmaf(ph, v1, O[h][1]);
            }
        }
        // the next page rewrites this wave's LDS rows
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }

    // ---- the wave's partial: (max, sum) per head, weighted values per head
    //      and channel; the four quarter lanes of a token hold equal weights,
    //      so the lane sum is four times the token sum (exact)
#pragma unroll
    for (int h = 0; h < G; h++) {
        const float l = over_quads<true>(quad_sum(l_lane[h]));
        if (lane == 0) {
            sm_ml[wave][2 * h] = m_run[h];
            sm_ml[wave][2 * h + 1] = 0.25f * l;
        }
        sm_o[wave][h * kHeadDim + 2 * lane] = O[h][0];
        sm_o[wave][h * kHeadDim + 2 * lane + 1] = O[h][1];
    }
    __syncthreads();
    // ---- merge the waves (thread: head h, channels 2c, 2c + 1) and write
    //      the split's partial
    const int h = (int)threadIdx.x >> 6;      // 8 heads x 64 channel pairs = 512 threads
    const int c = 2 * lane;
    if (h < p.g) {
        float M = -INFINITY;
#pragma unroll
        for (int w = 0; w < kVWaves; w++)
            M = fmaxf(M, sm_ml[w][2 * h]);
        float L = 0.0f, o0 = 0.0f, o1 = 0.0f;
        if (M != -INFINITY) {
#pragma unroll
            for (int w = 0; w < kVWaves; w++) {
                const float cw = __builtin_amdgcn_exp2f(sm_ml[w][2 * h] - M);
                L = fmaf(sm_ml[w][2 * h + 1], cw, L);
                o0 = fmaf(sm_o[w][h * kHeadDim + c], cw, o0);
                o1 = fmaf(sm_o[w][h * kHeadDim + c + 1], cw, o1);
            }
        }
        const int64_t slot = ((int64_t)(b * p.hkv + j) * p.n_splits + s) * p.g + h;
        if (lane == 0) {
            p.part_ml[2 * slot] = M;
            p.part_ml[2 * slot + 1] = L;
        }
        p.part_o[slot * kHeadDim + c] = o0;
        p.part_o[slot * kHeadDim + c + 1] = o1;
    }
}

// One workgroup of 128 threads (one per channel) per (sequence, KV head):
// log-sum-exp merge of the splits' partials, BF16 output and log-sum-exp.
__global__ __launch_bounds__(kHeadDim) void valu_attn_merge_kernel(ValuParams p)
{
    const int pair = (int)blockIdx.x;
    const int b = pair / p.hkv;
    const int j = pair % p.hkv;
    const int c = (int)threadIdx.x;
    for (int h = 0; h < p.g; h++) {
        float M = -INFINITY;
        for (int s = 0; s < p.n_splits; s++)
            M = fmaxf(M, p.part_ml[2 * (((int64_t)pair * p.n_splits + s) * p.g + h)]);
        float L = 0.0f, o = 0.0f;
        if (M != -INFINITY) {
            for (int s = 0; s < p.n_splits; s++) {
                const int64_t slot = ((int64_t)pair * p.n_splits + s) * p.g + h;
                const float cw = __builtin_amdgcn_exp2f(p.part_ml[2 * slot] - M);
                L = fmaf(p.part_ml[2 * slot + 1], cw, L);
                o = fmaf(p.part_o[slot * kHeadDim + c], cw, o);
            }
        }
        const int64_t row = (int64_t)b * p.hq + j * p.g + h;
        p.out[row * kHeadDim + c] = (uint16_t)(L > 0.0f ? rne_bf16(o / L) : 0u);
        if (p.lse && c == 0)
            p.lse[row] = L > 0.0f ? (M + log2f(L)) * kVLn2 : -INFINITY;
    }
}

}  // namespace

int launch_decode_attn_valu(const uint16_t *q, const uint8_t *k_mant, const uint8_t *k_exp, const uint8_t *v_mant,
                            const uint8_t *v_exp, const int32_t *page_table, int32_t max_pages,
                            const int32_t *ctx, int32_t max_ctx, int32_t batch, int32_t hq, int32_t hkv,
                            float scale, int32_t tps, int32_t n_splits, float *part_ml, float *part_o,
                            uint16_t *out, float *lse, hipStream_t stream)
{
    ValuParams p;
    p.q = q;
    p.k_mant = k_mant;
    p.k_exp = k_exp;
    p.v_mant = v_mant;
    p.v_exp = v_exp;
    p.page_table = page_table;
    p.ctx = ctx;
    p.part_ml = part_ml;
    p.part_o = part_o;
    p.out = out;
    p.lse = lse;
    p.max_pages = max_pages;
    p.max_ctx = max_ctx;
    p.batch = batch;
    p.hq = hq;
    p.hkv = hkv;
    p.g = hq / hkv;
    p.tps = tps;
    p.n_splits = n_splits;
    p.scale_log2 = scale * 1.44269504088896341f;
    const int64_t blocks = (int64_t)batch * hkv * n_splits;
    const dim3 grid((unsigned)blocks), block(64 * kVWaves);
    if (p.g <= 1)
        hipLaunchKernelGGL(valu_attn_partial_kernel<1>, grid, block, 0, stream, p);
    else if (p.g <= 2)
        hipLaunchKernelGGL(valu_attn_partial_kernel<2>, grid, block, 0, stream, p);
    else if (p.g <= 4)
        hipLaunchKernelGGL(valu_attn_partial_kernel<4>, grid, block, 0, stream, p);
    else
        hipLaunchKernelGGL(valu_attn_partial_kernel<8>, grid, block, 0, stream, p);
    if (hipGetLastError() != hipSuccess)
        return -1;
    hipLaunchKernelGGL(valu_attn_merge_kernel, dim3((unsigned)(batch * hkv)), dim3(kHeadDim), 0, stream, p);
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

}  // namespace hma
