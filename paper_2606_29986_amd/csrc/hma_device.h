// hma_device.h -- gfx950 device helpers shared by the libhma kernels.
//
// BFP8 element: byte = sign bit 7 | 7-bit magnitude m; block exponent byte E;
// value = (-1)^s * m * 2^(E-133).  Reconstruction (Sec. 3.3 of the paper:
// block-float decode is bit manipulation, not arithmetic) is done per 32-bit
// word of four mantissa bytes:
//   1. mask the sign bits off (one AND per four elements);
//   2. v_cvt_f32_ubyteN turns each magnitude byte into an exact float; the
//      hardware normalisation replaces a count-leading-zeros + shift;
//   3. v_ldexp_f32 adds E-133 to the exponent field, handling zero, BF16
//      subnormals (FP32 denormals are preserved in these kernels) and the
//      overflow of E = 255, m >= 64 to infinity;
//   4. v_perm_b32 keeps the upper halves of two floats (the value has at most
//      7 significant bits, so truncation to BF16 is exact);
//   5. a second v_perm_b32 moves the two sign bits to bits 15 and 31 and an
//      AND-OR inserts them.
// About 3.75 VALU operations per element.
//
// A faster route covers 7 <= E <= 133, where every nonzero element is a
// normal BF16: the BF16 bits of the magnitude itself (exact, at most 7
// significant bits) only need their exponent field lowered by 133 - E, which
// one saturating 16-bit packed subtract does for two elements at once while
// keeping zero at zero.  That replaces the two v_ldexp_f32 of a pair (about
// 3.25 operations per element).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hma {

constexpr int kHeadDim = 128;
constexpr int kPageSize = 16;
constexpr int kBlock = 16;            // channels per shared exponent
constexpr int kExpBias = 133;         // 127 + 6
constexpr int kExpPerRow = kHeadDim / kBlock;        // 8 exponent bytes per token row
constexpr int kTileMant = kPageSize * kHeadDim;      // 2048 mantissa bytes per (page, head)
constexpr int kTileExp = kPageSize * kExpPerRow;     // 128 exponent bytes per (page, head)
constexpr uint32_t kTagBf16 = 0x40000000u;
constexpr uint32_t kIdMask = 0x3FFFFFFFu;

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
typedef uint16_t u16x2_t __attribute__((ext_vector_type(2)));

// Packed 16-bit integer helpers (v_pk_*_u16; integer ops, no packed FP32).
__device__ __forceinline__ uint32_t pk_sub_u16(uint32_t a, uint32_t b)
{
    return __builtin_bit_cast(uint32_t, __builtin_bit_cast(u16x2_t, a) - __builtin_bit_cast(u16x2_t, b));
}
__device__ __forceinline__ uint32_t pk_sub_sat_u16(uint32_t a, uint32_t b)
{
    return __builtin_bit_cast(uint32_t, __builtin_elementwise_sub_sat(__builtin_bit_cast(u16x2_t, a),
                                                                      __builtin_bit_cast(u16x2_t, b)));
}
__device__ __forceinline__ uint32_t pk_add_sat_u16(uint32_t a, uint32_t b)
{
    return __builtin_bit_cast(uint32_t, __builtin_elementwise_add_sat(__builtin_bit_cast(u16x2_t, a),
                                                                      __builtin_bit_cast(u16x2_t, b)));
}
__device__ __forceinline__ uint32_t pk_max_u16(uint32_t a, uint32_t b)
{
    return __builtin_bit_cast(uint32_t, __builtin_elementwise_max(__builtin_bit_cast(u16x2_t, a),
                                                                  __builtin_bit_cast(u16x2_t, b)));
}
__device__ __forceinline__ uint32_t pk_shl7_u16(uint32_t a)
{
    return __builtin_bit_cast(uint32_t, __builtin_bit_cast(u16x2_t, a) << (uint16_t)7);
}

// byte-select constants for __builtin_amdgcn_perm(S0, S1, sel):
// result byte i = byte sel_i of the 64-bit value {S0 (bytes 4..7), S1 (bytes 0..3)};
// selector 0x0C yields 0x00.
constexpr uint32_t kPermHiHalves = 0x07060302u;    // {S0.hi16, S1.hi16}
constexpr uint32_t kPermLoHalves = 0x05040100u;    // {S0.lo16, S1.lo16}

// Sign bits of bytes a (from S1) and b (from S0) placed in bytes 1 and 3.
__device__ __forceinline__ constexpr uint32_t sign_sel(int a, int b)
{
    return ((uint32_t)(4 + b) << 24) | (0x0Cu << 16) | ((uint32_t)a << 8) | 0x0Cu;
}

// Clear the four sign bits of a mantissa word.  Written as one opaque
// v_and_b32 so the compiler does not fold the known-zero bits into each byte
// extraction (which would turn v_cvt_f32_ubyteN into a v_bfe_u32 + ubyte0).
__device__ __forceinline__ uint32_t magnitudes(uint32_t w)
{
    uint32_t r;
    asm("v_and_b32 %0, 0x7f7f7f7f, %1" : "=v"(r) : "v"(w));
    return r;
}

__device__ __forceinline__ float mag_byte(uint32_t mag_word, int k)
{
    // (float) of one byte: compiles to v_cvt_f32_ubyte{k}
    return (float)((mag_word >> (8 * k)) & 0xFFu);
}

// Exact float of the magnitude of byte k of `mag_word`, scaled by 2^es.
__device__ __forceinline__ float bfp8_mag_f32(uint32_t mag_word, int k, int es)
{
    return __builtin_amdgcn_ldexpf(mag_byte(mag_word, k), es);
}

// Pack two exact floats (lo, hi) into a BF16 pair and OR in two sign bits
// taken from byte ka of word wa (-> bit 15) and byte kb of word wb (-> bit 31).
__device__ __forceinline__ uint32_t pack_bf16_signed(float lo, float hi, uint32_t wa, int ka,
                                                     uint32_t wb, int kb)
{
    uint32_t m = __builtin_amdgcn_perm(__float_as_uint(hi), __float_as_uint(lo), kPermHiHalves);
    uint32_t s = __builtin_amdgcn_perm(wb, wa, sign_sel(ka, kb));
    return (s & 0x80008000u) | m;
}

// Decode one word of four BFP8 elements (same block exponent) into two BF16
// pairs in natural order: .x = {e1:e0}, .y = {e3:e2}.
__device__ __forceinline__ u32x2_t bfp8_word_to_bf16(uint32_t w, int es)
{
    const uint32_t mg = magnitudes(w);
    const float f0 = bfp8_mag_f32(mg, 0, es);
    const float f1 = bfp8_mag_f32(mg, 1, es);
    const float f2 = bfp8_mag_f32(mg, 2, es);
    const float f3 = bfp8_mag_f32(mg, 3, es);
    return u32x2_t{pack_bf16_signed(f0, f1, w, 0, w, 1), pack_bf16_signed(f2, f3, w, 2, w, 3)};
}

// Decode four words (16 elements of one block) into eight BF16 pairs.
__device__ __forceinline__ void bfp8_block_to_bf16(u32x4_t w, int es, u32x4_t &lo, u32x4_t &hi)
{
    const u32x2_t a = bfp8_word_to_bf16(w.x, es);
    const u32x2_t b = bfp8_word_to_bf16(w.y, es);
    const u32x2_t c = bfp8_word_to_bf16(w.z, es);
    const u32x2_t d = bfp8_word_to_bf16(w.w, es);
    lo = u32x4_t{a.x, a.y, b.x, b.y};
    hi = u32x4_t{c.x, c.y, d.x, d.y};
}

// ---- fast route (7 <= E <= 133): `d` holds (133 - E) << 7 in each 16-bit
// half, for the element that lands in that half.

// Two exact magnitudes (lo, hi) -> BF16 pair scaled by 2^(E-133), with the
// sign bits of byte ka of wa (-> bit 15) and byte kb of wb (-> bit 31).
__device__ __forceinline__ uint32_t pack_bf16_scaled_signed(float lo, float hi, uint32_t d, uint32_t wa,
                                                            int ka, uint32_t wb, int kb)
{
    uint32_t m = __builtin_amdgcn_perm(__float_as_uint(hi), __float_as_uint(lo), kPermHiHalves);
    m = pk_sub_sat_u16(m, d);
    uint32_t s = __builtin_amdgcn_perm(wb, wa, sign_sel(ka, kb));
    return (s & 0x80008000u) | m;
}

__device__ __forceinline__ u32x2_t bfp8_word_to_bf16_fast(uint32_t w, uint32_t d)
{
    const uint32_t mg = magnitudes(w);
    const float f0 = mag_byte(mg, 0);
    const float f1 = mag_byte(mg, 1);
    const float f2 = mag_byte(mg, 2);
    const float f3 = mag_byte(mg, 3);
    return u32x2_t{pack_bf16_scaled_signed(f0, f1, d, w, 0, w, 1),
                   pack_bf16_scaled_signed(f2, f3, d, w, 2, w, 3)};
}

__device__ __forceinline__ void bfp8_block_to_bf16_fast(u32x4_t w, uint32_t d, u32x4_t &lo, u32x4_t &hi)
{
    const u32x2_t a = bfp8_word_to_bf16_fast(w.x, d);
    const u32x2_t b = bfp8_word_to_bf16_fast(w.y, d);
    const u32x2_t c = bfp8_word_to_bf16_fast(w.z, d);
    const u32x2_t e = bfp8_word_to_bf16_fast(w.w, d);
    lo = u32x4_t{a.x, a.y, b.x, b.y};
    hi = u32x4_t{c.x, c.y, e.x, e.y};
}

}  // namespace hma
