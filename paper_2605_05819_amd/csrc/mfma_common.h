// Device helpers shared by the MFMA kernels (prefill GEMM, many-token decode,
// MoE): in-register unpack of 4-, 3- and 2-bit codes to exact fp16 integers q - z, the
// 4 x 4 transpose of code words across lane groups, and the fp16 MFMA.
#pragma once

#include "cl_device.h"

namespace cl {

// Row stride, in entries, of the MFMA backbones' scale and zero tables in
// LDS (decode and MoE): for a multiple of 8 groups, the groups rounded up to
// 16, plus 8 -- half of it is 4 mod 8 4-byte banks, so the 16 rows one read
// instruction touches fall in 16 distinct banks (a stride of 32 groups had
// put four rows in each bank) and 16-byte pieces of a row stay aligned;
// otherwise the groups themselves (the table stays one contiguous run, which
// 16-byte pieces fill across row boundaries).
__host__ __device__ constexpr int szl_stride(int groups) {
    return groups % 8 ? groups : (groups + 15) / 16 * 16 + 8;
}

// (x & m) | c in one instruction; m comes from a scalar register, c from a
// vector register (one scalar operand per instruction on this target).
__device__ __forceinline__ uint32_t and_or(uint32_t x, uint32_t m, uint32_t c) {
    uint32_t r;
    asm("v_and_or_b32 %0, %1, %2, %3" : "=v"(r) : "v"(x), "s"(m), "v"(c));
    return r;
}

// Zero-point constants of one quantization group for codes_minus_zero, both
// halves of each register equal: -(1024 + z) and -(64 + z) (exact: z < 16).
struct Zq {
    f16x2 lo, hi;
};

__device__ __forceinline__ Zq make_zq(uint32_t zbits) {
    const f16 z = __builtin_bit_cast(f16, static_cast<uint16_t>(zbits));
    const f16 a = -(static_cast<f16>(1024.0f) + z);
    const f16 b = -(static_cast<f16>(64.0f) + z);
    return Zq{f16x2{a, a}, f16x2{b, b}};
}

// One 32-bit word of 4-bit codes -> 8 fp16 values q - z, exact integers in
// -15..15, pair order (q0,q4),(q1,q5),(q2,q6),(q3,q7).  A code OR-ed into the
// mantissa of 1024.0 (bits 0x6400) reads as 1024 + q, so adding -(1024 + z)
// is exact; a code left in bits 4..7 of the half reads as 1024 + 16 q, and one
// fused multiply-add (1024 + 16 q) / 16 - (64 + z) is exact as well.  One
// shift, four v_and_or_b32, two packed adds and two packed FMAs per word.
__device__ __forceinline__ u32x4 codes_minus_zero(uint32_t w, const Zq& zq, uint32_t mlo, uint32_t mhi,
                                                  uint32_t bias) {
    const uint32_t w8 = w >> 8;
    const f16x2 sixteenth = {static_cast<f16>(0.0625f), static_cast<f16>(0.0625f)};
    u32x4 r;
    r[0] = __builtin_bit_cast(uint32_t, __builtin_bit_cast(f16x2, and_or(w, mlo, bias)) + zq.lo);
    r[1] = __builtin_bit_cast(
        uint32_t, __builtin_elementwise_fma(__builtin_bit_cast(f16x2, and_or(w, mhi, bias)), sixteenth, zq.hi));
    r[2] = __builtin_bit_cast(uint32_t, __builtin_bit_cast(f16x2, and_or(w8, mlo, bias)) + zq.lo);
    r[3] = __builtin_bit_cast(
        uint32_t, __builtin_elementwise_fma(__builtin_bit_cast(f16x2, and_or(w8, mhi, bias)), sixteenth, zq.hi));
    return r;
}

// 2-bit codes.  One 8-code half of a word (h = 0: codes 0..7, h = 1: codes
// 8..15) laid out for a mask per pair: bytes (b_2h, b_2h+1 | b_2h+1, 0), so
// bits 2p..2p+1 of the low fp16 half hold code p and those of the high half
// code p + 4 (one byte permute).
__device__ __forceinline__ uint32_t spread_half2(uint32_t w, int h) {
    return __builtin_amdgcn_perm(0u, w, h ? 0x0C030302u : 0x0C010100u);
}

// Zero-point constants of one 2-bit group: -(1024 / 4^p + z), p = 0..3, both
// halves equal (exact: z < 4).
struct Zq2 {
    f16x2 c[4];
};

__device__ __forceinline__ Zq2 make_zq2(uint32_t zbits) {
    const f16 z = __builtin_bit_cast(f16, static_cast<uint16_t>(zbits));
    Zq2 r;
#pragma unroll
    for (int p = 0; p < 4; ++p) {
        const f16 v = -(static_cast<f16>(1024.0f / static_cast<float>(1 << (2 * p))) + z);
        r.c[p] = f16x2{v, v};
    }
    return r;
}

// A spread 8-code half (spread_half2) -> 8 fp16 values q - z, exact integers
// in -3..3, pair order (q0,q4),(q1,q5),(q2,q6),(q3,q7) as codes_minus_zero.
// Pair p masked in place and OR-ed into the mantissa of 1024.0 reads as
// 1024 + 4^p q; one fused multiply-add (1024 + 4^p q) 4^-p - (1024 4^-p + z)
// is exact (p = 0: one add).  m[p] = 0x00030003 << 2p from scalar registers.
__device__ __forceinline__ u32x4 codes2_minus_zero(uint32_t v, const Zq2& zq, const uint32_t (&m)[4],
                                                   uint32_t bias) {
    u32x4 r;
    r[0] = __builtin_bit_cast(uint32_t, __builtin_bit_cast(f16x2, and_or(v, m[0], bias)) + zq.c[0]);
#pragma unroll
    for (int p = 1; p < 4; ++p) {
        const f16 sc = static_cast<f16>(1.0f / static_cast<float>(1 << (2 * p)));
        r[p] = __builtin_bit_cast(uint32_t, __builtin_elementwise_fma(__builtin_bit_cast(f16x2, and_or(v, m[p], bias)),
                                                                      f16x2{sc, sc}, zq.c[p]));
    }
    return r;
}

// 3-bit codes.  A lane's 32 codes are three words; 8-code unit t (codes
// 8t .. 8t + 7) is bytes 3t .. 3t + 2, code i at bits 3i of those 24.
// Spread for a mask per pair: a byte permute gives x = (b0 b1 | b1 b2) (bits
// 0..15 and 8..23 of the unit), then the low half keeps x's low half and the
// high half takes x >> 4, so codes 0..3 sit at bits 0, 3, 6, 9 of the low
// fp16 half and codes 4..7 at the same offsets of the high half.
__device__ __forceinline__ uint32_t spread_unit3(uint32_t w0, uint32_t w1, uint32_t w2, int t) {
    const uint32_t x = t == 0   ? __builtin_amdgcn_perm(w1, w0, 0x02010100u)
                       : t == 1 ? __builtin_amdgcn_perm(w1, w0, 0x05040403u)
                       : t == 2 ? __builtin_amdgcn_perm(w2, w1, 0x04030302u)
                                : __builtin_amdgcn_perm(0u, w2, 0x03020201u);
    return (x & 0x0000FFFFu) | ((x >> 4) & 0xFFFF0000u);
}

// Zero-point constants of one 3-bit group: -(1024 + z), -(128 + z), -(16 + z)
// in both halves (exact: z < 8).
struct Zq3 {
    f16x2 c[3];
};

__device__ __forceinline__ Zq3 make_zq3(uint32_t zbits) {
    const f16 z = __builtin_bit_cast(f16, static_cast<uint16_t>(zbits));
    const f16 a = -(static_cast<f16>(1024.0f) + z), b = -(static_cast<f16>(128.0f) + z),
              c = -(static_cast<f16>(16.0f) + z);
    return Zq3{{f16x2{a, a}, f16x2{b, b}, f16x2{c, c}}};
}

// A spread 3-bit unit (spread_unit3) -> 8 fp16 values q - z, exact integers
// in -7..7, pair order (q0,q4),(q1,q5),(q2,q6),(q3,q7) as codes_minus_zero.
// Pairs 0, 1, 2 are masked in place at bits 0, 3, 6 and OR-ed into 1024.0
// (1024 + q, 1024 + 8 q, 1024 + 64 q); pair 3 (bits 9..11, past the fp16
// mantissa) is shifted down to bits 6..8 first.  One add or fused
// multiply-add by 8^-p per pair is exact.  m[p] = 0x00070007 << 3p (p < 3)
// from scalar registers.
__device__ __forceinline__ u32x4 codes3_minus_zero(uint32_t v, const Zq3& zq, const uint32_t (&m)[3],
                                                   uint32_t bias) {
    const f16x2 e8 = {static_cast<f16>(0.125f), static_cast<f16>(0.125f)};
    const f16x2 e64 = {static_cast<f16>(0.015625f), static_cast<f16>(0.015625f)};
    u32x4 r;
    r[0] = __builtin_bit_cast(uint32_t, __builtin_bit_cast(f16x2, and_or(v, m[0], bias)) + zq.c[0]);
    r[1] = __builtin_bit_cast(uint32_t,
                              __builtin_elementwise_fma(__builtin_bit_cast(f16x2, and_or(v, m[1], bias)), e8, zq.c[1]));
    r[2] = __builtin_bit_cast(uint32_t,
                              __builtin_elementwise_fma(__builtin_bit_cast(f16x2, and_or(v, m[2], bias)), e64, zq.c[2]));
    r[3] = __builtin_bit_cast(
        uint32_t, __builtin_elementwise_fma(__builtin_bit_cast(f16x2, and_or(v >> 3, m[2], bias)), e64, zq.c[2]));
    return r;
}

// s (q - z) as fp16, one rounding per value (the dequantized tile of the
// prefill GEMM); the integer q - z is formed exactly first, so the rounding
// is relative 2^-11 down to the fp16 normal range whatever the scale.
__device__ __forceinline__ u32x4 dequant_word4x(uint32_t w, const Zq& zq, f16x2 s2, uint32_t mlo, uint32_t mhi,
                                               uint32_t bias) {
    u32x4 r = codes_minus_zero(w, zq, mlo, mhi, bias);
#pragma unroll
    for (int p = 0; p < 4; ++p) {
        const uint32_t v = r[p];
        r[p] = __builtin_bit_cast(uint32_t, __builtin_bit_cast(f16x2, v) * s2);
    }
    return r;
}

// One half of dequant_word4x: h = 0 gives r[0], r[1] (codes of the low
// byte of each half-word), h = 1 gives r[2], r[3]; the same values.
__device__ __forceinline__ void dequant_half4x(uint32_t w, int h, const Zq& zq, f16x2 s2, uint32_t mlo, uint32_t mhi,
                                               uint32_t bias, uint32_t& lo, uint32_t& hi) {
    const uint32_t v = h ? w >> 8 : w;
    const f16x2 sixteenth = {static_cast<f16>(0.0625f), static_cast<f16>(0.0625f)};
    const f16x2 a = __builtin_bit_cast(f16x2, and_or(v, mlo, bias)) + zq.lo;
    const f16x2 b = __builtin_elementwise_fma(__builtin_bit_cast(f16x2, and_or(v, mhi, bias)), sixteenth, zq.hi);
    lo = __builtin_bit_cast(uint32_t, a * s2);
    hi = __builtin_bit_cast(uint32_t, b * s2);
}

// 4 x 4 transpose across the four 16-lane groups of a wave: on entry lane
// group g holds words 4 g .. 4 g + 3 of a 16-word run in w[0..3]; on return
// w[t] holds word 4 t + g.  v_permlane32_swap exchanges rows 2-3 of its first
// operand with rows 0-1 of its second, v_permlane16_swap the odd rows of the
// first with the even rows of the second (a row is 16 lanes).
__device__ __forceinline__ void transpose_words(uint32_t (&w)[4]) {
    const auto a = __builtin_amdgcn_permlane32_swap(w[0], w[2], false, false);
    const auto b = __builtin_amdgcn_permlane32_swap(w[1], w[3], false, false);
    const auto c = __builtin_amdgcn_permlane16_swap(a[0], b[0], false, false);
    const auto d = __builtin_amdgcn_permlane16_swap(a[1], b[1], false, false);
    w[0] = c[0];
    w[1] = c[1];
    w[2] = d[0];
    w[3] = d[1];
}

__device__ __forceinline__ f32x4 mfma(const u32x4& a, const u32x4& b, const f32x4& c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c,
                                                  0, 0, 0);
}

// Two fp32 values as fp16 pairs hi = fp16(v) and lo = fp16(v - hi): an
// MFMA step over hi and one over lo carry v to about 2^-22 relative (the
// difference v - hi is exact in fp32), where hi alone would round it to
// 2^-11.
__device__ __forceinline__ void split_f16x2(float a, float b, uint32_t& hi, uint32_t& lo) {
    const f16 ha = static_cast<f16>(a), hb = static_cast<f16>(b);
    const f16 la = static_cast<f16>(a - static_cast<float>(ha)), lb = static_cast<f16>(b - static_cast<float>(hb));
    hi = __builtin_bit_cast(uint32_t, f16x2{ha, hb});
    lo = __builtin_bit_cast(uint32_t, f16x2{la, lb});
}

// acc += s * p, elementwise in fp32
__device__ __forceinline__ f32x4 fma4(float s, const f32x4& p, const f32x4& acc) {
    f32x4 r;
#pragma unroll
    for (int e = 0; e < 4; ++e) r[e] = fmaf(s, p[e], acc[e]);
    return r;
}

}  // namespace cl
