// Device helpers shared by the MFMA kernels (prefill GEMM, many-token decode):
// in-register dequantization of 4-bit codes to fp16 and the fp16 MFMA.
#pragma once

#include "cl_device.h"

namespace cl {

// (x & m) | c in one instruction; m comes from a scalar register, c from a
// vector register (one scalar operand per instruction on this target).
__device__ __forceinline__ uint32_t and_or(uint32_t x, uint32_t m, uint32_t c) {
    uint32_t r;
    asm("v_and_or_b32 %0, %1, %2, %3" : "=v"(r) : "v"(x), "s"(m), "v"(c));
    return r;
}

// Per-fragment constants of one quantization group for dequant_word4x, two
// halves per register: (s, s/16) and (1024 + z, 1024 + 16 z).
struct Dq {
    f16x2 s, z;
};

__device__ __forceinline__ Dq make_dq(uint32_t sbits, uint32_t zbits) {
    const f16 s = __builtin_bit_cast(f16, static_cast<uint16_t>(sbits));
    const f16 z = __builtin_bit_cast(f16, static_cast<uint16_t>(zbits));
    const f16 s16 = s * static_cast<f16>(0.0625f);                     // exact unless subnormal
    const f16 z1 = static_cast<f16>(1024.0f) + z;                      // exact: z < 16
    const f16 z16 = static_cast<f16>(1024.0f) + z * static_cast<f16>(16.0f);
    return Dq{f16x2{s, s16}, f16x2{z1, z16}};
}

// One 32-bit word of 4-bit codes -> 8 fp16 values s (q - z), pair order
// (q0,q4),(q1,q5),(q2,q6),(q3,q7), with one shift and four masks: a code
// left in bits 4..7 of a half reads as 1024 + 16 q, so its pair subtracts
// 1024 + 16 z (exact) and scales by s/16.
__device__ __forceinline__ u32x4 dequant_word4x(uint32_t w, const Dq& d, uint32_t mlo, uint32_t mhi,
                                               uint32_t bias) {
    const uint32_t w8 = w >> 8;
    const f16x2 s1 = {d.s.x, d.s.x}, s16 = {d.s.y, d.s.y};
    const f16x2 z1 = {d.z.x, d.z.x}, z16 = {d.z.y, d.z.y};
    u32x4 r;
    r[0] = __builtin_bit_cast(uint32_t, (__builtin_bit_cast(f16x2, and_or(w, mlo, bias)) - z1) * s1);
    r[1] = __builtin_bit_cast(uint32_t, (__builtin_bit_cast(f16x2, and_or(w, mhi, bias)) - z16) * s16);
    r[2] = __builtin_bit_cast(uint32_t, (__builtin_bit_cast(f16x2, and_or(w8, mlo, bias)) - z1) * s1);
    r[3] = __builtin_bit_cast(uint32_t, (__builtin_bit_cast(f16x2, and_or(w8, mhi, bias)) - z16) * s16);
    return r;
}

__device__ __forceinline__ f32x4 mfma(const u32x4& a, const u32x4& b, const f32x4& c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c,
                                                  0, 0, 0);
}

}  // namespace cl
