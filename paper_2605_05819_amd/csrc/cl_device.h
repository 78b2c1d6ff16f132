// Device-side helpers shared by the gfx950 kernels of the compensated linear.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cl {

typedef _Float16 f16;
typedef f16 f16x2 __attribute__((ext_vector_type(2)));
typedef f16 f16x8 __attribute__((ext_vector_type(8)));
typedef short bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

enum { DT_FP16 = 1, DT_BF16 = 2, DT_FP32 = 3 };

__device__ __forceinline__ float f16_bits_to_f32(uint16_t b) {
    return static_cast<float>(__builtin_bit_cast(f16, b));
}

__device__ __forceinline__ float bf16_bits_to_f32(uint16_t b) {
    return __builtin_bit_cast(float, static_cast<uint32_t>(b) << 16);
}

// float -> bf16, round to nearest, ties to even (NaN kept quiet).
__device__ __forceinline__ uint16_t f32_to_bf16_bits(float f) {
    uint32_t u = __builtin_bit_cast(uint32_t, f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return static_cast<uint16_t>((u >> 16) | 0x40);
    u += 0x7fffu + ((u >> 16) & 1u);
    return static_cast<uint16_t>(u >> 16);
}

__device__ __forceinline__ uint16_t f32_to_f16_bits(float f) {
    return __builtin_bit_cast(uint16_t, static_cast<f16>(f));
}

// fp64 -> fp16 bits, round to nearest, ties to even, in a single rounding
// (IEEE 754 binary16: 1 sign, 5 exponent, 10 fraction bits, bias 15).
__device__ __forceinline__ uint16_t f64_to_f16_rne(double v) {
    uint64_t b = __builtin_bit_cast(uint64_t, v);
    uint16_t sign = static_cast<uint16_t>((b >> 48) & 0x8000u);
    double a = fabs(v);
    if (a != a) return 0x7e00u;
    if (a >= 65520.0) return sign | 0x7c00u;          // rounds past the largest finite value
    int e = static_cast<int>((b >> 52) & 0x7ff) - 1023;  // a is finite, possibly subnormal in fp64
    if (a == 0.0) return sign;
    if (e < -14) {
        // subnormal fp16 range: the value in units of 2^-24 (exact scaling)
        double m = rint(a * 16777216.0);
        return sign | static_cast<uint16_t>(m);      // m == 1024 encodes the smallest normal
    }
    double m = rint(ldexp(a, 10 - e));                // in [1024, 2048]
    if (m == 2048.0) { m = 1024.0; e += 1; }
    if (e > 15) return sign | 0x7c00u;
    return sign | static_cast<uint16_t>(((e + 15) << 10) | (static_cast<int>(m) - 1024));
}

// An activation element as fp16.  bf16 inputs are converted (exact inside the
// fp16 range down to 2^-17, saturated at +-65504 above it).
__device__ __forceinline__ f16 act_to_f16(uint16_t b, int act) {
    if (act == DT_FP16) return __builtin_bit_cast(f16, b);
    float v = bf16_bits_to_f32(b);
    v = fminf(fmaxf(v, -65504.0f), 65504.0f);
    return static_cast<f16>(v);
}

// 8 activations (one 16-byte load) as fp16, natural order; bf16 converted.
__device__ __forceinline__ u32x4 act8_to_f16(u32x4 u, int act) {
    if (act == DT_FP16) return u;
    u32x4 o;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const uint32_t uk = u[k];
        f16x2 h;
        h.x = act_to_f16(static_cast<uint16_t>(uk & 0xffff), act);
        h.y = act_to_f16(static_cast<uint16_t>(uk >> 16), act);
        o[k] = __builtin_bit_cast(uint32_t, h);
    }
    return o;
}

__device__ __forceinline__ float act_to_f32(uint16_t b, int act) {
    return act == DT_FP16 ? f16_bits_to_f32(b) : bf16_bits_to_f32(b);
}

// SiLU(g) u = g / (1 + e^-g) * u in fp32 with a reciprocal-based quotient
// (a few ulp; the IEEE division sequence cost the one-token backbone a
// spilled register); for g far below zero e^-g is inf, its reciprocal 0 and
// the result a signed zero
__device__ __forceinline__ float silu_mul(float g, float u) { return __fdividef(g, 1.f + __expf(-g)) * u; }

// 8 gated activations h = SiLU(g) u from one 16-byte load of each input
// (fp16 or bf16, natural order) as fp16: each product in fp32, saturated at
// +-65504 like a converted bf16 activation, then rounded to nearest even.
__device__ __forceinline__ u32x4 gated8_to_f16(u32x4 g, u32x4 u, int act) {
    u32x4 o;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const uint32_t gk = g[k], uk = u[k];
        float h0 = silu_mul(act_to_f32(static_cast<uint16_t>(gk & 0xffff), act),
                            act_to_f32(static_cast<uint16_t>(uk & 0xffff), act));
        float h1 = silu_mul(act_to_f32(static_cast<uint16_t>(gk >> 16), act),
                            act_to_f32(static_cast<uint16_t>(uk >> 16), act));
        h0 = fminf(fmaxf(h0, -65504.0f), 65504.0f);
        h1 = fminf(fmaxf(h1, -65504.0f), 65504.0f);
        f16x2 h;
        h.x = static_cast<f16>(h0);
        h.y = static_cast<f16>(h1);
        o[k] = __builtin_bit_cast(uint32_t, h);
    }
    return o;
}

__device__ __forceinline__ void store_out(void* y, size_t idx, float v, int out) {
    if (out == DT_FP32) {
        static_cast<float*>(y)[idx] = v;
    } else if (out == DT_FP16) {
        static_cast<uint16_t*>(y)[idx] = f32_to_f16_bits(v);
    } else {
        static_cast<uint16_t*>(y)[idx] = f32_to_bf16_bits(v);
    }
}

// v_dot2_f32_f16: a.x*b.x + a.y*b.y + c with float accumulation.
__device__ __forceinline__ float dot2(f16x2 a, f16x2 b, float c) {
    return __builtin_amdgcn_fdot2(a, b, c, false);
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
    return v;
}

// Packed-code extraction into fp16 lanes.
//
// A 4-bit code q placed in the low mantissa bits of an fp16 with a zero
// exponent field is the subnormal q * 2^-24, exactly.  Masking one 32-bit word
// with 0x000F000F after a right shift by 4p therefore yields the pair
// (q_p, q_{p+4}) * 2^-24 as two fp16 lanes in a single AND; the 2-bit layout
// works the same way with mask 0x00030003 and pairs (q_p, q_{p+8}).  Products
// with fp16 activations are exact in the float accumulator of v_dot2, and the
// 2^24 is folded into the per-group scale.
template <int BITS>
__device__ __forceinline__ f16x2 code_pair(uint32_t w, int p) {
    constexpr uint32_t mask = BITS == 4 ? 0x000F000Fu : 0x00030003u;
    return __builtin_bit_cast(f16x2, (w >> (BITS * p)) & mask);
}

}  // namespace cl
