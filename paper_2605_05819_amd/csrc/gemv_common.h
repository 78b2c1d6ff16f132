// Device helpers shared by the decode GEMV kernels (dense windows and MoE).
#pragma once

#include "cl_device.h"

namespace cl {

// Load 8 consecutive activations as four f16x2 words (fp16 or bf16 input).
__device__ __forceinline__ void load8_f16(const uint16_t* p, int act, uint32_t out[4]) {
    const u32x4 u = act8_to_f16(*reinterpret_cast<const u32x4*>(p), act);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const uint32_t uk = u[k];
        out[k] = uk;
    }
}

// Activations of one 16-byte chunk of codes, in the pair order of the
// unpacked codes: word w, pair p = (x[w*CPW + p], x[w*CPW + p + CPW/2]).
template <int BITS>
__device__ __forceinline__ void load_chunk_x(const uint16_t* xr, int chunk, int act, f16x2* xv) {
    constexpr int CPW = 32 / BITS, HPW = CPW / 2;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
        const uint16_t* p = xr + (chunk * 4 + w) * CPW;
        uint32_t u[CPW / 2];                        // CPW halves as packed pairs
#pragma unroll
        for (int j = 0; j < CPW / 8; ++j) load8_f16(p + 8 * j, act, u + 4 * j);
        // u[i] holds (x[2i], x[2i+1]); pair p needs (x[p], x[p + HPW])
#pragma unroll
        for (int pp = 0; pp < HPW; ++pp) {
            const uint32_t lo = u[pp / 2], hi = u[(pp + HPW) / 2];
            const uint32_t a = (pp & 1) ? (lo >> 16) : (lo & 0xffff);
            const uint32_t b = (pp & 1) ? (hi & 0xffff0000u) : (hi << 16);
            xv[w * HPW + pp] = __builtin_bit_cast(f16x2, a | b);
        }
    }
}

// Sum R (2, 4 or 8) values over the 64 lanes of a wave with a transposing
// butterfly.  On return lane l holds the total of value index (l / (64/R)).
template <int R>
__device__ __forceinline__ float wave_sum_multi(float (&v)[R]) {
    const int lane = threadIdx.x & 63;
    float a[R];
#pragma unroll
    for (int i = 0; i < R; ++i) a[i] = v[i];
    int n = R;
    int bit = 32;
#pragma unroll
    for (int step = 0; step < 3; ++step) {
        if (n > 1) {
            const bool up = (lane & bit) != 0;
            const int h = n / 2;
#pragma unroll
            for (int i = 0; i < R / 2; ++i) {
                if (i < h) {
                    const float mine = up ? a[i + h] : a[i];
                    const float other = up ? a[i] : a[i + h];
                    a[i] = mine + __shfl_xor(other, bit, 64);
                }
            }
            n = h;
            bit >>= 1;
        }
    }
    float r = a[0];
    for (; bit > 0; bit >>= 1) r += __shfl_xor(r, bit, 64);
    return r;
}

// Unpack one 32-bit word of codes into fp16 pairs with masks only where the
// code still lands in the 10 mantissa bits of a zero-exponent fp16 (a
// subnormal, exact).  A 4-bit pair (c_p, c_{p+4}) left in bits 4..7 of each
// half reads as 16 * c * 2^-24; a 2-bit pair (c_p, c_{p+8}) left in bits
// 2k..2k+1 reads as 4^k * c * 2^-24.  Each such scale gets its own
// accumulator; combine() divides the scales back out (exact: powers of 2).
template <int BITS>
__device__ __forceinline__ void dot_word(uint32_t w, const f16x2* xv, float* d) {
    if (BITS == 4) {
        const uint32_t w8 = w >> 8;
        d[0] = dot2(__builtin_bit_cast(f16x2, w & 0x000F000Fu), xv[0], d[0]);
        d[1] = dot2(__builtin_bit_cast(f16x2, w & 0x00F000F0u), xv[1], d[1]);
        d[0] = dot2(__builtin_bit_cast(f16x2, w8 & 0x000F000Fu), xv[2], d[0]);
        d[1] = dot2(__builtin_bit_cast(f16x2, w8 & 0x00F000F0u), xv[3], d[1]);
    } else {
        const uint32_t w8 = w >> 8;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            d[k] = dot2(__builtin_bit_cast(f16x2, w & (0x00030003u << (2 * k))), xv[k], d[k]);
            d[k] = dot2(__builtin_bit_cast(f16x2, w8 & (0x00030003u << (2 * k))), xv[4 + k], d[k]);
        }
    }
}

// dot_word split in two: the unpacked fp16 lanes of a word (4-bit: 4 pairs,
// 2-bit: 8 pairs), kept in registers when one word meets several activation
// vectors, and the v_dot2 accumulation into the same per-scale accumulators.
// (x & m) as an instruction the compiler keeps where it is written: the
// unpacked lanes then stay in registers across the activation vectors
// instead of being recomputed for each one.
__device__ __forceinline__ uint32_t and_kept(uint32_t x, uint32_t m) {
    uint32_t r;
    asm("v_and_b32 %0, %1, %2" : "=v"(r) : "v"(x), "s"(m));
    return r;
}

template <int BITS>
__device__ __forceinline__ void unpack_word(uint32_t w, f16x2* u) {
    const uint32_t w8 = w >> 8;
    if (BITS == 4) {
        u[0] = __builtin_bit_cast(f16x2, and_kept(w, 0x000F000Fu));
        u[1] = __builtin_bit_cast(f16x2, and_kept(w, 0x00F000F0u));
        u[2] = __builtin_bit_cast(f16x2, and_kept(w8, 0x000F000Fu));
        u[3] = __builtin_bit_cast(f16x2, and_kept(w8, 0x00F000F0u));
    } else {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            u[k] = __builtin_bit_cast(f16x2, and_kept(w, 0x00030003u << (2 * k)));
            u[4 + k] = __builtin_bit_cast(f16x2, and_kept(w8, 0x00030003u << (2 * k)));
        }
    }
}

template <int BITS>
__device__ __forceinline__ void dot_unpacked(const f16x2* u, const f16x2* xv, float* d) {
    if (BITS == 4) {
        d[0] = dot2(u[0], xv[0], d[0]);
        d[1] = dot2(u[1], xv[1], d[1]);
        d[0] = dot2(u[2], xv[2], d[0]);
        d[1] = dot2(u[3], xv[3], d[1]);
    } else {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            d[k] = dot2(u[k], xv[k], d[k]);
            d[k] = dot2(u[4 + k], xv[4 + k], d[k]);
        }
    }
}

// sum of q * x * 2^-24 over the word(s): the per-scale accumulators with
// their power-of-two scales removed
template <int BITS>
__device__ __forceinline__ float combine(const float* d) {
    if (BITS == 4) return fmaf(d[1], 0.0625f, d[0]);
    return fmaf(d[3], 0.015625f, fmaf(d[2], 0.0625f, fmaf(d[1], 0.25f, d[0])));
}

}  // namespace cl
