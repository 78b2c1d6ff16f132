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

// 3-bit codes come in chunks of 32 codes = 3 words (the row's bit string cut
// into words: codes 8k .. 8k + 7 fill bytes 3k .. 3k + 2 of the chunk's 12).
// The activations of a chunk are prepared as 16 fp16 pairs: pair i < 8 is
// (x[i], x[i + 8]), pair 8 + i is (x[16 + i], x[24 + i]); see dot_chunk3.
__device__ __forceinline__ void load_chunk_x3(const uint16_t* xr, int chunk, int act, f16x2* xv) {
    uint32_t u[16];                                // u[i] holds (x[2i], x[2i+1]) of the chunk
#pragma unroll
    for (int j = 0; j < 4; ++j) load8_f16(xr + chunk * 32 + 8 * j, act, u + 4 * j);
#pragma unroll
    for (int h = 0; h < 2; ++h)                    // codes 0..15, then 16..31
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const uint32_t lo = u[8 * h + i / 2], hi = u[8 * h + 4 + i / 2];
            const uint32_t a = (i & 1) ? (lo >> 16) : (lo & 0xffff);
            const uint32_t b = (i & 1) ? (hi & 0xffff0000u) : (hi << 16);
            xv[8 * h + i] = __builtin_bit_cast(f16x2, a | b);
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

// One chunk of 3-bit codes (words w0, w1, w2) against its 16 prepared
// activation pairs, into 8 accumulators.  A byte permute puts two 8-code
// groups side by side, one in each fp16 half: bytes (b0 b1 | b3 b4) hold bits
// 0..15 of codes 0..7 and of codes 8..15, so code i and code i + 8 sit at the
// same bit offset in both halves and one AND leaves the pair as exact fp16
// subnormals (code << k) * 2^-24 with the code in mantissa bits k .. k + 2,
// k <= 7.  Codes 0, 1, 2 come from (b0 b1 | b3 b4) at offsets 0, 3, 6; codes
// 3, 4, 5 from (b1 b2 | b4 b5) at 1, 4, 7; codes 6, 7 from (b2 | b5) at 2, 5;
// bytes b6 .. b11 give codes 16 .. 31 the same way.  Accumulator i collects
// code i's pairs (scale 2^k(i)); combine<3> divides the scales out.  Six
// permutes, 16 ANDs and 16 v_dot2 per 32 codes.
__device__ __forceinline__ uint32_t byte_perm(uint32_t hi, uint32_t lo, uint32_t sel) {
    // byte j of the result is byte s_j of the 8 bytes (hi:lo), s_j = byte j of
    // the selector: 0..3 pick bytes of lo, 4..7 bytes of hi, 12 gives 0
    return __builtin_amdgcn_perm(hi, lo, sel);
}

__device__ __forceinline__ void dot_chunk3(uint32_t w0, uint32_t w1, uint32_t w2, const f16x2* xv, float* d) {
    constexpr uint32_t m[8] = {0x00070007u, 0x00380038u, 0x01C001C0u, 0x000E000Eu,
                               0x00700070u, 0x03800380u, 0x001C001Cu, 0x00E000E0u};
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const uint32_t lo = h ? w1 : w0, hi = h ? w2 : w1;
        // h = 0: bytes b0..b5 (w0 bytes 0-3, w1 bytes 0-1); h = 1: b6..b11
        // (w1 bytes 2-3, w2 bytes 0-3)
        const uint32_t p1 = byte_perm(hi, lo, h ? 0x06050302u : 0x04030100u);
        const uint32_t p2 = byte_perm(hi, lo, h ? 0x07060403u : 0x05040201u);
        const uint32_t p3 = byte_perm(hi, lo, h ? 0x0C070C04u : 0x0C050C02u);
        const f16x2* x = xv + 8 * h;
        d[0] = dot2(__builtin_bit_cast(f16x2, p1 & m[0]), x[0], d[0]);
        d[1] = dot2(__builtin_bit_cast(f16x2, p1 & m[1]), x[1], d[1]);
        d[2] = dot2(__builtin_bit_cast(f16x2, p1 & m[2]), x[2], d[2]);
        d[3] = dot2(__builtin_bit_cast(f16x2, p2 & m[3]), x[3], d[3]);
        d[4] = dot2(__builtin_bit_cast(f16x2, p2 & m[4]), x[4], d[4]);
        d[5] = dot2(__builtin_bit_cast(f16x2, p2 & m[5]), x[5], d[5]);
        d[6] = dot2(__builtin_bit_cast(f16x2, p3 & m[6]), x[6], d[6]);
        d[7] = dot2(__builtin_bit_cast(f16x2, p3 & m[7]), x[7], d[7]);
    }
}

// sum of q * x * 2^-24 over the word(s): the per-scale accumulators with
// their power-of-two scales removed
template <int BITS>
__device__ __forceinline__ float combine(const float* d) {
    if (BITS == 4) return fmaf(d[1], 0.0625f, d[0]);
    if (BITS == 3)   // code i's accumulator carries 2^k(i), k = 0 3 6 1 4 7 2 5
        return fmaf(d[5], 0.0078125f, fmaf(d[2], 0.015625f, fmaf(d[7], 0.03125f, fmaf(d[4], 0.0625f,
                    fmaf(d[1], 0.125f, fmaf(d[6], 0.25f, fmaf(d[3], 0.5f, d[0])))))));
    return fmaf(d[3], 0.015625f, fmaf(d[2], 0.0625f, fmaf(d[1], 0.25f, d[0])));
}

}  // namespace cl
