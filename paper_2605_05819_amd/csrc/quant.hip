// Group-wise asymmetric round-to-nearest quantization + LSB-first packing (2,
// 3 or 4 bits; the row is one bit string cut into 32-bit words), and the
// matching dequantization, for gfx950.
//
// The backbone quantizer of the paper is GPTQ (Section 5.1); without
// calibration data its error feedback vanishes and it is round-to-nearest on a
// per-group min/max grid that contains 0.  Every step runs in fp64 with IEEE
// division and round-half-to-even, and the fp16 scale is rounded once,
// directly from fp64, so the codes are bit-identical to that definition.
// This file is compiled with -ffp-contract=off.

#include "cl_device.h"
#include "cl_internal.h"

namespace cl {

__device__ double f16_bits_to_f64(uint16_t h) {
    return static_cast<double>(static_cast<float>(__builtin_bit_cast(f16, h)));
}

// One thread per (row, group).  Offline step: simple and exact over fast.
__global__ void quantize_pack_kernel(const float* __restrict__ W, int d_out, int d_in, int bits,
                                     int G, uint32_t* __restrict__ q, uint16_t* __restrict__ s,
                                     uint16_t* __restrict__ z) {
    const int groups = d_in / G;
    const long long gid = static_cast<long long>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (gid >= static_cast<long long>(d_out) * groups) return;
    const int o = static_cast<int>(gid / groups);
    const int g = static_cast<int>(gid % groups);
    const float* w = W + static_cast<size_t>(o) * d_in + static_cast<size_t>(g) * G;
    const int qmax = (1 << bits) - 1;

    double lo = 0.0, hi = 0.0;
    for (int c = 0; c < G; ++c) {
        double v = static_cast<double>(w[c]);
        lo = v < lo ? v : lo;
        hi = v > hi ? v : hi;
    }
    if (hi == lo) { lo = -1.0; hi = 1.0; }
    const double step = (hi - lo) / static_cast<double>(qmax);
    uint16_t sb = f64_to_f16_rne(step);
    if (sb == 0) sb = 0x0001u;                 // smallest positive subnormal, 2^-24
    if (sb >= 0x7c00u) sb = 0x7bffu;           // largest finite, 65504
    const double s16 = f16_bits_to_f64(sb);
    double zf = rint(-lo / s16);
    zf = zf < 0.0 ? 0.0 : (zf > qmax ? static_cast<double>(qmax) : zf);

    const size_t gi = static_cast<size_t>(o) * groups + g;
    s[gi] = sb;
    z[gi] = f32_to_f16_bits(static_cast<float>(zf));  // small integer: exact

    // the group's codes as a bit string, LSB first (code j at bits bits * j ..
    // bits * j + bits - 1), cut into 32-bit words; G * bits is a multiple of
    // 32, so the group owns whole words.  A 3-bit code can straddle two words:
    // each word takes the bits of every code that overlaps it.
    const int wpg = G * bits / 32;
    uint32_t* qrow = q + static_cast<size_t>(o) * (static_cast<size_t>(d_in) * bits / 32) +
                     static_cast<size_t>(g) * wpg;
    for (int wi = 0; wi < wpg; ++wi) {
        uint32_t word = 0;
        for (int j = (32 * wi) / bits; j < G && bits * j < 32 * wi + 32; ++j) {
            double r = rint(static_cast<double>(w[j]) / s16) + zf;
            r = r < 0.0 ? 0.0 : (r > qmax ? static_cast<double>(qmax) : r);
            const uint32_t code = static_cast<uint32_t>(r);
            const int bp = bits * j - 32 * wi;        // -bits < bp < 32
            word |= bp >= 0 ? code << bp : code >> (-bp);
        }
        qrow[wi] = word;
    }
}

__global__ void dequantize_kernel(const uint32_t* __restrict__ q, const uint16_t* __restrict__ s,
                                  const uint16_t* __restrict__ z, int d_out, int d_in, int bits,
                                  int G, float* __restrict__ out) {
    const long long i = static_cast<long long>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i >= static_cast<long long>(d_out) * d_in) return;
    const int o = static_cast<int>(i / d_in);
    const int c = static_cast<int>(i % d_in);
    // code c: bits bits * c .. of the row's bit string (possibly two words)
    const uint32_t* row = q + static_cast<size_t>(o) * (static_cast<size_t>(d_in) * bits / 32);
    const int bp = bits * c;
    const int wi = bp >> 5, off = bp & 31;
    uint64_t two = row[wi];
    if (off + bits > 32) two |= static_cast<uint64_t>(row[wi + 1]) << 32;
    const int code = static_cast<int>((two >> off) & ((1u << bits) - 1u));
    const size_t gi = static_cast<size_t>(o) * (d_in / G) + c / G;
    out[i] = f16_bits_to_f32(s[gi]) * (static_cast<float>(code) - f16_bits_to_f32(z[gi]));
}

hipError_t launch_quantize_pack(const float* W, int d_out, int d_in, int bits, int G, uint32_t* q,
                                uint16_t* s, uint16_t* z, hipStream_t st) {
    const long long n = static_cast<long long>(d_out) * (d_in / G);
    const int block = 256;
    const unsigned grid = static_cast<unsigned>((n + block - 1) / block);
    hipLaunchKernelGGL(quantize_pack_kernel, dim3(grid), dim3(block), 0, st, W, d_out, d_in, bits,
                       G, q, s, z);
    return hipGetLastError();
}

hipError_t launch_dequantize(const QW& w, float* out, hipStream_t st) {
    const long long n = static_cast<long long>(w.d_out) * w.d_in;
    const int block = 256;
    const unsigned grid = static_cast<unsigned>((n + block - 1) / block);
    hipLaunchKernelGGL(dequantize_kernel, dim3(grid), dim3(block), 0, st, w.q, w.s, w.z, w.d_out,
                       w.d_in, w.bits, w.G, out);
    return hipGetLastError();
}

}  // namespace cl
