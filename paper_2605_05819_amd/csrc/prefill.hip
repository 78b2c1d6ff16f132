// Prefill path of the error-compensated quantized linear (many tokens):
//
//     Y = X deq(Q)^T + (X A[:r]^T) B[:, :r]^T                   (Section 4.1)
//
// X [M][K] activations, Q [N][K] packed codes, A [r_max][K], B [N][r_max].
// This is a dense contraction, so it runs on MFMA (v_mfma_f32_16x16x32_f16):
//
//  1. lowrank_t_kernel: T = X A[:r]^T in fp32, rounded to fp16, zero-padded
//     to a multiple of 32 columns (a few percent of the work).
//  2. prefill_kernel: 256 x 128 output tiles (tokens x weight rows), K in
//     steps of 64, double-buffered LDS.  Each K step's packed codes are
//     dequantized by the workgroup into an fp16 tile s * (q - z) (exact q - z
//     via the 1024 + q trick, one rounding for the scale) and written to LDS
//     in the pair order the unpack produces; the activation tile is written
//     in the same permuted k order (bf16 converted to fp16 on the way), so
//     the contraction is unchanged.  Four waves compute 128 x 64 each
//     (8 x 4 MFMA tiles).  The rank-r correction is one or more extra K steps
//     over [T | B] accumulated into the same tile before the store.
//  Workgroups are numbered so that the N tiles of one 256-token block run on
//  one XCD (workgroup i runs on XCD i mod 8) and share its L2 copy of X.

#include "cl_device.h"
#include "cl_internal.h"

namespace cl {

namespace {

constexpr int BM = 256, BN = 128, BK = 64;
constexpr int LDK = BK + 8;          // LDS row pitch in halves (padding against bank conflicts)

// 8 activations -> fp16, in the pair order (x0,x4),(x1,x5),(x2,x6),(x3,x7)
__device__ __forceinline__ u32x4 act8_permuted(u32x4 u, int act) {
    if (act != DT_FP16) {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            f16x2 h;
            h.x = act_to_f16(static_cast<uint16_t>(u[k] & 0xffff), act);
            h.y = act_to_f16(static_cast<uint16_t>(u[k] >> 16), act);
            u[k] = __builtin_bit_cast(uint32_t, h);
        }
    }
    const uint32_t u0 = u[0], u1 = u[1], u2 = u[2], u3 = u[3];
    u32x4 r;
    r[0] = (u0 & 0xffffu) | (u2 << 16);           // x0, x4
    r[1] = (u0 >> 16) | (u2 & 0xffff0000u);       // x1, x5
    r[2] = (u1 & 0xffffu) | (u3 << 16);           // x2, x6
    r[3] = (u1 >> 16) | (u3 & 0xffff0000u);       // x3, x7
    return r;
}

// 8 activations -> fp16, natural order
__device__ __forceinline__ u32x4 act8_natural(u32x4 u, int act) {
    if (act != DT_FP16) {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            f16x2 h;
            h.x = act_to_f16(static_cast<uint16_t>(u[k] & 0xffff), act);
            h.y = act_to_f16(static_cast<uint16_t>(u[k] >> 16), act);
            u[k] = __builtin_bit_cast(uint32_t, h);
        }
    }
    return u;
}

// One 32-bit word of 4-bit codes -> 8 fp16 values s * (q - z) in the order
// (q0,q4),(q1,q5),(q2,q6),(q3,q7).  (q | 0x6400) is the fp16 1024 + q; minus
// (1024 + z) is the exact small integer q - z; one multiply rounds.
__device__ __forceinline__ u32x4 dequant_word4(uint32_t w, f16x2 s2, f16x2 zz) {
    u32x4 r;
#pragma unroll
    for (int p = 0; p < 4; ++p) {
        const f16x2 h = __builtin_bit_cast(f16x2, ((w >> (4 * p)) & 0x000F000Fu) | 0x64006400u);
        r[p] = __builtin_bit_cast(uint32_t, (h - zz) * s2);
    }
    return r;
}

// One 8-code half (h = 0: codes 0..7, h = 1: codes 8..15) of a 32-bit word of
// 2-bit codes -> 8 fp16 values s * (q - z) in the same pair order as the
// 4-bit path, (q0,q4),(q1,q5),(q2,q6),(q3,q7) of the half: the half is copied
// into the low 16 bits and its upper four codes into bits 16..23, so one
// shift-and-mask yields each pair.
__device__ __forceinline__ u32x4 dequant_half2(uint32_t w, int h, f16x2 s2, f16x2 zz) {
    const uint32_t v = h == 0 ? ((w & 0xFFFFu) | ((w & 0xFF00u) << 8)) : ((w >> 16) | ((w >> 24) << 16));
    u32x4 r;
#pragma unroll
    for (int p = 0; p < 4; ++p) {
        const f16x2 q = __builtin_bit_cast(f16x2, ((v >> (2 * p)) & 0x00030003u) | 0x64006400u);
        r[p] = __builtin_bit_cast(uint32_t, (q - zz) * s2);
    }
    return r;
}

__device__ __forceinline__ f32x4 mfma(const u32x4& a, const u32x4& b, const f32x4& c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c,
                                                  0, 0, 0);
}

struct PrefillArgs {
    const uint32_t* q;
    const uint16_t* s;
    const uint16_t* z;
    const uint16_t* B;       // [N][r_max] fp16
    const uint16_t* X;       // [M][K] fp16/bf16 bits
    const uint16_t* T;       // [M][r_pad] fp16 (workspace)
    void* Y;                 // [M][N]
    int M, N, K, G, rank, r_max, r_pad, act, out;
    int mblocks;             // ceil(M / BM)
};

// T = X A[:r]^T for 16 tokens x 64 factor columns per workgroup; the four
// waves split K and every wave keeps 8 k-blocks of loads in flight; partial
// tiles are summed through LDS in a fixed order.  MFMA A operand = X rows,
// B operand = rows of A.  Output fp16, zero for columns >= rank.
__global__ __launch_bounds__(256) void lowrank_t_kernel(const uint16_t* __restrict__ X,
                                                        const uint16_t* __restrict__ A, uint16_t* __restrict__ T,
                                                        int M, int K, int rank, int r_pad, int act) {
    constexpr int U = 8;                               // k blocks of 32 per batch
    __shared__ f32x4 part[4][4][64];
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int mtile = blockIdx.x;                      // 16 tokens
    const int ntile = blockIdx.y;                      // 64 factor columns
    const int m = mtile * 16 + (lane & 15);
    const int kq = 8 * (lane >> 4);                    // this lane's 8 k within a 32 block
    const bool mval = m < M;
    const uint16_t* xr = X + static_cast<size_t>(mval ? m : 0) * K;
    f32x4 acc[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
    const uint16_t* ar[4];
    bool nval[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int n = ntile * 64 + j * 16 + (lane & 15);
        nval[j] = n < rank;
        ar[j] = A + static_cast<size_t>(nval[j] ? n : 0) * K;
    }
    const int nkb = K / 32;                            // k blocks of 32; this wave takes a quarter
    const int kbeg = 32 * (wave * nkb / 4), kend = 32 * ((wave + 1) * nkb / 4);
    for (int k0 = kbeg; k0 < kend; k0 += 32 * U) {
        u32x4 xa[U], av[U][4];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int k = k0 + 32 * u;
            const int kc = k < kend ? k : (kbeg < kend ? kbeg : 0);
            xa[u] = *reinterpret_cast<const u32x4*>(xr + kc + kq);
#pragma unroll
            for (int j = 0; j < 4; ++j) av[u][j] = *reinterpret_cast<const u32x4*>(ar[j] + kc + kq);
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const bool live = k0 + 32 * u < kend;
            u32x4 x8 = act8_natural(xa[u], act);
            if (!mval || !live) x8 = u32x4{0, 0, 0, 0};
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                u32x4 a8 = av[u][j];
                if (!nval[j]) a8 = u32x4{0, 0, 0, 0};
                acc[j] = mfma(x8, a8, acc[j]);
            }
        }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) part[wave][j][lane] = acc[j];
    __syncthreads();
    if (wave != 0) return;
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[j] = part[0][j][lane] + part[1][j][lane] + part[2][j][lane] + part[3][j][lane];
    // acc[j][e] = T[mtile*16 + 4*(lane/16) + e][ntile*64 + j*16 + lane%16]
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int n = ntile * 64 + j * 16 + (lane & 15);
        if (n >= r_pad) continue;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int mm = mtile * 16 + 4 * (lane >> 4) + e;
            if (mm < M) T[static_cast<size_t>(mm) * r_pad + n] = f32_to_f16_bits(n < rank ? acc[j][e] : 0.f);
        }
    }
}

template <int BITS>
__global__ __launch_bounds__(256) void prefill_kernel(PrefillArgs a) {
    extern __shared__ uint32_t smem[];
    // two stages of [BM][LDK] activations and [BN][LDK] weights (fp16)
    constexpr int XS = BM * LDK / 2;   // words per activation stage
    constexpr int WS = BN * LDK / 2;   // words per weight stage
    // stage b: activations at smem + b (XS + WS), weights right after them

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    // XCD-aware order: consecutive workgroups take consecutive M blocks
    const int mb = blockIdx.x % a.mblocks;
    const int nb = blockIdx.x / a.mblocks;
    const int m0 = mb * BM, n0 = nb * BN;
    const int wm = (wave & 1) * 128;    // this wave's rows within the tile
    const int wn = (wave >> 1) * 64;    // and columns

    const int groups = a.K / a.G;
    const int words_row = a.K * BITS / 32;
    const int nsteps = a.K / BK;

    // ---- global -> register staging for one K step
    // activations: 256 rows x 64 k = 2048 x 16 B; thread t loads rows
    // (t / 8) + 32 i, 16-byte column (t % 8)
    u32x4 xr[8];
    u32x4 wr;
    uint16_t sr = 0, zr = 0;
    const int xcol = (tid & 7) * 8;
    auto load_stage = [&](int step) {
        const int k0 = step * BK;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int m = m0 + (tid >> 3) + 32 * i;
            xr[i] = *reinterpret_cast<const u32x4*>(a.X + static_cast<size_t>(m < a.M ? m : 0) * a.K + k0 + xcol);
        }
        // weights: 4-bit: thread t -> row t/2, 32 codes (k0 + 32 (t%2)); 2-bit:
        // thread t -> row t/2, 32 codes too (half of the row's 16-byte load)
        const int row = n0 + (tid >> 1);
        const int rowc = row < a.N ? row : 0;
        if (BITS == 4) {
            wr = *reinterpret_cast<const u32x4*>(a.q + static_cast<size_t>(rowc) * words_row + k0 / 8 + 4 * (tid & 1));
        } else {
            wr = *reinterpret_cast<const u32x4*>(a.q + static_cast<size_t>(rowc) * words_row + k0 / 16);
        }
        const int g = (k0 + 32 * (tid & 1)) / a.G;
        sr = a.s[static_cast<size_t>(rowc) * groups + g];
        zr = a.z[static_cast<size_t>(rowc) * groups + g];
    };
    auto store_stage = [&](int buf, int step) {
        uint32_t* xd = smem + buf * (XS + WS);
        const int k0 = step * BK;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int r = (tid >> 3) + 32 * i;
            const bool ok = m0 + r < a.M;
            u32x4 v = act8_permuted(xr[i], a.act);
            if (!ok) v = u32x4{0, 0, 0, 0};
            *reinterpret_cast<u32x4*>(xd + r * (LDK / 2) + xcol / 2) = v;
        }
        const int r = tid >> 1;
        const bool ok = n0 + r < a.N;
        const f16 s = __builtin_bit_cast(f16, sr);
        const f16 zf = static_cast<f16>(1024.0f) + __builtin_bit_cast(f16, zr);   // exact: z <= 15
        const f16x2 s2 = {s, s}, zz = {zf, zf};
        uint32_t* wd = smem + buf * (XS + WS) + XS + r * (LDK / 2) + 16 * (tid & 1);
        if (BITS == 4) {
#pragma unroll
            for (int w = 0; w < 4; ++w) {
                u32x4 v = dequant_word4(wr[w], s2, zz);
                if (!ok) v = u32x4{0, 0, 0, 0};
                *reinterpret_cast<u32x4*>(wd + 4 * w) = v;
            }
        } else {
            // the row's 64 codes are 4 words of 16; this thread takes words
            // 2 (t%2) and 2 (t%2) + 1, each as two halves of 8 codes
#pragma unroll
            for (int w = 0; w < 2; ++w) {
                const uint32_t word = wr[2 * (tid & 1) + w];
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    u32x4 v = dequant_half2(word, h, s2, zz);
                    if (!ok) v = u32x4{0, 0, 0, 0};
                    *reinterpret_cast<u32x4*>(wd + 8 * w + 4 * h) = v;
                }
            }
        }
        (void)k0;
    };

    f32x4 acc[8][4];
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    // MFMA over one LDS stage: A operand from activations, B from weights
    auto mma_stage = [&](int buf) {
        const uint32_t* xsb = smem + buf * (XS + WS);
        const uint32_t* wsb = xsb + XS;
#pragma unroll
        for (int kk = 0; kk < BK; kk += 32) {
            const int kq = kk + 8 * (lane >> 4);        // this lane's 8 k
            u32x4 bf[4];
#pragma unroll
            for (int j = 0; j < 4; ++j)
                bf[j] = *reinterpret_cast<const u32x4*>(wsb + (wn + 16 * j + (lane & 15)) * (LDK / 2) + kq / 2);
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const u32x4 af = *reinterpret_cast<const u32x4*>(xsb + (wm + 16 * i + (lane & 15)) * (LDK / 2) + kq / 2);
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = mfma(af, bf[j], acc[i][j]);
            }
        }
    };

    // ---- main loop: double-buffered LDS, next step's global loads in flight
    load_stage(0);
    store_stage(0, 0);
    __syncthreads();
    for (int step = 0; step < nsteps; ++step) {
        const int buf = step & 1;
        if (step + 1 < nsteps) load_stage(step + 1);
        mma_stage(buf);
        if (step + 1 < nsteps) store_stage(buf ^ 1, step + 1);
        __syncthreads();
    }

    // ---- rank-r correction: K steps over [T | B] (natural order), same tile
    for (int k0 = 0; k0 < a.r_pad; k0 += BK) {
        const int buf = 0;
        uint32_t* xd = smem + buf * (XS + WS);
        uint32_t* wd = xd + XS;
        // T tile: 256 rows x 64 (zero past r_pad); B tile: 128 rows x 64
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int r = (tid >> 3) + 32 * i;
            const int m = m0 + r;
            const int k = k0 + xcol;
            u32x4 v = u32x4{0, 0, 0, 0};
            if (m < a.M && k < a.r_pad) v = *reinterpret_cast<const u32x4*>(a.T + static_cast<size_t>(m) * a.r_pad + k);
            *reinterpret_cast<u32x4*>(xd + r * (LDK / 2) + xcol / 2) = v;
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int r = (tid >> 3) + 32 * i;          // 128 rows, 8 x 8 halves each
            const int n = n0 + r;
            uint32_t v[4] = {0, 0, 0, 0};
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int k = k0 + xcol + e;
                const uint16_t bv = (n < a.N && k < a.rank) ? a.B[static_cast<size_t>(n) * a.r_max + k] : 0;
                v[e / 2] |= static_cast<uint32_t>(bv) << (16 * (e & 1));
            }
            *reinterpret_cast<u32x4*>(wd + r * (LDK / 2) + xcol / 2) = u32x4{v[0], v[1], v[2], v[3]};
        }
        __syncthreads();
        mma_stage(buf);
        __syncthreads();
    }

    // ---- store: acc[i][j][e] = Y[m0 + wm + 16 i + 4 (lane/16) + e][n0 + wn + 16 j + lane%16]
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int n = n0 + wn + 16 * j + (lane & 15);
            if (n >= a.N) continue;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int m = m0 + wm + 16 * i + 4 * (lane >> 4) + e;
                if (m < a.M) store_out(a.Y, static_cast<size_t>(m) * a.N + n, acc[i][j][e], a.out);
            }
        }
}

size_t up256(size_t n) { return (n + 255) / 256 * 256; }

}  // namespace

size_t prefill_workspace_bytes(const QW&, const LR& c, int M) {
    const int r_pad = (c.rank + 31) / 32 * 32;
    return up256(static_cast<size_t>(M) * r_pad * 2);
}

size_t prefill_lds_bytes() { return static_cast<size_t>(2) * (BM + BN) * LDK * 2; }

hipError_t launch_linear_prefill(const QW& w, const LR& c, const void* X, int M, int act, void* Y, int out,
                                 void* ws, hipStream_t st) {
    PrefillArgs a;
    a.q = w.q; a.s = w.s; a.z = w.z; a.B = c.B;
    a.X = static_cast<const uint16_t*>(X);
    a.T = static_cast<const uint16_t*>(ws);
    a.Y = Y;
    a.M = M; a.N = w.d_out; a.K = w.d_in; a.G = w.G;
    a.rank = c.rank; a.r_max = c.r_max; a.r_pad = (c.rank + 31) / 32 * 32;
    a.act = act; a.out = out;
    a.mblocks = (M + BM - 1) / BM;
    if (c.rank > 0) {
        const dim3 grid((M + 15) / 16, (a.r_pad + 63) / 64);
        hipLaunchKernelGGL(lowrank_t_kernel, grid, dim3(256), 0, st, a.X, c.A, static_cast<uint16_t*>(ws), M, w.d_in,
                           c.rank, a.r_pad, act);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    const size_t lds = prefill_lds_bytes();
    const unsigned blocks = static_cast<unsigned>(a.mblocks * ((w.d_out + BN - 1) / BN));
    if (w.bits == 4) {
        static bool attr4 = false;
        if (!attr4) {
            (void)hipFuncSetAttribute(reinterpret_cast<const void*>(prefill_kernel<4>),
                                hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
            attr4 = true;
        }
        hipLaunchKernelGGL(prefill_kernel<4>, dim3(blocks), dim3(256), lds, st, a);
    } else {
        static bool attr2 = false;
        if (!attr2) {
            (void)hipFuncSetAttribute(reinterpret_cast<const void*>(prefill_kernel<2>),
                                hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
            attr2 = true;
        }
        hipLaunchKernelGGL(prefill_kernel<2>, dim3(blocks), dim3(256), lds, st, a);
    }
    return hipGetLastError();
}

}  // namespace cl
