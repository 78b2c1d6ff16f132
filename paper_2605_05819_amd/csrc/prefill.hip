// Prefill path of the error-compensated quantized linear (many tokens):
//
//     Y = X deq(Q)^T + (X A[:r]^T) B[:, :r]^T                   (Section 4.1)
//
// X [M][K] activations, Q [N][K] packed codes, A [r_max][K], B [N][r_max].
// This is a dense contraction, so it runs on MFMA (v_mfma_f32_16x16x32_f16):
//
//  1. xt_partial_kernel writes X' (below) and the fp32 partial products of
//     X A[:r]^T over 512-column parts of K; t_reduce_kernel sums the parts
//     in order into T, rounded to fp16 and zero-padded to a multiple of 32
//     columns.  Without a rank term, xprep_kernel writes X' alone.
//     X' = X as fp16 (bf16 converted) with every 8 consecutive k reordered
//     (k0,k4,k1,k5,k2,k6,k3,k7): the order in which the code unpack below
//     produces weights, so the contraction is unchanged.
//  2. prefill_kernel: 128 x 256 output tiles (tokens x weight rows; 128 x 128
//     when 256-row tiles would leave CUs without two workgroups: 4096 x 4096
//     at M = 2048 went from 133 to 117 us, while 14336 x 4096 stays faster
//     with 256 rows, 322 against 350 us), K in steps of 128 codes.  X' tiles
//     go from global memory straight into LDS (global_load_lds, 16 bytes per
//     lane, two 32 KB stages, chunks XOR-swizzled by row so the MFMA operand
//     reads are bank-conflict free).  Each of the four waves owns 128 tokens
//     x 16 JT weight rows (8 x JT MFMA tiles): it loads its rows' packed
//     codes for the next K step into registers (one 16-byte load per lane
//     and fragment: 32 codes of one quantization group, so one scale and zero
//     per lane) and dequantizes them as s * (q - z) in fp16 (the integer
//     q - z is formed exactly from the code OR-ed into the mantissa of
//     1024.0, then one rounding for the scale).  The K step is software-
//     pipelined: the code words of MFMA step t + 1 are dequantized in halves
//     between the MFMAs of step t, and each X' operand is read from LDS a
//     few MFMA groups before its use (14336 x 4096: 320 -> 308 us; 4096 x
//     4096: 122 -> 113 us).  No weight tile goes through LDS and no wave
//     repeats another's dequantization.  The workgroup's scales and zeros do
//     go through LDS, in double-buffered windows of 8 groups per row (one
//     16-byte load per thread and array per window): per-lane 2-byte
//     gathers had cost 13 % of the kernel's time.  The rank-r correction is
//     extra MFMA steps over [T | B] (read from global memory) into the same
//     accumulators.
//     A 256-token tile (one workgroup per CU, 16 token tiles per wave, so
//     each dequantized operand feeds 16 MFMAs) was built and measured: with
//     32 rows per wave it ran 401 us on 14336 x 4096 (X' operand reads at
//     512 bytes of LDS per MFMA, one wave per SIMD to hide latency), and 64
//     rows per wave need more than the 512 registers a lane can hold.
//  Workgroups are numbered so that the N tiles of one 128-token block run on
//  one XCD (workgroup i runs on XCD i mod 8) and share its L2 copy of X'.

#include "cl_device.h"
#include "cl_internal.h"
#include "mfma_common.h"

namespace cl {

namespace {

constexpr int BK = 128;

// 8 activations -> fp16, in the pair order (x0,x4),(x1,x5),(x2,x6),(x3,x7)
__device__ __forceinline__ u32x4 act8_permuted(u32x4 u, int act) {
    u = act8_to_f16(u, act);
    const uint32_t u0 = u[0], u1 = u[1], u2 = u[2], u3 = u[3];
    u32x4 r;
    r[0] = (u0 & 0xffffu) | (u2 << 16);           // x0, x4
    r[1] = (u0 >> 16) | (u2 & 0xffff0000u);       // x1, x5
    r[2] = (u1 & 0xffffu) | (u3 << 16);           // x2, x6
    r[3] = (u1 >> 16) | (u3 & 0xffff0000u);       // x3, x7
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

// One 8-code unit t (codes 8t .. 8t + 7) of a lane's 3-bit chunk -> 8 fp16
// values s * (q - z), pair order as above: q - z exact (codes3_minus_zero),
// then one rounding per value.
__device__ __forceinline__ u32x4 dequant_unit3(const uint32_t (&w)[3], int t, const Zq3& zq, f16x2 s2,
                                               const uint32_t (&m)[3], uint32_t bias) {
    u32x4 r = codes3_minus_zero(spread_unit3(w[0], w[1], w[2], t), zq, m, bias);
#pragma unroll
    for (int p = 0; p < 4; ++p) {
        const uint32_t v = r[p];
        r[p] = __builtin_bit_cast(uint32_t, __builtin_bit_cast(f16x2, v) * s2);
    }
    return r;
}

// One half of dequant_half2's result: pairs 2 h and 2 h + 1 of the 8-code
// half u of the word; the same values.
__device__ __forceinline__ void dequant_quarter2(uint32_t w, int u, int h, f16x2 s2, f16x2 zz, uint32_t& lo,
                                                 uint32_t& hi) {
    const uint32_t v = u == 0 ? ((w & 0xFFFFu) | ((w & 0xFF00u) << 8)) : ((w >> 16) | ((w >> 24) << 16));
    const f16x2 a = __builtin_bit_cast(f16x2, ((v >> (4 * h)) & 0x00030003u) | 0x64006400u);
    const f16x2 b = __builtin_bit_cast(f16x2, ((v >> (4 * h + 2)) & 0x00030003u) | 0x64006400u);
    lo = __builtin_bit_cast(uint32_t, (a - zz) * s2);
    hi = __builtin_bit_cast(uint32_t, (b - zz) * s2);
}

// One half of dequant_unit3: h = 0 gives pairs 0 and 1 (r[0], r[1]), h = 1
// pairs 2 and 3; the same values.
__device__ __forceinline__ void dequant_half3(const uint32_t (&w)[3], int t, int h, const Zq3& zq, f16x2 s2,
                                              const uint32_t (&m)[3], uint32_t bias, uint32_t& lo, uint32_t& hi) {
    const uint32_t v = spread_unit3(w[0], w[1], w[2], t);
    const f16x2 e8 = {static_cast<f16>(0.125f), static_cast<f16>(0.125f)};
    const f16x2 e64 = {static_cast<f16>(0.015625f), static_cast<f16>(0.015625f)};
    f16x2 a, b;
    if (h == 0) {
        a = __builtin_bit_cast(f16x2, and_or(v, m[0], bias)) + zq.c[0];
        b = __builtin_elementwise_fma(__builtin_bit_cast(f16x2, and_or(v, m[1], bias)), e8, zq.c[1]);
    } else {
        a = __builtin_elementwise_fma(__builtin_bit_cast(f16x2, and_or(v, m[2], bias)), e64, zq.c[2]);
        b = __builtin_elementwise_fma(__builtin_bit_cast(f16x2, and_or(v >> 3, m[2], bias)), e64, zq.c[2]);
    }
    lo = __builtin_bit_cast(uint32_t, a * s2);
    hi = __builtin_bit_cast(uint32_t, b * s2);
}

struct PrefillArgs {
    const uint32_t* q;
    const uint16_t* s;
    const uint16_t* z;
    const uint16_t* B;       // [N][r_max] fp16
    const uint16_t* Xp;      // [M][K] X' fp16, k-reordered (workspace)
    const uint16_t* T;       // [M][r_pad] fp16 (workspace)
    void* Y;                 // [M][N]
    int M, N, K, G, rank, r_max, r_pad, out;
    int mblocks;             // ceil(M / tokens per workgroup)
};

// X' for 8 activations of a 16-byte chunk: fp16, order (k0,k4,k1,k5,...).
__device__ __forceinline__ void store_xp(uint16_t* Xp, size_t idx, u32x4 raw, int act) {
    *reinterpret_cast<u32x4*>(Xp + idx) = act8_permuted(raw, act);
}

// X' alone (no rank term): one thread per 16-byte chunk of X.
__global__ __launch_bounds__(256) void xprep_kernel(const uint16_t* __restrict__ X, uint16_t* __restrict__ Xp,
                                                    long long chunks, int act) {
    const long long c = static_cast<long long>(blockIdx.x) * 256 + threadIdx.x;
    if (c >= chunks) return;
    store_xp(Xp, static_cast<size_t>(c) * 8, *reinterpret_cast<const u32x4*>(X + static_cast<size_t>(c) * 8), act);
}

// One launch for X' and the partial low-rank products: workgroup (64-token
// tile, 256-column part of K).  Its threads convert the tile's X to X' and
// write it both to the workspace (the GEMM's operand) and to LDS (each row's
// 16-byte chunk c at c ^ (row % 16), so the 16 rows of an MFMA operand read
// land in distinct banks); then wave w multiplies the tile by rank rows
// 16 w .. 16 w + 15 (then + 64, ...) of A over the part's columns on MFMA
// (A's 8-element runs reordered in registers as X' is, so each product pairs
// the same elements) and writes the fp32 partial P[part][token][column].
// Each X element is read once and each A row once per 64 tokens (one
// workgroup per 16 tokens and 32 factor columns over all of K had read A 128
// times and X twice, 16 rows x 64 bytes per load instruction: 20.4 us for
// M = 2048, K = 4096 with X' written beside it; now 11.3 us, and 12.4 /
// 13.3 / 11.6 us with 512 columns / 32 tokens and 512 columns / 128 tokens
// per workgroup).
constexpr int XT_M = 64, XT_K = 256;

__global__ __launch_bounds__(256) void xt_partial_kernel(const uint16_t* __restrict__ X,
                                                         const uint16_t* __restrict__ A, uint16_t* __restrict__ Xp,
                                                         float* __restrict__ P, int M, int K, int rank, int r_pad,
                                                         int act, int mtiles) {
    constexpr int CPR = XT_K / 8;                  // 16-byte chunks per tile row
    constexpr int PER = XT_M * CPR / 256;          // chunks per thread
    constexpr int MTL = XT_M / 16;                 // MFMA token tiles
    __shared__ u32x4 xs[XT_M * CPR];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int mt = static_cast<int>(blockIdx.x) % mtiles, part = static_cast<int>(blockIdx.x) / mtiles;
    const int m0 = mt * XT_M, k0 = part * XT_K;
    const int kw = min(XT_K, K - k0);              // a multiple of 64
    const u32x4 zero = {0u, 0u, 0u, 0u};
    // X' of the tile: every load first (clamped addresses), then the stores
    u32x4 v[PER];
#pragma unroll
    for (int i = 0; i < PER; ++i) {
        const int c = tid + 256 * i, row = c / CPR, cc = c % CPR;
        const bool ok = m0 + row < M && 8 * cc < kw;
        v[i] = *reinterpret_cast<const u32x4*>(X + static_cast<size_t>(ok ? m0 + row : 0) * K + k0 + (ok ? 8 * cc : 0));
    }
#pragma unroll
    for (int i = 0; i < PER; ++i) {
        const int c = tid + 256 * i, row = c / CPR, cc = c % CPR;
        const bool ok = m0 + row < M && 8 * cc < kw;
        const u32x4 xp = act8_permuted(v[i], act);
        if (ok) *reinterpret_cast<u32x4*>(Xp + static_cast<size_t>(m0 + row) * K + k0 + 8 * cc) = xp;
        xs[row * CPR + (cc ^ (row & 15))] = ok ? xp : zero;
    }
    __syncthreads();
    const int g = lane >> 4, r = lane & 15;
    const int nsteps = kw / 32;
    for (int nt = wave; nt * 16 < r_pad; nt += 4) {
        const int n = nt * 16 + r;
        const bool nv = n < rank;
        const uint16_t* ar = A + static_cast<size_t>(nv ? n : 0) * K + k0;
        f32x4 acc[MTL];
#pragma unroll
        for (int i = 0; i < MTL; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
        for (int s0 = 0; s0 < nsteps; s0 += 8) {
            u32x4 av[8];                           // 8 steps of A loads in flight
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int st = s0 + u < nsteps ? s0 + u : 0;
                av[u] = *reinterpret_cast<const u32x4*>(ar + st * 32 + 8 * g);
            }
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const bool live = s0 + u < nsteps;
                const int ch = (live ? s0 + u : 0) * 4 + g;
                const u32x4 a8 = (nv && live) ? act8_permuted(av[u], DT_FP16) : zero;
#pragma unroll
                for (int i = 0; i < MTL; ++i) acc[i] = mfma(xs[(16 * i + r) * CPR + (ch ^ r)], a8, acc[i]);
            }
        }
        // acc[i][e] = partial T[m0 + 16 i + 4 g + e][n]
#pragma unroll
        for (int i = 0; i < MTL; ++i)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int m = m0 + 16 * i + 4 * g + e;
                if (m < M) P[(static_cast<size_t>(part) * M + m) * r_pad + n] = acc[i][e];
            }
    }
}

// T = the partials summed in part order, rounded to fp16 (zero for columns
// at or past the rank): four elements of T per thread (r_pad is a multiple
// of 32, so four never straddle a row), eight parts' loads in flight.
__global__ __launch_bounds__(256) void t_reduce_kernel(const float* __restrict__ P, uint16_t* __restrict__ T, int M,
                                                       int rank, int r_pad, int parts) {
    const long long i4 = static_cast<long long>(blockIdx.x) * 256 + threadIdx.x;
    const long long n_all = static_cast<long long>(M) * r_pad;
    if (4 * i4 >= n_all) return;
    const f32x4* P4 = reinterpret_cast<const f32x4*>(P);
    f32x4 sum = {0.f, 0.f, 0.f, 0.f};
    for (int p0 = 0; p0 < parts; p0 += 8) {
        f32x4 v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = P4[static_cast<size_t>(p0 + u < parts ? p0 + u : 0) * (n_all / 4) + i4];
#pragma unroll
        for (int u = 0; u < 8; ++u)
            if (p0 + u < parts) sum += v[u];
    }
    const int n0 = static_cast<int>((4 * i4) % r_pad);
    uint32_t h[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) h[e] = f32_to_f16_bits(n0 + e < rank ? sum[e] : 0.f);
    reinterpret_cast<uint2*>(T)[i4] = make_uint2(h[0] | (h[1] << 16), h[2] | (h[3] << 16));
}

// 16 bytes per lane from global memory straight into LDS (lane l's bytes
// land at dst + 16 l; dst is wave-uniform).  A plain function, so the
// builtin never sees a template-dependent LDS operand (the host compiler
// then drops the kernel's launch stub).
__device__ __forceinline__ void global_to_lds16(const uint16_t* src, u32x4* dst) {
    __builtin_amdgcn_global_load_lds(src, (__attribute__((address_space(3))) void*)dst, 16, 0, 0);
}

// LDS slot of X' chunk c in a row whose low four index bits are r: c ^ f(r)
// with f(r) = (r >> 1 & 3) | (r & 1) << 2 | (r & 8), a permutation of 0..15.
// An MFMA operand read has lanes r = 0..15 of lane group g on chunk 4 g + t;
// the 16 rows give 16 distinct slots, and the two lane groups of one 32-lane
// half (chunks differing in bit 2) land in opposite bank halves for odd and
// even rows, so a 128-bit read has no bank conflict.
__device__ __forceinline__ int xswz(int r) { return ((r >> 1) & 3) | ((r & 1) << 2) | (r & 8); }

// One K step's packed codes of a lane: 32 codes of one weight row (4-bit:
// four words; 3-bit: three; 2-bit: two), with their group's scale and zero.
template <int BITS>
struct WStep {
    uint32_t w[BITS];        // 32 codes = BITS words
};

template <int BITS, int JT>
__global__ __launch_bounds__(256, 2) void prefill_kernel(PrefillArgs a) {
    // MT token tiles and JT row tiles of 16 per wave: the workgroup covers
    // BM = 16 MT tokens x 64 JT weight rows
    constexpr int MT = 8;
    constexpr int BM = 16 * MT;
    constexpr int BNT = 64 * JT;
    // LDS (dynamic, prefill_lds_bytes): two stages of X', [BM rows][16
    // chunks of 8 k], chunk c of row r stored at slot c ^ xswz(r & 15); then
    // the scales and zeros of the workgroup's BNT rows, windows of 8
    // consecutive groups, double-buffered: [buffer][scale, zero][group][row]
    // (a lane's read of its row's value is then one of 16 consecutive 2-byte
    // entries: no bank conflicts, where [row][8] had 16-byte strides)
    extern __shared__ u32x4 smem[];
    u32x4 (*xs)[BM * 16] = reinterpret_cast<u32x4 (*)[BM * 16]>(smem);
    uint16_t (*szw)[2][8][BNT] = reinterpret_cast<uint16_t (*)[2][8][BNT]>(smem + 2 * BM * 16);

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 4;               // lane group: k sub-block of an MFMA step
    const int r = lane & 15;
    // XCD-aware order: consecutive workgroups take consecutive M blocks
    const int mb = blockIdx.x % a.mblocks;
    const int nb = blockIdx.x / a.mblocks;
    const int m0 = mb * BM, n0 = nb * BNT + wave * 16 * JT;
    const int nk = (a.K + BK - 1) / BK;
    const int groups = a.K / a.G;
    const int words_row = a.K * BITS / 32;

    // X' tile of K step kb into stage st: wave w fills slots [64 MT w, 64 MT (w + 1))
    // Rows past M read the workspace's padding (X' holds a whole number of
    // 128-token blocks): their values only reach output rows that are never
    // stored, so the row offset splits into a wave-uniform part and one of
    // four per-lane patterns, and no per-load offset stays live in a
    // register.
    auto load_x = [&](int kb, int st) {
        const int k0 = kb * BK;
#pragma unroll
        for (int j = 0; j < MT; ++j) {
            const int blk = wave * MT + j;                 // 64 slots = 4 rows
            const int rl = lane >> 4;
            // (4 blk + rl) & 15 == (4 j + rl) & 15: MT is a multiple of 4
            const int chunk = (lane & 15) ^ xswz((4 * j + rl) & 15);
            int k = 8 * chunk;
            if (k0 + k >= a.K) k = 0;                      // half K step: weights there are zero
            // 32-bit element offsets (the entry point bounds M K): uniform + per lane
            const unsigned ubase = static_cast<unsigned>(m0 + 4 * blk) * static_cast<unsigned>(a.K) + k0;
            const unsigned voff = static_cast<unsigned>(rl) * static_cast<unsigned>(a.K) + static_cast<unsigned>(k);
            global_to_lds16(a.Xp + ubase + voff, &xs[st][blk * 64]);
        }
    };
    // scales and zeros, window wnd (groups 8 wnd .. 8 wnd + 7) of the
    // workgroup's rows: thread tid < BNT takes row nb BNT + tid.  fetch_sz issues
    // the loads (one 16-byte load per array when the rows are 16-byte
    // aligned); store_sz writes them to LDS buffer wnd % 2 a step later,
    // when they have landed, so no wave waits on them (direct global-to-LDS
    // loads of the windows measured 11 % slower)
    const bool sz16 = groups % 8 == 0 && (reinterpret_cast<uintptr_t>(a.s) & 15) == 0 &&
                      (reinterpret_cast<uintptr_t>(a.z) & 15) == 0;
    u32x4 szs, szz;
    auto fetch_sz = [&](int wnd) {
        const int n = nb * BNT + (tid < BNT ? tid : 0);
        const int nc = n < a.N ? n : a.N - 1;
        const unsigned base = static_cast<unsigned>(nc) * static_cast<unsigned>(groups) + 8u * wnd;
        if (sz16 && 8 * wnd + 8 <= groups) {
            szs = *reinterpret_cast<const u32x4*>(a.s + base);
            szz = *reinterpret_cast<const u32x4*>(a.z + base);
        } else {
            uint32_t hs[8], hz[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const bool v = 8 * wnd + e < groups;
                hs[e] = v ? a.s[base + e] : 0u;
                hz[e] = v ? a.z[base + e] : 0u;
            }
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                szs[e] = hs[2 * e] | (hs[2 * e + 1] << 16);
                szz[e] = hz[2 * e] | (hz[2 * e + 1] << 16);
            }
        }
    };
    auto store_sz = [&](int wnd) {
        if (tid >= BNT) return;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const uint32_t se = szs[e / 2], ze = szz[e / 2];
            szw[wnd & 1][0][e][tid] = static_cast<uint16_t>(se >> (16 * (e & 1)));
            szw[wnd & 1][1][e][tid] = static_cast<uint16_t>(ze >> (16 * (e & 1)));
        }
    };
    // K steps per window of 8 groups (G / 16 >= 2: G is a multiple of 128 / bits)
    const int spw = a.G / 16;

    // this lane's codes of K step kb for its JT weight rows
    auto load_w = [&](int kb, WStep<BITS> (&ws)[JT]) {
        const int kc = kb * BK + 32 * g;                   // first code of this lane's 32
        const bool kval = kc < a.K;
#pragma unroll
        for (int j = 0; j < JT; ++j) {
            const int n = n0 + 16 * j + r;
            const int nc = n < a.N ? n : a.N - 1;
            const uint32_t* src = a.q + (static_cast<unsigned>(nc) * static_cast<unsigned>(words_row) +
                                         static_cast<unsigned>(kval ? kc * BITS / 32 : 0));
            if constexpr (BITS == 4) {
                const u32x4 v = *reinterpret_cast<const u32x4*>(src);
#pragma unroll
                for (int e = 0; e < 4; ++e) { const uint32_t ve = v[e]; ws[j].w[e] = ve; }
            } else if constexpr (BITS == 3) {
                // the 32 codes are the row's 3-word chunk kc / 32
#pragma unroll
                for (int e = 0; e < 3; ++e) ws[j].w[e] = src[e];
            } else {
                const uint2 v = *reinterpret_cast<const uint2*>(src);
                ws[j].w[0] = v.x;
                ws[j].w[1] = v.y;
            }
            // raw loads only: nothing here consumes a loaded value, so the
            // loads stay in flight through the current step's MFMAs
        }
    };

    f32x4 acc[MT][JT];
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int j = 0; j < JT; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    // four MFMA steps of 32 codes: lane group g's 8 codes of step t are codes
    // 32 g + 8 t .. + 7 of the K step, X' chunk 4 g + t
    // loop-invariant operands of the unpack: masks in scalar registers
    const uint32_t mlo = __builtin_amdgcn_readfirstlane(0x000F000Fu);
    const uint32_t mhi = __builtin_amdgcn_readfirstlane(0x00F000F0u);
    uint32_t m3[3];
#pragma unroll
    for (int p = 0; p < 3; ++p) m3[p] = __builtin_amdgcn_readfirstlane(0x00070007u << (3 * p));
    const uint32_t bias = 0x64006400u;
    const int fr = xswz(r);
    auto compute = [&](int kb, int st, const WStep<BITS> (&ws)[JT]) {
        Zq zq[JT];
        Zq3 zq3[JT];
        f16x2 s2[JT], zz[JT];
        const bool kval = kb * BK + 32 * g < a.K;
        const int gi = kval ? (kb * BK + 32 * g) / a.G : 0;
        const int wb = (gi >> 3) & 1, we = gi & 7;
#pragma unroll
        for (int j = 0; j < JT; ++j) {
            // past K or N the scale is 0: q - z is finite, so the weight is 0
            const int nl = wave * 16 * JT + 16 * j + r;
            const uint32_t zb = szw[wb][1][we][nl];
            const uint32_t sb = (kval && n0 + 16 * j + r < a.N) ? static_cast<uint32_t>(szw[wb][0][we][nl]) : 0u;
            if constexpr (BITS == 4) {
                const f16 sv = __builtin_bit_cast(f16, static_cast<uint16_t>(sb));
                zq[j] = make_zq(zb);
                s2[j] = f16x2{sv, sv};
            } else if constexpr (BITS == 3) {
                const f16 sv = __builtin_bit_cast(f16, static_cast<uint16_t>(sb));
                zq3[j] = make_zq3(zb);
                s2[j] = f16x2{sv, sv};
            } else {
                const f16 sv = __builtin_bit_cast(f16, static_cast<uint16_t>(sb));
                const f16 zf = static_cast<f16>(1024.0f) + __builtin_bit_cast(f16, static_cast<uint16_t>(zb));
                s2[j] = f16x2{sv, sv};
                zz[j] = f16x2{zf, zf};
            }
        }
        {
            // Software pipeline over the 4 MT regions of the step (region =
            // MFMA step t, token tile i: one X' operand, JT MFMAs): the X'
            // operand of the region PD ahead is read from LDS (PD regions
            // of MFMAs cover the read's latency), and the code words of step
            // t + 1 are dequantized in halves spread over the regions of
            // step t, so MFMA, LDS and VALU work interleave.  The
            // scheduling fence after each region keeps that order.
            constexpr int PD = 8 / JT;
            constexpr int NREG = 4 * MT;
            auto xop = [&](int reg) {
                const int i = reg % MT, t = reg / MT;
                return xs[st][(16 * i + r) * 16 + ((4 * g + t) ^ fr)];
            };
            u32x4 bc[JT], bn[JT], ap[PD];
#pragma unroll
            for (int q = 0; q < PD; ++q) ap[q] = xop(q);
            // the 8-code unit of step t of row tile j (4-bit: word t; 3-bit:
            // unit t of the 3-word chunk; 2-bit: half t % 2 of word t / 2),
            // whole or one half of its pairs
            auto deq_full = [&](int j, int t) {
                if constexpr (BITS == 4) return dequant_word4x(ws[j].w[t], zq[j], s2[j], mlo, mhi, bias);
                else if constexpr (BITS == 3) return dequant_unit3(ws[j].w, t, zq3[j], s2[j], m3, bias);
                else return dequant_half2(ws[j].w[t >> 1], t & 1, s2[j], zz[j]);
            };
            auto deq_half = [&](int j, int t, int h, uint32_t& lo, uint32_t& hi) {
                if constexpr (BITS == 4) dequant_half4x(ws[j].w[t], h, zq[j], s2[j], mlo, mhi, bias, lo, hi);
                else if constexpr (BITS == 3) dequant_half3(ws[j].w, t, h, zq3[j], s2[j], m3, bias, lo, hi);
                else dequant_quarter2(ws[j].w[t >> 1], t & 1, h, s2[j], zz[j], lo, hi);
            };
#pragma unroll
            for (int j = 0; j < JT; ++j) bc[j] = deq_full(j, 0);
#pragma unroll
            for (int t = 0; t < 4; ++t) {
#pragma unroll
                for (int i = 0; i < MT; ++i) {
                    const int reg = t * MT + i;
                    const u32x4 a0 = ap[reg % PD];
                    if (reg + PD < NREG) ap[reg % PD] = xop(reg + PD);
#pragma unroll
                    for (int j = 0; j < JT; ++j) acc[i][j] = mfma(a0, bc[j], acc[i][j]);
                    constexpr int NH = 2 * JT;             // word halves per step
                    if (t < 3 && (i * NH) % MT == 0) {
                        const int hx = i * NH / MT, j = hx / 2, h = hx % 2;
                        uint32_t lo, hi;
                        deq_half(j, t + 1, h, lo, hi);
                        bn[j][2 * h] = lo;
                        bn[j][2 * h + 1] = hi;
                    }
                    // region order: MFMA, the prefetch read, then VALU work
                    // between the MFMAs (masks: 0x008 MFMA, 0x100 LDS read,
                    // 0x002 VALU)
#pragma unroll
                    for (int m = 0; m < JT; ++m) {
                        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                        if (m == 0) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
                        __builtin_amdgcn_sched_group_barrier(0x002, 2, 0);
                    }
                    __builtin_amdgcn_sched_barrier(0);
                }
                if (t < 3)
#pragma unroll
                    for (int j = 0; j < JT; ++j) bc[j] = bn[j];
            }
        }
    };

    // ---- main loop: double-buffered X' stages, next step's codes in
    // registers; the scale/zero window after the current one is loaded at
    // the first step of each window (its buffer's previous window retired at
    // the barrier before) and is complete at the barrier after
    const int nwnd = (groups + 7) / 8;
    WStep<BITS> wa[JT], wb[JT];
    load_x(0, 0);
    load_w(0, wa);
    fetch_sz(0);
    store_sz(0);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    // step k: the window after the current one is fetched at the window's
    // first step and stored at its end (its buffer's previous window retired
    // at the barrier before the fetch; the barrier after the store publishes
    // it)
    {
    for (int kb = 0; kb < nk; kb += 2) {
        const bool f0 = kb % spw == 0 && kb / spw + 1 < nwnd;
        if (f0) fetch_sz(kb / spw + 1);
        if (kb + 1 < nk) { load_x(kb + 1, 1); load_w(kb + 1, wb); }
        compute(kb, 0, wa);
        if (f0) store_sz(kb / spw + 1);
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
        if (kb + 1 >= nk) break;
        const bool f1 = (kb + 1) % spw == 0 && (kb + 1) / spw + 1 < nwnd;
        if (f1) fetch_sz((kb + 1) / spw + 1);
        if (kb + 2 < nk) { load_x(kb + 2, 0); load_w(kb + 2, wa); }
        compute(kb + 1, 1, wb);
        if (f1) store_sz((kb + 1) / spw + 1);
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
    }

    }

    // ---- rank-r correction: MFMA steps of 32 over [T | B] (natural k order)
    for (int kr = 0; kr < a.r_pad; kr += 32) {
        const int k = kr + 8 * g;
        u32x4 bf[JT];
#pragma unroll
        for (int j = 0; j < JT; ++j) {
            const int n = n0 + 16 * j + r;
            uint32_t v[4] = {0, 0, 0, 0};
            if (n < a.N) {
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const uint16_t bv = k + e < a.rank ? a.B[static_cast<size_t>(n) * a.r_max + k + e] : 0;
                    v[e / 2] |= static_cast<uint32_t>(bv) << (16 * (e & 1));
                }
            }
            bf[j] = u32x4{v[0], v[1], v[2], v[3]};
        }
#pragma unroll
        for (int i = 0; i < MT; ++i) {
            const int m = m0 + 16 * i + r;
            const u32x4 af = *reinterpret_cast<const u32x4*>(a.T + static_cast<size_t>(m < a.M ? m : a.M - 1) * a.r_pad + k);
#pragma unroll
            for (int j = 0; j < JT; ++j) acc[i][j] = mfma(af, bf[j], acc[i][j]);
        }
    }

    // ---- store: acc[i][j][e] = Y[m0 + 16 i + 4 g + e][n0 + 16 j + r]
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int j = 0; j < JT; ++j) {
            const int n = n0 + 16 * j + r;
            if (n >= a.N) continue;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int m = m0 + 16 * i + 4 * g + e;
                if (m < a.M) store_out(a.Y, static_cast<size_t>(m) * a.N + n, acc[i][j][e], a.out);
            }
        }
}

size_t up256(size_t n) { return (n + 255) / 256 * 256; }

int prefill_cus() {
    static int cus[64] = {0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
    if (!cus[dev]) {
        int n = 0;
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
        cus[dev] = n;
    }
    return cus[dev];
}

// Row tiles per wave: 256-row workgroup tiles, or 128-row ones when 256-row
// tiles would not give every CU two workgroups (4096 x 4096 at M = 2048:
// 256 tiles; 117 against 133 us, while 14336 x 4096 stays faster with 256
// rows, 322 against 350 us)
int prefill_jt(int M, int N) {
    const long long tiles256 = static_cast<long long>((M + 127) / 128) * ((N + 255) / 256);
    return tiles256 < 2ll * prefill_cus() ? 2 : 4;
}

}  // namespace

// X' rows padded to whole 128-token blocks (prefill_kernel reads them)
size_t xp_rows(int M) { return (static_cast<size_t>(M) + 127) / 128 * 128; }

int xt_parts(int K) { return (K + XT_K - 1) / XT_K; }

size_t prefill_workspace_bytes(const QW& w, const LR& c, int M) {
    const int r_pad = (c.rank + 31) / 32 * 32;
    return up256(xp_rows(M) * w.d_in * 2) + up256(static_cast<size_t>(M) * r_pad * 2) +
           (c.rank > 0 ? up256(static_cast<size_t>(xt_parts(w.d_in)) * M * r_pad * 4) : 0);
}

hipError_t launch_linear_prefill(const QW& w, const LR& c, const void* X, int M, int act, void* Y, int out,
                                 void* ws, hipStream_t st) {
    uint16_t* Xp = static_cast<uint16_t*>(ws);
    uint16_t* T = reinterpret_cast<uint16_t*>(static_cast<char*>(ws) + up256(xp_rows(M) * w.d_in * 2));
    float* P = reinterpret_cast<float*>(reinterpret_cast<char*>(T) +
                                        up256(static_cast<size_t>(M) * ((c.rank + 31) / 32 * 32) * 2));
    PrefillArgs a;
    a.q = w.q; a.s = w.s; a.z = w.z; a.B = c.B;
    a.Xp = Xp;
    a.T = T;
    a.Y = Y;
    a.M = M; a.N = w.d_out; a.K = w.d_in; a.G = w.G;
    a.rank = c.rank; a.r_max = c.r_max; a.r_pad = (c.rank + 31) / 32 * 32;
    a.out = out;
    const int jt = prefill_jt(M, w.d_out);
    a.mblocks = (M + 127) / 128;
    const uint16_t* Xa = static_cast<const uint16_t*>(X);
    if (c.rank > 0) {
        const int mtiles = (M + XT_M - 1) / XT_M, parts = xt_parts(w.d_in);
        hipLaunchKernelGGL(xt_partial_kernel, dim3(static_cast<unsigned>(mtiles * parts)), dim3(256), 0, st, Xa, c.A,
                           Xp, P, M, w.d_in, c.rank, a.r_pad, act, mtiles);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        const long long n_all = static_cast<long long>(M) * a.r_pad;
        hipLaunchKernelGGL(t_reduce_kernel, dim3(static_cast<unsigned>((n_all / 4 + 255) / 256)), dim3(256), 0, st, P,
                           T, M, c.rank, a.r_pad, parts);
    } else {
        const long long chunks = static_cast<long long>(M) * w.d_in / 8;
        hipLaunchKernelGGL(xprep_kernel, dim3(static_cast<unsigned>((chunks + 255) / 256)), dim3(256), 0, st, Xa, Xp,
                           chunks, act);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const unsigned blocks = static_cast<unsigned>(a.mblocks * ((w.d_out + 64 * jt - 1) / (64 * jt)));
    const dim3 grid(blocks), block(256);
    // X' stages and scale/zero windows (see prefill_kernel)
    const size_t lds = (2 * 128 * 16 + 64 * jt * 4) * sizeof(u32x4);
    if (w.bits == 4 && jt == 4) hipLaunchKernelGGL((prefill_kernel<4, 4>), grid, block, lds, st, a);
    else if (w.bits == 4) hipLaunchKernelGGL((prefill_kernel<4, 2>), grid, block, lds, st, a);
    else if (w.bits == 3 && jt == 4) hipLaunchKernelGGL((prefill_kernel<3, 4>), grid, block, lds, st, a);
    else if (w.bits == 3) hipLaunchKernelGGL((prefill_kernel<3, 2>), grid, block, lds, st, a);
    else if (jt == 4) hipLaunchKernelGGL((prefill_kernel<2, 4>), grid, block, lds, st, a);
    else hipLaunchKernelGGL((prefill_kernel<2, 2>), grid, block, lds, st, a);
    return hipGetLastError();
}

}  // namespace cl
