// Decode path of the error-compensated quantized linear (few tokens):
//
//     y_i[t] = deq(Q_i) x[t] + B_i[:, :r_i] (A_i[:r_i] x[t])     (Section 4.1)
//
// for a compensation window of n <= 8 linears that read the same activations
// x (the paper fuses Q/K/V and gate/up into such windows, Section 4.2.2 and
// Appendix A.1); a single linear is the window n = 1.
//
// Two launches per call:
//  * prep: t_i = A_i[:r_i] x for every linear (one wave per row of A_i)
//    and the activations converted to fp16, permuted into the pair order
//    of the unpacked codes, with each 16-byte chunk's sum of activations --
//    all into the workspace;
//  * backbone: one grouped, persistent kernel over all row batches of all the
//    window's linears.
// A x stays in its own launch.  Handing it from producer to backbone
// workgroups of one launch was built and measured on MI355X: with
// release/acquire fences the per-XCD L2 writeback/invalidate cost 12-90 us;
// with fence-free device-coherent accesses (replicated, call-tagged
// entries) it still lost above ~8 MB of weights, because the producers'
// loads, their stores and the consumers' poll each wait in memory queues
// filled by the backbone's own streaming loads -- three round trips that
// take about as long as the stream.
//
// The backbone is HBM-bound (about half a byte per weight at 4 bits, a
// quarter at 2 bits):
//  * a "row group" of KS waves owns R consecutive rows of one linear; the
//    row's 16-byte chunks of packed codes are split into KS slices and lane l
//    of slice k handles chunks k*cps + l + 64j (j < CPL), so every load
//    instruction reads R fully coalesced segments;
//  * one token per pass: each wave holds one batch (codes, scales, zeros,
//    factor entries, A x) at a time and the chip holds many waves -- the
//    single-batch kernel needs 72 VGPRs against 120 with a second batch
//    prefetched, so 7 waves per SIMD stay resident instead of 4, and on
//    MI355X the gate matrix call went from 13.8 us to 11.9 us; several
//    tokens per pass at 4 bits keep the next batch's loads in flight during
//    the current batch's arithmetic, with raw loads only -- nothing consumes
//    a prefetched value before the compute that needs it; other shapes hold
//    one batch per wave (a second set would spill to scratch);
//  * codes are unpacked with one AND per pair straight into fp16 lanes (a
//    code in the mantissa bits of a zero-exponent fp16 is an exact subnormal)
//    and multiplied with the prepared activations by v_dot2 into fp32; each
//    chunk's scale and zero point are applied in fp32:
//        s * (sum q x - z * sum x);
//  * the rank-r term B[row, :r] . t rides in the same lane partial sums;
//  * sums over lanes use a transposing butterfly (R values in log steps),
//    K slices are combined through LDS in a fixed order: results are bitwise
//    reproducible.

#include <type_traits>

#include "cl_device.h"
#include "cl_internal.h"
#include "gemv_common.h"
#include "mfma_common.h"

namespace cl {

namespace {

constexpr int kMaxWin = 8;   // linears per window
constexpr int kMaxKp = 16;   // K parts of the many-token A x partials
constexpr int kPrefKp = 4;   // of them loaded ahead of the backbone's K loop
// Windows with this many tokens use the MFMA backbone (measured on the 4-bit
// Llama-8B layer: 2 tokens 72 us on the dot2 backbone against 88 us on MFMA,
// 3 tokens 123 against 88, 5-7 tokens ~185 against ~90)
constexpr int kMfmaMinTokens = 3;

// One linear of a window, as the backbone kernel sees it.
struct Lin {
    const uint32_t* q;
    const uint16_t* s;
    const uint16_t* z;
    const uint16_t* B;
    void* y;                 // [T][d_out]
    const float* t;          // [T][rank] (workspace); MFMA path: [kp][T][rpad] partials
    int d_out, rank, r_max;
    int batch_end;           // exclusive prefix sum of the linears' batches
    int rpad;                // MFMA path: rank rounded up to 32
};

struct DecodeArgs {
    Lin lin[kMaxWin];
    int n;
    const f16x2* xp;         // [T][d_in / 2] activations, fp16, pair-permuted
    const float* sx;         // [T][chunks] per-chunk sums of activations
    int d_in, G, T, tok0, out;
    int ks;                  // K slices (waves per row group)
    int cps;                 // chunks per slice
    int kp;                  // MFMA path: K parts of the A x partials
    const u32x4* xf;         // MFMA path: activations, word-major and token-minor (see PrepMArgs)
    void* h;                 // gated window: SiLU(y_0) * y_1 [T][d_out] (lin[].y unused)
};

// Preparation for the MFMA path: A x on MFMA as K-part partials.
struct PrepMArgs {
    const uint16_t* A[kMaxWin];
    float* tp[kMaxWin];      // [kp][T][rpad]
    int rank[kMaxWin];
    int rpad[kMaxWin];
    int tile_end[kMaxWin];   // exclusive prefix sum of (rpad / 16) * npass * kp
    int n;
    const uint16_t* x;       // [T][d_in] fp16/bf16 bits
    u32x4* xf;               // [pass][d_in / 8][16]: 8 activations of one token, unpack order
    int d_in, T, act;
    int kp;                  // K parts
    int spw;                 // 32-code steps per wave and K part
    int npass;               // passes of 16 tokens
};

struct PrepArgs {
    const uint16_t* A[kMaxWin];
    float* t[kMaxWin];
    int rank_end[kMaxWin];   // exclusive prefix sum of the ranks
    int n;
    const uint16_t* x;       // [T][d_in] fp16/bf16 bits
    f16x2* xp;
    float* sx;
    int d_in, T, act;
    int wpr;                 // waves per row of A (1, 2 or 4)
};

// Columns [k0, k1) of one row of A times the activations of tokens tok0 ..
// tok0 + NTOK - 1, by one wave: lane l takes the 8-element runs starting at
// k0 + 8 l + 512 m in increasing m (eight 16-byte loads of A in flight per
// lane), adds each run's v_dot2 chain to a float accumulator, and the wave
// sums its lanes with a butterfly.  Each token's result does not depend on
// NTOK.  k0 and k1 - k0 are multiples of 8.
template <int NTOK>
__device__ __forceinline__ void row_times_x(const uint16_t* ar, const uint16_t* x, int d_in, int k0, int k1, int tok0,
                                            int act, float (&out)[NTOK]) {
    constexpr int KB = 8;
    const int lane = threadIdx.x & 63;
    float acc[NTOK];
#pragma unroll
    for (int tk = 0; tk < NTOK; ++tk) acc[tk] = 0.f;
    for (int base = k0; base < k1; base += 64 * 8 * KB) {
        u32x4 av[KB];
        int col[KB];
#pragma unroll
        for (int k = 0; k < KB; ++k) {
            col[k] = base + (lane + 64 * k) * 8;
            av[k] = *reinterpret_cast<const u32x4*>(ar + (col[k] < k1 ? col[k] : k0));
        }
#pragma unroll
        for (int tk = 0; tk < NTOK; ++tk) {
            const uint16_t* xr = x + static_cast<size_t>(tok0 + tk) * d_in;
#pragma unroll
            for (int k = 0; k < KB; ++k) {
                uint32_t xw[4];
                load8_f16(xr + (col[k] < k1 ? col[k] : k0), act, xw);
                float d = 0.f;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    // copy the vector element to a scalar first: a bit_cast
                    // of a subscripted ext_vector reads element 0
                    const uint32_t ak = av[k][e], xk = xw[e];
                    d = dot2(__builtin_bit_cast(f16x2, ak), __builtin_bit_cast(f16x2, xk), d);
                }
                acc[tk] += col[k] < k1 ? d : 0.f;
            }
        }
    }
#pragma unroll
    for (int tk = 0; tk < NTOK; ++tk) out[tk] = wave_sum(acc[tk]);
}

// Preparation kernel.  Workgroups [0, rank_blocks) compute A x: each row i
// of some linear's A is split over wpr waves (wpr = 1, 2 or 4 by the row
// length, so a wave issues one round of loads: rows of 14336 took four
// dependent round trips on one wave), for every token in passes of 4, then 2,
// then 1 tokens; the wpr partial sums meet in LDS and are added in part
// order.  The remaining workgroups prepare the activations, one thread per
// (token, chunk).
template <int BITS>
__global__ __launch_bounds__(256) void decode_prep_kernel(PrepArgs a) {
    constexpr int CPC = BITS == 3 ? 32 : 128 / BITS;   // codes per chunk
    constexpr int PPC = CPC / 2;
    __shared__ float part[4][4];
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int tid = threadIdx.x;
    const int d_in = a.d_in, T = a.T;
    const int nrank = a.n > 0 ? a.rank_end[a.n - 1] : 0;
    const int wpr = a.wpr;
    const int rows_per_block = 4 / wpr;
    const int rank_blocks = (nrank + rows_per_block - 1) / rows_per_block;
    const int blk = blockIdx.x;
    if (blk < rank_blocks) {
        const int j = blk * rows_per_block + wave / wpr;
        const int pi = wave % wpr;                       // this wave's part of the row
        const bool valid = j < nrank;                    // every wave reaches the barriers
        const int jj = valid ? j : nrank - 1;
        int li = 0;
        while (jj >= a.rank_end[li]) ++li;
        const int i = jj - (li ? a.rank_end[li - 1] : 0);
        const int rank = a.rank_end[li] - (li ? a.rank_end[li - 1] : 0);
        const uint16_t* ar = a.A[li] + static_cast<size_t>(i) * d_in;
        float* t = a.t[li];
        const int kc = (d_in / 8 + wpr - 1) / wpr * 8;   // columns per part, a multiple of 8
        const int k0 = min(d_in, pi * kc), k1 = min(d_in, k0 + kc);
        auto pass = [&](auto ntok, int tb) {
            constexpr int N = decltype(ntok)::value;
            float v[N];
            row_times_x<N>(ar, a.x, d_in, k0, k1, tb, a.act, v);
            if (wpr == 1) {
#pragma unroll
                for (int tk = 0; tk < N; ++tk)
                    if (valid && lane == tk) t[static_cast<size_t>(tb + tk) * rank + i] = v[tk];
                return;
            }
#pragma unroll
            for (int tk = 0; tk < N; ++tk)
                if (lane == tk) part[wave][tk] = v[tk];
            __syncthreads();
            if (valid && pi == 0 && lane < N) {
                float sum = 0.f;
                for (int q = 0; q < wpr; ++q) sum += part[wave + q][lane];
                t[static_cast<size_t>(tb + lane) * rank + i] = sum;
            }
            __syncthreads();
        };
        int tb = 0;
        for (; tb + 4 <= T; tb += 4) pass(std::integral_constant<int, 4>{}, tb);
        if (tb + 2 <= T) { pass(std::integral_constant<int, 2>{}, tb); tb += 2; }
        if (tb < T) pass(std::integral_constant<int, 1>{}, tb);
        return;
    }
    const int chunks = d_in / CPC;
    const long long item = static_cast<long long>(blk - rank_blocks) * 256 + tid;
    if (item >= static_cast<long long>(T) * chunks) return;
    const int tok = static_cast<int>(item / chunks);
    const int c = static_cast<int>(item % chunks);
    f16x2 v[PPC];
    if constexpr (BITS == 3) load_chunk_x3(a.x + static_cast<size_t>(tok) * d_in, c, a.act, v);
    else load_chunk_x<BITS>(a.x + static_cast<size_t>(tok) * d_in, c, a.act, v);
    const f16x2 one = {static_cast<f16>(1.0f), static_cast<f16>(1.0f)};
    float sum = 0.f;
    f16x2* dst = a.xp + static_cast<size_t>(tok) * (d_in / 2) + static_cast<size_t>(c) * PPC;
#pragma unroll
    for (int p = 0; p < PPC; ++p) {
        sum = dot2(v[p], one, sum);
        dst[p] = v[p];
    }
    a.sx[static_cast<size_t>(tok) * chunks + c] = sum;
}

// One batch of a wave: R rows x CPL chunks of packed codes, the matching
// scales and zeros, the rows' factor entries and this lane's entries of A x.
// Raw loads only: nothing may consume a value at load time, or the wave would
// stall on the prefetch it is meant to overlap.
template <int R, int CPL, int NB, int NT, int QW = 4>
struct Batch {
    uint32_t q[R][CPL][QW];  // a chunk's code words: 4 (2/4-bit), 3 (3-bit)
    uint16_t s[R][CPL];      // fp16 scale bits
    uint16_t z[R][CPL];      // fp16 zero-point bits
    uint16_t b[R][NB];       // B[row][i] for this lane's factor columns
    float t[NT][NB];         // (A x)[tok][i] for the same columns
};

// NB: factor columns of B per lane (rank <= NB * 64 * ks); 0 when every
// linear of the window has rank 0.
// The one-token 4-bit kernel with at most one factor column per lane fits
// 72 VGPRs without spills: it is held to that (7 waves per SIMD); its gated
// instance needs one more and is held to 80 (6 waves per SIMD).
// GLU: a gated window of two linears with the same d_out (gate, up) launched
// with one workgroup per batch of the gate, so a workgroup's second batch is
// the up batch of the same rows: the lanes that hold a gate total keep it and
// write SiLU(gate) * up for the same row and token to a.h.
// MAXT: the largest block the instance is launched with.  Instances for
// several tokens per pass launched with 256 threads (one wave per SIMD per
// workgroup) are built for that size, so registers beyond 256 per lane come
// from the accumulation registers rather than from scratch memory.
template <int BITS, int NT, int CPL, int R, int NB, bool GLU, int MAXT = 512>
__global__ __launch_bounds__(MAXT)
__attribute__((amdgpu_waves_per_eu(BITS == 4 && NT == 1 && CPL == 1 && NB <= 1 ? (GLU ? 6 : 7) : 1)))
void decode_kernel(DecodeArgs a) {
    // a chunk is one lane's unit of codes: 16 bytes = 4 words of 32 / BITS
    // codes at 2 and 4 bits, 3 words = 32 codes at 3 bits
    constexpr int QW = BITS == 3 ? 3 : 4;        // words per chunk
    constexpr int CPC = BITS == 3 ? 32 : 128 / BITS;   // codes per chunk
    constexpr int HPW = BITS == 3 ? 0 : 16 / BITS;     // fp16 pairs per word (2/4-bit)
    constexpr int PPC = CPC / 2;      // pairs per chunk
    constexpr int NACC = BITS == 4 ? 2 : (BITS == 2 ? 4 : 8);
    constexpr int NBA = NB > 0 ? NB : 1;
    constexpr bool XREG = NT * CPL * PPC <= 32;   // activations stay in registers

    __shared__ float red[2][8][R][NT];
    // GLU: the gate totals a lane holds, kept in LDS between its two batches
    // (a register kept live across them spilled at 72 VGPRs)
    __shared__ float gl[GLU ? 512 : 1][NT];

    const int lane = threadIdx.x & 63;
    // wave-uniform values in scalar registers: row addressing stays scalar
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int waves = blockDim.x >> 6;
    const int words = a.d_in / CPC * QW;          // per row
    const int chunks = a.d_in / CPC;
    const int groups = a.d_in / a.G;
    const int ks = a.ks;
    const int rg_per_block = waves / ks;
    const int slice = wave % ks;
    const int rgw = wave / ks;
    const int nbatch = a.lin[a.n - 1].batch_end;
    const int c_begin = slice * a.cps;
    const int c_end = min(chunks, c_begin + a.cps);

    int cidx[CPL];
    float cmask[CPL];                      // 1 for a real chunk, 0 for a padding lane
#pragma unroll
    for (int j = 0; j < CPL; ++j) {
        cidx[j] = c_begin + lane + 64 * j;
        const bool valid = cidx[j] < c_end;
        cmask[j] = valid ? 1.f : 0.f;
        if (!valid) cidx[j] = c_begin;     // in-bounds dummy chunk, weighted by 0
    }

    // prepared activations of this lane's chunks and their sums
    f16x2 xv[XREG ? NT : 1][XREG ? CPL : 1][PPC];
    float sx[NT][CPL];
#pragma unroll
    for (int tk = 0; tk < NT; ++tk) {
        const int tok = min(a.tok0 + tk, a.T - 1);
#pragma unroll
        for (int j = 0; j < CPL; ++j) {
            sx[tk][j] = a.sx[static_cast<size_t>(tok) * chunks + cidx[j]];
            if (XREG) {
                const u32x4* src = reinterpret_cast<const u32x4*>(a.xp + static_cast<size_t>(tok) * (a.d_in / 2) +
                                                                  static_cast<size_t>(cidx[j]) * PPC);
#pragma unroll
                for (int p4 = 0; p4 < PPC / 4; ++p4) {
                    const u32x4 u = src[p4];
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const uint32_t ue = u[e];
                        xv[XREG ? tk : 0][XREG ? j : 0][4 * p4 + e] = __builtin_bit_cast(f16x2, ue);
                    }
                }
            }
        }
    }

    // global batch b -> (linear, first row of this wave's row group)
    auto locate = [&](int b, int& li, int& row0) {
        li = 0;
        while (b >= a.lin[li].batch_end) ++li;
        const int lb = b - (li ? a.lin[li - 1].batch_end : 0);
        row0 = (lb * rg_per_block + rgw) * R;
    };

    auto load_batch = [&](Batch<R, CPL, NBA, NT, QW>& bt, int b) {
        int li, row0;
        locate(b, li, row0);
        const Lin& L = a.lin[li];
        const int base = row0 < L.d_out ? row0 : 0;
        const int nrows = row0 < L.d_out ? min(R, L.d_out - row0) : 1;
        // a rank-0 linear has no factors: its loads read valid placeholder
        // memory (masked to zero in compute_batch) instead of branching on data
        const uint16_t* Bp = L.rank > 0 ? L.B : L.s;
        const int bstride = L.rank > 0 ? L.r_max : 0;
        const float* tp = L.rank > 0 ? L.t : a.sx;
        const int tstride = L.rank > 0 ? L.rank : 0;
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int row = base + (r < nrows ? r : 0);
            const uint32_t* qrow = L.q + static_cast<size_t>(row) * words;
#pragma unroll
            for (int j = 0; j < CPL; ++j) {
                if constexpr (QW == 4) {
                    const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(qrow) + cidx[j]);
#pragma unroll
                    for (int e = 0; e < 4; ++e) { const uint32_t ve = v[e]; bt.q[r][j][e] = ve; }
                } else {
#pragma unroll
                    for (int e = 0; e < QW; ++e) bt.q[r][j][e] = __builtin_nontemporal_load(qrow + QW * cidx[j] + e);
                }
            }
#pragma unroll
            for (int j = 0; j < CPL; ++j) {
                const size_t gi = static_cast<size_t>(row) * groups + (cidx[j] * CPC) / a.G;
                bt.s[r][j] = L.s[gi];
                bt.z[r][j] = L.z[gi];
            }
#pragma unroll
            for (int m = 0; m < NB; ++m) {
                // columns past the rank read column 0 (valid data) and meet t = 0
                const int i = lane + 64 * (slice + ks * m);
                bt.b[r][m] = Bp[static_cast<size_t>(row) * bstride + (i < L.rank ? i : 0)];
            }
        }
#pragma unroll
        for (int tk = 0; tk < NT; ++tk)
#pragma unroll
            for (int m = 0; m < NB; ++m) {
                const int i = lane + 64 * (slice + ks * m);
                const int tok = min(a.tok0 + tk, a.T - 1);
                bt.t[tk][m] = tp[static_cast<size_t>(tok) * tstride + (i < L.rank ? i : 0)];
            }
    };

    auto compute_batch = [&](const Batch<R, CPL, NBA, NT, QW>& bt, int b, int buf) {
        int li, row0;
        locate(b, li, row0);
        const Lin& L = a.lin[li];
        float acc[R][NT];
#pragma unroll
        for (int r = 0; r < R; ++r)
#pragma unroll
            for (int tk = 0; tk < NT; ++tk) acc[r][tk] = 0.f;
#pragma unroll
        for (int tk = 0; tk < NT; ++tk) {
#pragma unroll
            for (int j = 0; j < CPL; ++j) {
                f16x2 xl[XREG ? 1 : PPC];
                if (!XREG) {
                    const u32x4* src = reinterpret_cast<const u32x4*>(
                        a.xp + static_cast<size_t>(min(a.tok0 + tk, a.T - 1)) * (a.d_in / 2) + static_cast<size_t>(cidx[j]) * PPC);
#pragma unroll
                    for (int p4 = 0; p4 < PPC / 4; ++p4) {
                        const u32x4 u = src[p4];
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const uint32_t ue = u[e];
                            xl[4 * p4 + e] = __builtin_bit_cast(f16x2, ue);
                        }
                    }
                }
                const f16x2* xq = XREG ? xv[XREG ? tk : 0][XREG ? j : 0] : xl;
#pragma unroll
                for (int r = 0; r < R; ++r) {
                    float d[NACC];
#pragma unroll
                    for (int k = 0; k < NACC; ++k) d[k] = 0.f;
                    if constexpr (BITS == 3) {
                        dot_chunk3(bt.q[r][j][0], bt.q[r][j][1], bt.q[r][j][2], xq, d);
                    } else {
#pragma unroll
                        for (int w = 0; w < 4; ++w) dot_word<BITS>(bt.q[r][j][w], xq + w * HPW, d);
                    }
                    const float sc = f16_bits_to_f32(bt.s[r][j]) * cmask[j];
                    const float zc = f16_bits_to_f32(bt.z[r][j]);
                    // s * (2^24 * sum q x - z * sum x): the codes were subnormals q * 2^-24
                    const float v = fmaf(combine<BITS>(d), 16777216.0f, -zc * sx[tk][j]);
                    acc[r][tk] = fmaf(sc, v, acc[r][tk]);
                }
            }
        }
        // rank-r up-projection B[row, i] * t[i] over this lane's factor columns
        // (entries past the rank were loaded from column 0 and are masked here)
#pragma unroll
        for (int m = 0; m < NB; ++m) {
            const int i = lane + 64 * (slice + ks * m);
            const float on = i < L.rank ? 1.f : 0.f;
#pragma unroll
            for (int r = 0; r < R; ++r) {
                const float bv = f16_bits_to_f32(bt.b[r][m]) * on;
#pragma unroll
                for (int tk = 0; tk < NT; ++tk) acc[r][tk] = fmaf(bv, bt.t[tk][m], acc[r][tk]);
            }
        }
        // reduce over lanes, then over the K slices in a fixed order, store
#pragma unroll
        for (int tk = 0; tk < NT; ++tk) {
            float v[R];
#pragma unroll
            for (int r = 0; r < R; ++r) v[r] = acc[r][tk];
            const float tot = wave_sum_multi<R>(v);
            constexpr int SPAN = 64 / R;      // lanes that share one total
            const int rr = (lane / SPAN) & (R - 1);
            if ((lane & (SPAN - 1)) == 0) {
                if (ks == 1) {
                    if (row0 + rr < L.d_out && a.tok0 + tk < a.T) {
                        const size_t idx = static_cast<size_t>(a.tok0 + tk) * L.d_out + row0 + rr;
                        if constexpr (GLU) {
                            if (li == 0) gl[threadIdx.x][tk] = tot;
                            else store_out(a.h, idx, silu_mul(gl[threadIdx.x][tk], tot), a.out);
                        } else {
                            store_out(L.y, idx, tot, a.out);
                        }
                    }
                } else {
                    red[buf][wave][rr][tk] = tot;
                }
            }
        }
        if (ks == 1) return;
        __syncthreads();
        if (slice == 0 && lane < R * NT) {
            const int r = lane / NT, tk = lane - r * NT;
            const int row = row0 + r;
            if (row < L.d_out && a.tok0 + tk < a.T) {
                float v = 0.f;
                for (int k = 0; k < ks; ++k) v += red[buf][wave + k][r][tk];
                const size_t idx = static_cast<size_t>(a.tok0 + tk) * L.d_out + row;
                if constexpr (GLU) {
                    if (li == 0) gl[threadIdx.x][0] = v;
                    else store_out(a.h, idx, silu_mul(gl[threadIdx.x][0], v), a.out);
                } else {
                    store_out(L.y, idx, v, a.out);
                }
            }
        }
    };

    const int stride = gridDim.x;
    int b = blockIdx.x;
    if (b >= nbatch) return;
    // A second register set for the next batch pays where it costs no
    // spills: two tokens per pass at 4 bits and one chunk per lane (measured
    // on MI355X: the T = 2 layer 72 us with it, 73 us without).  Everywhere
    // else a wave holds one batch at a time (alternating LDS buffers).
    constexpr bool kPrefetch = BITS == 4 && CPL == 1 && NT == 2;
    if constexpr (!kPrefetch) {
        for (int it = 0; b < nbatch; b += stride, ++it) {
            Batch<R, CPL, NBA, NT, QW> bt;
            load_batch(bt, b);
            compute_batch(bt, b, it & 1);
        }
        return;
    }
    // Persistent loop over batches with the next batch's loads in flight
    // during the current batch's arithmetic (two register sets, alternating
    // LDS buffers).  Every compute site has a single predecessor shape (next
    // batch issued, or this is the last batch) so the compiler's wait counts
    // let the prefetch stay in flight.
    Batch<R, CPL, NBA, NT, QW> b0, b1;
    load_batch(b0, b);
    for (;;) {
        if (b + stride >= nbatch) { compute_batch(b0, b, 0); break; }
        load_batch(b1, b + stride);
        compute_batch(b0, b, 0);
        b += stride;
        if (b + stride >= nbatch) { compute_batch(b1, b, 1); break; }
        load_batch(b0, b + stride);
        compute_batch(b1, b, 1);
        b += stride;
    }
}

// Preparation for the MFMA backbone.  Workgroups [0, tiles): (linear, 16 rows
// of A, pass of 16 tokens, K part kp): t partial[kp][tok][i] = sum over the
// part's k of A[i][k] x[tok][k] for the pass's tokens on
// v_mfma_f32_16x16x32_f16 (A rows as the A operand, tokens as the B
// operand; the workgroup's 4, 8 or 16 waves split the part, up to eight
// 32-code steps of loads in flight per wave; the waves' tiles are summed
// through LDS in a fixed order).  Rows past the rank are written as zero.
// The remaining workgroups write the activations in the backbone's operand
// layout: for each pass of 16 tokens and each 8-code word of K, the 16
// tokens' 8 activations (16 bytes each, unpack order) side by side, so one
// load instruction reads 256 contiguous bytes per lane group.
__global__ __launch_bounds__(1024) void decode_prep_mfma_kernel(PrepMArgs a) {
    constexpr int CPW = 8, HPW = 4, PPC = 16;        // 8-code units, the backbone's unpack order
    __shared__ f32x4 red[16][64];
    const int nw = blockDim.x >> 6;                  // waves per K part: 4, 8 or 16
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int g = lane >> 4, r = lane & 15;
    const int tid = threadIdx.x;
    const int d_in = a.d_in, T = a.T;
    const int ntile = a.n > 0 ? a.tile_end[a.n - 1] : 0;
    const int blk = blockIdx.x;
    if (blk < ntile) {
        int li = 0;
        while (blk >= a.tile_end[li]) ++li;
        const int local = blk - (li ? a.tile_end[li - 1] : 0);
        const int tp_ = local / a.kp, kp = local - tp_ * a.kp;
        const int tile = tp_ / a.npass, pass = tp_ - tile * a.npass;
        const int rank = a.rank[li];
        const int arow = tile * 16 + r;
        const bool av = arow < rank;
        const uint16_t* ar = a.A[li] + static_cast<size_t>(av ? arow : 0) * d_in;
        const int tokr = pass * 16 + r;
        const bool tv = tokr < T;
        const uint16_t* xr = a.x + static_cast<size_t>(tv ? tokr : 0) * d_in;
        const int nsteps = d_in / 32;
        const int s0 = (kp * nw + wave) * a.spw;
        const int s1 = min(s0 + a.spw, nsteps);
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
        for (int sb = s0; sb < s1; sb += 8) {
            u32x4 am[8], xm[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int k = (sb + u < s1 ? sb + u : s0) * 32 + 8 * g;
                am[u] = *reinterpret_cast<const u32x4*>(ar + k);
                xm[u] = *reinterpret_cast<const u32x4*>(xr + k);
            }
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const bool live = sb + u < s1;
                const u32x4 zero = {0, 0, 0, 0};
                const u32x4 a8 = (av && live) ? am[u] : zero;
                const u32x4 x8 = (tv && live) ? act8_to_f16(xm[u], a.act) : zero;
                acc = mfma(a8, x8, acc);
            }
        }
        red[wave][lane] = acc;
        __syncthreads();
        if (wave != 0 || !tv) return;
        acc = red[0][lane];
        for (int w = 1; w < nw; ++w) acc += red[w][lane];
        // acc[e] = partial t[tok tokr][row tile*16 + 4 g + e]
        float* dst = a.tp[li] + (static_cast<size_t>(kp) * T + tokr) * a.rpad[li] + tile * 16 + 4 * g;
#pragma unroll
        for (int e = 0; e < 4; ++e) dst[e] = tile * 16 + 4 * g + e < rank ? acc[e] : 0.f;
        return;
    }
    // activations: item (pass, word wi, token lane r) -> 16 bytes, the 8
    // activations of codes 8 wi .. 8 wi + 7 of token 16 pass + r in the
    // unpack's pair order (x0, x4), (x1, x5), (x2, x6), (x3, x7); a pass of
    // tp <= 16 tokens stores its words tp entries apart (word wi of token r at
    // wi tp + r), so fewer tokens are fewer bytes for the backbone to read
    const int wpr = d_in / CPW;
    const int npass = (T + 15) / 16;
    const long long item = static_cast<long long>(blk - ntile) * blockDim.x + tid;
    if (item >= static_cast<long long>(npass) * wpr * 16) return;
    const int rt = static_cast<int>(item & 15);
    const int wi = static_cast<int>((item >> 4) % wpr);
    const int pass = static_cast<int>(item / (16ll * wpr));
    const int tp = min(16, T - 16 * pass);
    if (rt >= tp) return;
    const int tok = pass * 16 + rt;
    u32x4 o = {0u, 0u, 0u, 0u};
    {
        const u32x4 u = act8_to_f16(*reinterpret_cast<const u32x4*>(a.x + static_cast<size_t>(tok) * d_in + 8 * wi),
                                 a.act);
        // u[i] holds (x[2i], x[2i + 1]); pair p needs (x[p], x[p + 4])
#pragma unroll
        for (int pp = 0; pp < HPW; ++pp) {
            const uint32_t lo = u[pp / 2], hi = u[(pp + HPW) / 2];
            const uint32_t av = (pp & 1) ? (lo >> 16) : (lo & 0xffff);
            const uint32_t bv = (pp & 1) ? (hi & 0xffff0000u) : (hi << 16);
            o[pp] = av | bv;
        }
    }
    a.xf[static_cast<size_t>(pass) * wpr * 16 + static_cast<size_t>(wi) * tp + rt] = o;
    (void)PPC;
}

// Many-token backbone (4-, 3- or 2-bit codes, T >= 3): the contraction has
// enough columns to use MFMA (tokens padded to 16).  One workgroup per TPW
// 16-row tiles of one linear; its four waves split the 128-code blocks of K
// (wave w takes blocks w, w + 4, ...), NBUF blocks per wave in flight.  Per
// block a lane loads, for each of its TPW tiles, its 32 codes of row
// r = lane % 16 (16 bytes at 4 bits, 12 at 3, 8 at 2), and once for all
// tiles the matching activations of token r (four 16-byte loads from the
// word-major layout, 256 or 1024 contiguous bytes per load instruction).
// The MFMA takes the activations as its A operand and the codes as its B
// operand, so lane (g, r) accumulates tokens 4 g .. 4 g + 3 of weight row r.
// The codes of each 8-code unit become the exact fp16 integers q - z (4-bit:
// the unit is a word, codes_minus_zero; 2- and 3-bit: the unit is first
// spread by a byte permute, then one mask and one packed add or FMA per
// pair, codes2_minus_zero, codes3_minus_zero), and every quantization
// group's MFMA steps run into a fresh fp32 partial that is scaled by the
// group's fp16 scale in fp32 and added to the accumulator: the backbone is
// s (sum (q - z) x) with fp32 rounding only, whatever the scale (a weight
// tile rounded to fp16 would carry 2^-11 relative error, and lose precision
// once s / 16 falls below the fp16 normal range).  GPB (groups per 128-code
// block) = 128 / G: with one group per block each MFMA step takes unit t of
// every lane group (the four steps cover the block); with 2 or 4 groups the
// units are transposed across the lane groups first, so step t covers the
// 32 codes 32 t .. 32 t + 31, which lie in one group.  The rank-r term is
// extra MFMA steps over [t | B] spread over the waves (t from the K-part
// partials of decode_prep_mfma_kernel, summed in a fixed order and split
// into fp16 hi and lo parts, one step each); the waves' tiles are summed
// through LDS in a fixed order; one rounding to the output dtype.
template <int BITS, int TPW, int NBUF, bool GLU, int GPB, int NW, bool LONGK>
__global__ __launch_bounds__((GLU ? 2 : 1) * 64 * NW) void decode_mfma_kernel(DecodeArgs a) {
    static_assert(BITS == 4 || BITS == 3 || BITS == 2, "4-, 3- or 2-bit codes");
    // NW waves split K.  GLU: 2 NW waves, the first NW on the gate's tiles
    // and the other NW on the up tiles of the same rows (phase 1); the two
    // sets of sums meet in LDS and the first NW waves store SiLU(gate) * up
    constexpr int NPH = GLU ? 2 : 1;
    constexpr int TPH = 64 * NW;                  // threads per phase
    static_assert(TPW <= NW, "one stored tile per wave");
    __shared__ f32x4 red[NW * NPH][TPW][64];
    extern __shared__ uint16_t szl_all[];         // per phase [2][16 TPW][RS]: the rows' scales, then zeros
    const int lane = threadIdx.x & 63;
    const int wave_all = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int ph = GLU ? wave_all / NW : 0;
    const int wave = wave_all % NW;               // wave within the phase
    const int tid = threadIdx.x % TPH;            // thread within the phase
    const int g = lane >> 4, r = lane & 15;
    // workgroup -> (linear, TPW tiles of 16 rows); batch_end counts workgroups
    int li0 = 0;
    while (static_cast<int>(blockIdx.x) >= a.lin[li0].batch_end) ++li0;
    const int row0 = (blockIdx.x - (li0 ? a.lin[li0 - 1].batch_end : 0)) * 16 * TPW;
    const Lin& L = a.lin[GLU ? ph : li0];
    int row[TPW];
    bool rowv[TPW];
#pragma unroll
    for (int j = 0; j < TPW; ++j) {
        rowv[j] = row0 + 16 * j + r < L.d_out;
        row[j] = rowv[j] ? row0 + 16 * j + r : L.d_out - 1;
    }
    const int tok = a.tok0 + r;                    // this lane's token column of the B operand
    const bool tokv = tok < a.T;
    const int K = a.d_in;
    const int nkb = (K + 127) / 128;
    const int words_row = K / 8;                  // 8-code units of a row (activation words)
    const int qwords_row = K * BITS / 32;         // 32-bit code words of a row
    const int groups = K / a.G;
    const int RS = szl_stride(groups);            // padded row stride of the tables
    uint16_t* const szl = szl_all + ph * (2 * 16 * TPW * RS);
    const uint32_t mlo = __builtin_amdgcn_readfirstlane(0x000F000Fu);
    const uint32_t mhi = __builtin_amdgcn_readfirstlane(0x00F000F0u);
    uint32_t m2[4], m3[3];
#pragma unroll
    for (int p = 0; p < 4; ++p) m2[p] = __builtin_amdgcn_readfirstlane(0x00030003u << (2 * p));
#pragma unroll
    for (int p = 0; p < 3; ++p) m3[p] = __builtin_amdgcn_readfirstlane(0x00070007u << (3 * p));
    const uint32_t bias = 0x64006400u;
    // this pass's activations, tp tokens per word: lane row r reads token
    // min(r, tp - 1) (rows past the pass's tokens repeat the last one; their
    // output rows are never stored)
    const int tp = min(16, a.T - a.tok0);
    const u32x4* xf = a.xf + static_cast<size_t>(a.tok0 / 16) * words_row * 16 + (r < tp ? r : tp - 1);
    // the workgroup's scales and zeros go to LDS (rows are consecutive, so
    // each array's part is one contiguous run; rows past the matrix are not
    // loaded and never used).  Vector loads complete in issue order, so the
    // first 16-byte piece of each array is loaded here, before the K loop's
    // first code blocks, and stored to LDS after those are issued: the copy
    // waits for the scales and zeros only.
    const int nval = min(16 * TPW, L.d_out - row0) * groups;
    const uint16_t* ssrc = L.s + static_cast<size_t>(row0) * groups;
    const uint16_t* zsrc = L.z + static_cast<size_t>(row0) * groups;
    // 16-byte pieces only where both runs start 16-byte aligned (the caller's
    // arrays need only 2-byte alignment)
    const bool al = ((reinterpret_cast<uintptr_t>(ssrc) | reinterpret_cast<uintptr_t>(zsrc)) & 15) == 0;
    const int n16 = al ? nval / 8 : 0;
    uint16_t* const zl = szl + 16 * TPW * RS;
    // table entry of the run's value i (row i / groups, column i % groups;
    // the identity on an unpadded table, where pieces may span rows)
    auto tix = [&](int i) { return RS == groups ? i : i / groups * RS + i % groups; };
    const u32x4* s16p = n16 ? reinterpret_cast<const u32x4*>(ssrc) + min(tid, n16 - 1)
                            : reinterpret_cast<const u32x4*>(a.xf);
    const u32x4* z16p = n16 ? reinterpret_cast<const u32x4*>(zsrc) + min(tid, n16 - 1)
                            : reinterpret_cast<const u32x4*>(a.xf);
    const u32x4 s_first = *s16p, z_first = *z16p;

    // the lane's 32 codes of each tile row: 4 words (4-bit), 3 (3-bit) or 2
    // (2-bit)
    struct U3 {
        uint32_t e[3];
        __device__ uint32_t operator[](int i) const { return e[i]; }
    };
    using CodeW = std::conditional_t<BITS == 4, u32x4, std::conditional_t<BITS == 3, U3, u32x2>>;
    struct Blk {
        CodeW w[TPW];
        u32x4 x[4];
    };
    // rank-r term, 32 factor columns per step, wave w taking steps w, w + 4:
    // A operand t[tok][k .. k + 8) = the sum of the K-part partials in order
    // (as fp16 hi and lo parts, one MFMA step each), B operand
    // B[row][k .. k + 8).  The first step's operands are loaded before the K
    // loop, so their latency is hidden.
    const bool bvec = (L.r_max & 7) == 0 && (reinterpret_cast<uintptr_t>(L.B) & 15) == 0;
    f32x4 acc[TPW];
#pragma unroll
    for (int j = 0; j < TPW; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
    struct RankOp {
        uint32_t bw[TPW][4];
        f32x4 tp[kPrefKp][2];
    };
    auto rank_load = [&](int kr, RankOp& o) {
        const int k = kr + 8 * g;
        if (kr >= L.rank) return;
#pragma unroll
        for (int j = 0; j < TPW; ++j) {
            const uint16_t* brow = L.B + static_cast<size_t>(row[j]) * L.r_max;
            if (bvec && k + 8 <= L.r_max) {
                const u32x4 v = *reinterpret_cast<const u32x4*>(brow + k);
#pragma unroll
                for (int e = 0; e < 4; ++e) { const uint32_t ve = v[e]; o.bw[j][e] = ve; }
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const uint32_t lo = k + 2 * e < L.r_max ? brow[k + 2 * e] : 0u;
                    const uint32_t hi = k + 2 * e + 1 < L.r_max ? brow[k + 2 * e + 1] : 0u;
                    o.bw[j][e] = lo | (hi << 16);
                }
            }
        }
        const int tk = tokv ? tok : 0;
#pragma unroll
        for (int p = 0; p < kPrefKp; ++p) {
            const int pp = p < a.kp ? p : 0;
            const f32x4* src = reinterpret_cast<const f32x4*>(L.t + (static_cast<size_t>(pp) * a.T + tk) * L.rpad + k);
            o.tp[p][0] = src[0];
            o.tp[p][1] = src[1];
        }
    };
    auto rank_mma = [&](int kr, const RankOp& o) {
        if (kr >= L.rank) return;
        const int k = kr + 8 * g;
        float tsum[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int p = 0; p < kPrefKp; ++p) {
            if (p < a.kp) {
#pragma unroll
                for (int e = 0; e < 4; ++e) { tsum[e] += o.tp[p][0][e]; tsum[4 + e] += o.tp[p][1][e]; }
            }
        }
        // long rows (more than kPrefKp K parts): the other partials now, in
        // the same order (holding them through the K loop cost a wave per
        // SIMD; fewer parts had made each preparation workgroup read ~230 KB
        // of scattered 64-byte runs: the 14336-wide down took 9.9 us to prepare
        // at 16 tokens, 5.1 with 14 parts)
        if (LONGK && a.kp > kPrefKp) {
            f32x4 more[kMaxKp - kPrefKp][2];
            const int tk = tokv ? tok : 0;
#pragma unroll
            for (int p = kPrefKp; p < kMaxKp; ++p) {
                const int pp = p < a.kp ? p : 0;
                const f32x4* src =
                    reinterpret_cast<const f32x4*>(L.t + (static_cast<size_t>(pp) * a.T + tk) * L.rpad + k);
                more[p - kPrefKp][0] = src[0];
                more[p - kPrefKp][1] = src[1];
            }
#pragma unroll
            for (int p = kPrefKp; p < kMaxKp; ++p) {
                if (p < a.kp) {
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        tsum[e] += more[p - kPrefKp][0][e];
                        tsum[4 + e] += more[p - kPrefKp][1][e];
                    }
                }
            }
        }
        // t as fp16 hi + lo parts, two MFMA steps (absent tokens zero)
        uint32_t tw[4], tl[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            split_f16x2(tsum[2 * e], tsum[2 * e + 1], tw[e], tl[e]);
            if (!tokv) tw[e] = tl[e] = 0u;
        }
#pragma unroll
        for (int j = 0; j < TPW; ++j) {
            uint32_t aw[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                // entries past the rank (or past the matrix) and absent tokens are zero
                const uint32_t lo = (rowv[j] && k + 2 * e < L.rank) ? (o.bw[j][e] & 0xffffu) : 0u;
                const uint32_t hi = (rowv[j] && k + 2 * e + 1 < L.rank) ? (o.bw[j][e] >> 16) : 0u;
                aw[e] = lo | (hi << 16);
            }
            const u32x4 bop = {aw[0], aw[1], aw[2], aw[3]};
            acc[j] = mfma(u32x4{tw[0], tw[1], tw[2], tw[3]}, bop, acc[j]);
            acc[j] = mfma(u32x4{tl[0], tl[1], tl[2], tl[3]}, bop, acc[j]);
        }
    };
    RankOp rb;
    rank_load(32 * wave, rb);

    // loads are unconditional (valid addresses always) and nothing consumes a
    // loaded value before compute: the compiler's wait counts then let every
    // prefetched block stay in flight
    auto load = [&](int kb, Blk& b) {
        const int kc = kb * 128 + 32 * g;          // first of this lane's 32 codes
        const int wi = kc < K ? kc / 8 : 0;        // its first 8-code unit
#pragma unroll
        for (int j = 0; j < TPW; ++j) {
            if constexpr (BITS == 4) {
                b.w[j] = __builtin_nontemporal_load(
                    reinterpret_cast<const u32x4*>(L.q + static_cast<size_t>(row[j]) * words_row + wi));
            } else if constexpr (BITS == 3) {
                // chunk wi / 4 of the row: words 3 (wi / 4) .. + 2
                const uint32_t* src = L.q + static_cast<size_t>(row[j]) * qwords_row + 3 * (wi / 4);
#pragma unroll
                for (int e = 0; e < 3; ++e) b.w[j].e[e] = __builtin_nontemporal_load(src + e);
            } else {
                b.w[j] = __builtin_nontemporal_load(
                    reinterpret_cast<const u32x2*>(L.q + static_cast<size_t>(row[j]) * qwords_row + wi / 2));
            }
        }
        // the activations of the words this lane feeds to MFMA step t: word
        // 4 g + t of the block, or 4 t + g once the codes are transposed
        // (a word past K reads word g, met by a zero scale)
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            const int xw = GPB == 1 ? wi + t : (kb * 128 + 32 * t < K ? kb * 16 + 4 * t + g : g);
            b.x[t] = xf[static_cast<size_t>(xw) * tp];
        }
    };
    auto compute = [&](int kb, const Blk& b) {
        // per group: MFMA steps into a fresh partial of sum (q - z) x, then
        // acc += s * partial in fp32; past K, past the matrix or a padding
        // block the scale is 0 (the partial is finite)
        constexpr int SPG = 4 / GPB;               // MFMA steps per group
#pragma unroll
        for (int j = 0; j < TPW; ++j) {
            // w[t]: the lane's 8-code unit t (2-bit: spread for the masks)
            uint32_t w[4];
            if constexpr (BITS == 4) {
#pragma unroll
                for (int t = 0; t < 4; ++t) { const uint32_t v = b.w[j][t]; w[t] = v; }
            } else if constexpr (BITS == 3) {
#pragma unroll
                for (int t = 0; t < 4; ++t) w[t] = spread_unit3(b.w[j][0], b.w[j][1], b.w[j][2], t);
            } else {
#pragma unroll
                for (int t = 0; t < 4; ++t) w[t] = spread_half2(b.w[j][t >> 1], t & 1);
            }
            if constexpr (GPB > 1) transpose_words(w);
#pragma unroll
            for (int q = 0; q < GPB; ++q) {
                const int kc = kb * 128 + 32 * SPG * q;   // first code of the group's steps
                const bool on = kb < nkb && kc < K && rowv[j];
                const int lr = (16 * j + r) * RS + (on ? kc / a.G : 0);
                const uint32_t sb = szl[lr], zb = szl[16 * TPW * RS + lr];
                f32x4 p;
                if constexpr (BITS == 4) {
                    const Zq zq = make_zq(zb);
                    p = mfma(b.x[SPG * q], codes_minus_zero(w[SPG * q], zq, mlo, mhi, bias),
                             f32x4{0.f, 0.f, 0.f, 0.f});
#pragma unroll
                    for (int t = SPG * q + 1; t < SPG * q + SPG; ++t)
                        p = mfma(b.x[t], codes_minus_zero(w[t], zq, mlo, mhi, bias), p);
                } else if constexpr (BITS == 3) {
                    const Zq3 zq = make_zq3(zb);
                    p = mfma(b.x[SPG * q], codes3_minus_zero(w[SPG * q], zq, m3, bias), f32x4{0.f, 0.f, 0.f, 0.f});
#pragma unroll
                    for (int t = SPG * q + 1; t < SPG * q + SPG; ++t)
                        p = mfma(b.x[t], codes3_minus_zero(w[t], zq, m3, bias), p);
                } else {
                    const Zq2 zq = make_zq2(zb);
                    p = mfma(b.x[SPG * q], codes2_minus_zero(w[SPG * q], zq, m2, bias), f32x4{0.f, 0.f, 0.f, 0.f});
#pragma unroll
                    for (int t = SPG * q + 1; t < SPG * q + SPG; ++t)
                        p = mfma(b.x[t], codes2_minus_zero(w[t], zq, m2, bias), p);
                }
                acc[j] = fma4(on ? f16_bits_to_f32(static_cast<uint16_t>(sb)) : 0.f, p, acc[j]);
            }
        }
    };
    // blocks of this wave: kb = wave + NW i, NBUF in flight.  Rounds of NBUF:
    // block j of a round is computed, then its registers take block
    // j + NBUF (past the last block they reload the current one, already
    // cached).
    constexpr int SPAN = NW * NBUF;                // blocks per round over the NW waves
    const int rounds = (nkb + SPAN - 1) / SPAN;
    Blk b[NBUF];
#pragma unroll
    for (int j = 0; j < NBUF; ++j) load(wave + NW * j < nkb ? wave + NW * j : 0, b[j]);
    // the scales and zeros into LDS (the code loads stay in flight)
    if (tid < n16) {
        *reinterpret_cast<u32x4*>(szl + tix(8 * tid)) = s_first;
        *reinterpret_cast<u32x4*>(zl + tix(8 * tid)) = z_first;
    }
    for (int i = tid + TPH; i < n16; i += TPH) {           // more pieces than threads
        *reinterpret_cast<u32x4*>(szl + tix(8 * i)) = reinterpret_cast<const u32x4*>(ssrc)[i];
        *reinterpret_cast<u32x4*>(zl + tix(8 * i)) = reinterpret_cast<const u32x4*>(zsrc)[i];
    }
    for (int i = 8 * n16 + tid; i < nval; i += TPH) {      // misaligned runs, the last few values
        szl[tix(i)] = ssrc[i];
        zl[tix(i)] = zsrc[i];
    }
    __syncthreads();
    for (int rd = 0; rd < rounds; ++rd) {
#pragma unroll
        for (int j = 0; j < NBUF; ++j) {
            const int kb = wave + SPAN * rd + NW * j;
            compute(kb, b[j]);
            const int kn = kb + SPAN;
            load(kn < nkb ? kn : (kb < nkb ? kb : 0), b[j]);
        }
    }
    // rank-r term (operands loaded before the K loop, see rank_load)
    rank_mma(32 * wave, rb);
    for (int kr = 32 * wave + 32 * NW; kr < L.rank; kr += 32 * NW) {
        RankOp ro;
        rank_load(kr, ro);
        rank_mma(kr, ro);
    }
#pragma unroll
    for (int j = 0; j < TPW; ++j) red[NW * ph + wave][j][lane] = acc[j];
    __syncthreads();
    // wave w sums and stores tiles w, w + NW, ... in a fixed order
    if (ph == 0) {
#pragma unroll
        for (int j = 0; j < TPW; ++j) {
            if (j % NW != wave || !rowv[j]) continue;
            f32x4 v = red[0][j][lane];
#pragma unroll
            for (int w2 = 1; w2 < NW; ++w2) v += red[w2][j][lane];
            f32x4 u = {0.f, 0.f, 0.f, 0.f};
            if constexpr (GLU) {
                u = red[NW][j][lane];
#pragma unroll
                for (int w2 = 1; w2 < NW; ++w2) u += red[NW + w2][j][lane];
            }
            // v[e] = y[tok0 + 4 g + e][row0 + 16 j + r] (GLU: the gate's; u the up's)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int tk = a.tok0 + 4 * g + e;
                if (tk >= a.T) continue;
                const size_t idx = static_cast<size_t>(tk) * L.d_out + row[j];
                if (GLU) store_out(a.h, idx, silu_mul(v[e], u[e]), a.out);
                else store_out(L.y, idx, v[e], a.out);
            }
        }
    }
}

struct Plan {
    int cpl, R, ks, cps, nt, nb, threads;
};

// codes per lane chunk: 16 bytes at 2 and 4 bits, 3 words at 3 bits
int codes_per_chunk(int bits) { return bits == 3 ? 32 : 128 / bits; }

Plan plan(int d_in, int bits, int max_rank, int T) {
    const int chunks = d_in / codes_per_chunk(bits);
    Plan p;
    p.nt = T >= 4 ? 4 : (T >= 2 ? 2 : 1);
    // One 16-byte chunk per lane and 4 rows per batch measured best on
    // MI355X for every shape of the Llama-8B layer (more waves beat deeper
    // per-wave prefetch); rows wider than 8 slices of 64 chunks use 2.
    p.cpl = 1;
    auto slices = [&](int cpl) {
        int ks = (chunks + 64 * cpl - 1) / (64 * cpl);
        while (ks & (ks - 1)) ++ks;               // 1, 2, 4 or 8
        return ks;
    };
    if (slices(p.cpl) > 8) p.cpl = 2;
    p.ks = slices(p.cpl);
    p.R = 4;
    p.cps = (chunks + p.ks - 1) / p.ks;
    p.threads = 64 * (p.ks > 4 ? p.ks : 4);
    const int per = 64 * p.ks;                     // factor columns per lane pass
    p.nb = max_rank == 0 ? 0 : (max_rank <= per ? 1 : (max_rank <= 2 * per ? 2 : 4));
    return p;
}

int device_cus() {
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

template <int BITS, int NT, int CPL, int R, int NB>
hipError_t launch5(const DecodeArgs& a, const Plan& p, hipStream_t st) {
    // the 256-thread build of the multi-token one-chunk instances (the rest
    // are built for 512 threads only)
    constexpr bool kSmall = NT > 1 && CPL == 1;
    const bool small = kSmall && p.threads <= 256;
    if (a.h) {
        // gated window: workgroup i takes gate batch i, then up batch i
        auto gk = small ? decode_kernel<BITS, NT, CPL, R, NB, true, kSmall ? 256 : 512>
                        : decode_kernel<BITS, NT, CPL, R, NB, true>;
        hipLaunchKernelGGL(gk, dim3(a.lin[0].batch_end), dim3(p.threads), 0, st, a);
        return hipGetLastError();
    }
    auto kern = small ? decode_kernel<BITS, NT, CPL, R, NB, false, kSmall ? 256 : 512>
                      : decode_kernel<BITS, NT, CPL, R, NB, false>;
    // resident workgroups per CU for this instance and block size (cached
    // once per process)
    static int occ[2] = {0, 0};
    int& o = occ[p.threads > 256 ? 1 : 0];
    if (!o) {
        int n = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kern, p.threads, 0) != hipSuccess || n <= 0) n = 1;
        o = n;
    }
    const int nbatch = a.lin[a.n - 1].batch_end;
    // at most one resident wave of workgroups, each with the same number of
    // batches (no partial second wave)
    const int cap = o * device_cus();
    const int per = (nbatch + cap - 1) / cap;
    const int blocks = (nbatch + per - 1) / per;
    hipLaunchKernelGGL(kern, dim3(blocks), dim3(p.threads), 0, st, a);
    return hipGetLastError();
}

template <int BITS, int NT, int CPL>
hipError_t launch4(const DecodeArgs& a, const Plan& p, hipStream_t st) {
    switch (p.nb) {
        case 0: return launch5<BITS, NT, CPL, 4, 0>(a, p, st);
        case 1: return launch5<BITS, NT, CPL, 4, 1>(a, p, st);
        case 2: return launch5<BITS, NT, CPL, 4, 2>(a, p, st);
        default: return launch5<BITS, NT, CPL, 4, 4>(a, p, st);
    }
}

template <int BITS, int NT>
hipError_t launch3(const DecodeArgs& a, const Plan& p, hipStream_t st) {
    return p.cpl == 2 ? launch4<BITS, NT, 2>(a, p, st) : launch4<BITS, NT, 1>(a, p, st);
}

template <int BITS>
hipError_t launch2(const DecodeArgs& a, const Plan& p, hipStream_t st) {
    if (p.nt == 1) return launch3<BITS, 1>(a, p, st);
    if (p.nt == 2) return launch3<BITS, 2>(a, p, st);
    return launch3<BITS, 4>(a, p, st);
}

// Waves per row of A in the preparation: one round of eight 16-byte loads
// per lane covers 4096 columns.
int prep_waves_per_row(int d_in) { return d_in <= 4096 ? 1 : (d_in <= 8192 ? 2 : 4); }

// Workspace: per linear t_i [T][rank_i] float | xp [T][d_in/2] fp16 pairs |
// sx [T][chunks] float; every region 256-byte aligned.
size_t up256(size_t n) { return (n + 255) / 256 * 256; }

}  // namespace

namespace {

// Enough tokens, and at most 512 quantization groups per row (the MFMA
// backbone keeps its rows' scales and zeros in LDS)
bool use_mfma(const QW& w, int T) { return T >= kMfmaMinTokens && w.d_in / w.G <= 512; }

// K parts of the MFMA preparation (at most 16, about 1024 codes each), the
// waves of a part's workgroup (4, 8 or 16: enough that each wave has at most
// eight 32-code steps, one round of loads -- the 14336-code rows took four
// dependent rounds on four waves) and the steps each wave takes
struct MfmaPlan {
    int kp, nw, spw;
};

MfmaPlan mfma_plan(int d_in, int max_kp = kMaxKp) {
    const int nsteps = d_in / 32;
    int kp = (d_in + 1023) / 1024;
    if (kp > max_kp) kp = max_kp;
    int nw = 4;
    while (nw < 16 && nsteps > nw * kp * 8) nw *= 2;
    return MfmaPlan{kp, nw, (nsteps + nw * kp - 1) / (nw * kp)};
}

int pad32(int r) { return (r + 31) / 32 * 32; }

// Quantization groups a 128-code block can meet, as the MFMA backbone sees
// them: 1 when G is a multiple of 128, 2 when it is a multiple of 64 (each
// half of a block lies in one group), else 4 (each 32-code step does)
int mfma_groups_per_block(int G) { return G % 128 == 0 ? 1 : (G % 64 == 0 ? 2 : 4); }

// Launch shape of the MFMA backbone: 16-row tiles per wave (tpw), K blocks
// in flight per wave (nbuf; halved when a block holds several groups, whose
// partials and scales need the registers) and waves splitting K (nw).
struct MfmaCfg {
    int tpw, nbuf, nw;
};

MfmaCfg mfma_cfg(int tiles, int groups) {
    if (tiles >= 1024 && 2 * 64 * szl_stride(groups) * 2 <= 32768) return MfmaCfg{4, 2, 4};
    return MfmaCfg{1, 4, 4};
}

// More than kPrefKp K parts (rows longer than 4096 codes) only on the
// one-tile instance with one group per block, the only one whose registers
// take the extra partials without losing a wave per SIMD.
bool long_k_ok(const MfmaCfg& c, int gpb) { return c.tpw == 1 && gpb == 1; }

template <int BITS, bool GLU, int GPB>
auto pick_cfg(const MfmaCfg& c, bool longk) {
    constexpr int H = GPB == 1 ? 1 : 2;           // nbuf divisor
    if (c.tpw == 4) return decode_mfma_kernel<BITS, 4, 2 / H, GLU, GPB, 4, false>;
    if (GPB == 1 && longk) return decode_mfma_kernel<BITS, 1, 4, GLU, 1, 4, true>;
    return decode_mfma_kernel<BITS, 1, 4 / H, GLU, GPB, 4, false>;
}

template <int BITS, bool GLU>
auto pick_gpb(const MfmaCfg& c, int gpb, bool longk) {
    if (gpb == 1) return pick_cfg<BITS, GLU, 1>(c, longk);
    // 2-bit groups are multiples of 64 codes: at most two per block
    if constexpr (BITS == 2) return pick_cfg<BITS, GLU, 2>(c, longk);
    else return gpb == 2 ? pick_cfg<BITS, GLU, 2>(c, longk) : pick_cfg<BITS, GLU, 4>(c, longk);
}

template <int BITS>
auto pick_glu(const MfmaCfg& c, bool glu, int gpb, bool longk) {
    return glu ? pick_gpb<BITS, true>(c, gpb, longk) : pick_gpb<BITS, false>(c, gpb, longk);
}

auto pick_mfma_kernel(const MfmaCfg& c, int bits, bool glu, int gpb, bool longk) {
    if (bits == 3) return pick_glu<3>(c, glu, gpb, longk);
    return bits == 2 ? pick_glu<2>(c, glu, gpb, longk) : pick_glu<4>(c, glu, gpb, longk);
}

}  // namespace

size_t decode_workspace_bytes(int n, const QW* w, const LR* c, int T) {
    size_t total = 0;
    const bool mf = use_mfma(w[0], T);
    const int kp = mf ? mfma_plan(w[0].d_in).kp : 0;
    for (int i = 0; i < n; ++i)
        total += mf ? up256(static_cast<size_t>(kp) * T * pad32(c[i].rank) * sizeof(float))
                    : up256(static_cast<size_t>(c[i].rank) * T * sizeof(float));
    if (mf) return total + up256(static_cast<size_t>((T + 15) / 16) * 16 * w[0].d_in * 2);
    const size_t chunks = static_cast<size_t>(w[0].d_in) / codes_per_chunk(w[0].bits);
    total += up256(static_cast<size_t>(T) * w[0].d_in * 2);
    total += up256(static_cast<size_t>(T) * chunks * sizeof(float));
    return total;
}

bool decode_fits(const QW& w) {
    const int chunks = w.d_in / codes_per_chunk(w.bits);
    return chunks <= 8 * 64 * 2;     // at most 8 K slices of 128 chunks
}

namespace {

// The many-token path: MFMA preparation (A x partials, activations), then
// the MFMA backbone in passes of 16 tokens.
hipError_t launch_decode_mfma(int n, const QW* w, const LR* c, const void* x, int T, int act, void* const* y,
                              int out, void* ws, hipStream_t st, bool glu) {
    const int d_in = w[0].d_in;
    char* wsb = static_cast<char*>(ws);
    PrepMArgs pa{};
    DecodeArgs a{};
    size_t off = 0;
    // row tiles per wave: four share each activation load (a quarter of the
    // activation traffic from L2: the gate+up window at 16 tokens went from
    // 45 us with one tile to ~34 us); small windows keep one tile per wave
    // for enough workgroups
    int tiles = 0;
    for (int i = 0; i < n; ++i) tiles += (w[i].d_out + 15) / 16;
    const int groups = d_in / w[0].G;
    // four tiles per wave when the workgroup's scales and zeros fit 32 KB of LDS
    const MfmaCfg cfg = mfma_cfg(tiles, groups);
    const int tpw = cfg.tpw;
    const int gpb = mfma_groups_per_block(w[0].G);
    // (the workspace query sizes the partials for the most parts)
    const MfmaPlan mp = mfma_plan(d_in, long_k_ok(cfg, gpb) ? kMaxKp : kPrefKp);
    int wg_end = 0, rtiles = 0, wg_first = 0;
    for (int i = 0; i < n; ++i) {
        float* tp = reinterpret_cast<float*>(wsb + off);
        const int rp = pad32(c[i].rank);
        off += up256(static_cast<size_t>(mp.kp) * T * rp * sizeof(float));
        pa.A[i] = c[i].A;
        pa.tp[i] = tp;
        pa.rank[i] = c[i].rank;
        pa.rpad[i] = rp;
        rtiles += rp / 16 * ((T + 15) / 16) * mp.kp;
        pa.tile_end[i] = rtiles;
        wg_end += ((w[i].d_out + 15) / 16 + tpw - 1) / tpw;
        if (i == 0) wg_first = wg_end;
        a.lin[i] = Lin{w[i].q, w[i].s, w[i].z, c[i].B, y[i], tp, w[i].d_out, c[i].rank, c[i].r_max, wg_end, rp};
    }
    const int npass = (T + 15) / 16;
    u32x4* xf = reinterpret_cast<u32x4*>(wsb + off);
    pa.n = n;
    pa.x = static_cast<const uint16_t*>(x);
    pa.xf = xf;
    pa.d_in = d_in;
    pa.T = T;
    pa.act = act;
    pa.kp = mp.kp;
    pa.spw = mp.spw;
    pa.npass = npass;
    const long long items = static_cast<long long>(npass) * (d_in / 8) * 16;
    const int pthreads = 64 * mp.nw;
    const unsigned grid = static_cast<unsigned>(rtiles + (items + pthreads - 1) / pthreads);
    hipLaunchKernelGGL(decode_prep_mfma_kernel, dim3(grid), dim3(pthreads), 0, st, pa);
    hipError_t e = hipGetLastError();
    a.n = n;
    a.xf = xf;
    a.d_in = d_in;
    a.G = w[0].G;
    a.T = T;
    a.out = out;
    a.ks = 4;
    a.cps = 0;
    a.kp = mp.kp;
    a.h = glu ? y[0] : nullptr;
    auto kern = pick_mfma_kernel(cfg, w[0].bits, glu, gpb, mp.kp > kPrefKp);
    // a gated window runs one workgroup of eight waves per gate workgroup
    // (four waves on the gate's tiles, four on the up tiles of the same rows),
    // with both linears' scales and zeros in LDS
    const size_t lds = static_cast<size_t>(2) * 16 * tpw * szl_stride(groups) * 2 * (glu ? 2 : 1);
    const int bgrid = glu ? wg_first : wg_end;
    for (int tok0 = 0; tok0 < T && e == hipSuccess; tok0 += 16) {
        a.tok0 = tok0;
        hipLaunchKernelGGL(kern, dim3(bgrid), dim3((glu ? 2 : 1) * 64 * cfg.nw), lds, st, a);
        e = hipGetLastError();
    }
    return e;
}

}  // namespace

hipError_t launch_linear_decode(int n, const QW* w, const LR* c, const void* x, int T, int act,
                                void* const* y, int out, void* ws, hipStream_t st, bool glu) {
    const int d_in = w[0].d_in, bits = w[0].bits;
    if (n < 1 || n > kMaxWin) return hipErrorInvalidConfiguration;
    if (glu && (n != 2 || w[0].d_out != w[1].d_out)) return hipErrorInvalidConfiguration;
    if (use_mfma(w[0], T)) return launch_decode_mfma(n, w, c, x, T, act, y, out, ws, st, glu);
    int max_rank = 0;
    for (int i = 0; i < n; ++i) max_rank = max(max_rank, c[i].rank);
    const Plan p = plan(d_in, bits, max_rank, T);
    // the kernel is built for at most 8 waves (launch bounds, LDS arrays)
    if (n < 1 || n > kMaxWin || p.ks > 8 || p.threads > 512 || p.threads % (64 * p.ks))
        return hipErrorInvalidConfiguration;
    char* wsb = static_cast<char*>(ws);
    PrepArgs pa;
    DecodeArgs a;
    size_t off = 0;
    int rank_end = 0, batch_end = 0;
    const int rg_per_block = p.threads / 64 / p.ks;
    for (int i = 0; i < n; ++i) {
        float* t = reinterpret_cast<float*>(wsb + off);
        off += up256(static_cast<size_t>(c[i].rank) * T * sizeof(float));
        rank_end += c[i].rank;
        pa.A[i] = c[i].A;
        pa.t[i] = t;
        pa.rank_end[i] = rank_end;
        const int rgroups = (w[i].d_out + p.R - 1) / p.R;
        batch_end += (rgroups + rg_per_block - 1) / rg_per_block;
        a.lin[i] = Lin{w[i].q, w[i].s, w[i].z, c[i].B, y[i], t, w[i].d_out, c[i].rank, c[i].r_max, batch_end};
    }
    const int chunks = d_in / codes_per_chunk(bits);
    f16x2* xp = reinterpret_cast<f16x2*>(wsb + off);
    off += up256(static_cast<size_t>(T) * d_in * 2);
    float* sx = reinterpret_cast<float*>(wsb + off);
    pa.n = n;
    pa.x = static_cast<const uint16_t*>(x);
    pa.xp = xp;
    pa.sx = sx;
    pa.d_in = d_in;
    pa.T = T;
    pa.act = act;
    pa.wpr = prep_waves_per_row(d_in);
    const long long items = static_cast<long long>(T) * chunks;
    const int rows_per_block = 4 / pa.wpr;
    const unsigned grid = static_cast<unsigned>((rank_end + rows_per_block - 1) / rows_per_block + (items + 255) / 256);
    if (bits == 4)
        hipLaunchKernelGGL(decode_prep_kernel<4>, dim3(grid), dim3(256), 0, st, pa);
    else if (bits == 3)
        hipLaunchKernelGGL(decode_prep_kernel<3>, dim3(grid), dim3(256), 0, st, pa);
    else
        hipLaunchKernelGGL(decode_prep_kernel<2>, dim3(grid), dim3(256), 0, st, pa);
    hipError_t e = hipGetLastError();
    a.n = n;
    a.xp = xp;
    a.sx = sx;
    a.d_in = d_in;
    a.G = w[0].G;
    a.T = T;
    a.out = out;
    a.ks = p.ks;
    a.cps = p.cps;
    a.h = glu ? y[0] : nullptr;
    for (int tok0 = 0; tok0 < T && e == hipSuccess; tok0 += p.nt) {
        a.tok0 = tok0;
        e = bits == 4 ? launch2<4>(a, p, st) : (bits == 3 ? launch2<3>(a, p, st) : launch2<2>(a, p, st));
    }
    return e;
}

}  // namespace cl
