// Decode path of the error-compensated quantized linear (few tokens):
//
//     y[t] = deq(Q) x[t] + B[:, :r] (A[:r] x[t])          (Section 4.1)
//
// Two launches per call (one when rank = 0).  The backbone is HBM-bound (about half a byte per
// weight at 4 bits, a quarter at 2 bits), so the kernel is built around the
// memory stream:
//
//  * A "row group" of KS waves owns R consecutive rows.  The row's 16-byte
//    chunks of packed codes are split into KS slices; lane l of slice k
//    handles chunks k*cps + l + 64j (j < CPL).  Every wave issues all R*CPL of
//    its 16-byte loads before it computes anything, so each lane has 8-16
//    independent loads in flight and each load instruction reads R fully
//    coalesced segments.
//  * Codes are unpacked with one AND per pair straight into fp16 lanes (the
//    code q in the low mantissa bits of a zero-exponent fp16 is the subnormal
//    q * 2^-24, exact), multiplied with the lane's activations by v_dot2 into
//    fp32, and each chunk's scale and zero point are applied in fp32:
//    s * (sum q x) - s * z * (sum x), with the 2^24 folded into s.
//  * Activations of the lane's chunks live in registers for the whole kernel,
//    pre-permuted to the (q_p, q_{p+CPW/2}) pair order of the unpacked codes.
//  * The rank-r term needs t = A[:r] x before any row can finish.  A small
//    kernel ahead of the backbone kernel computes it (one workgroup per row
//    of A, every load in flight at once, fixed-order reduction) into the
//    workspace; the stream order makes it visible to the backbone kernel.
//    Synchronising inside one launch instead would need device-scope
//    release/acquire between workgroups on different XCDs, whose L2
//    writeback/invalidate costs far more than the second launch.
//  * Sums over lanes use a transposing butterfly (R values in log steps), the
//    KS slices are combined through LDS in a fixed order: results are bitwise
//    reproducible.

#include "cl_device.h"
#include "cl_internal.h"

namespace cl {

namespace {

struct DecodeArgs {
    const uint32_t* q;
    const uint16_t* s;
    const uint16_t* z;
    const uint16_t* A;
    const uint16_t* B;
    const f16x2* xp;       // [T][d_in / 2] activations, fp16, pair-permuted
    const float* sx;       // [T][chunks] per-chunk sums of activations
    void* y;               // [T][d_out]
    const float* t;        // [T][rank]
    int d_out, d_in, G, rank, r_max, T, tok0, act, out;
    int ks;                // K slices (waves per row group)
    int cps;               // chunks per slice
};

// Load 8 consecutive activations as four f16x2 words (fp16 or bf16 input).
__device__ __forceinline__ void load8_f16(const uint16_t* p, int act, uint32_t out[4]) {
    const u32x4 u = *reinterpret_cast<const u32x4*>(p);
    if (act == DT_FP16) {
        out[0] = u[0]; out[1] = u[1]; out[2] = u[2]; out[3] = u[3];
    } else {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            f16x2 h;
            h.x = act_to_f16(static_cast<uint16_t>(u[k] & 0xffff), act);
            h.y = act_to_f16(static_cast<uint16_t>(u[k] >> 16), act);
            out[k] = __builtin_bit_cast(uint32_t, h);
        }
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

// Preparation kernel, run once per call ahead of the backbone kernel:
//  * workgroups [0, rank): t[tok][i] = A[i] . x[tok] for every token (one row
//    of A per workgroup, every thread's 16-byte loads issued before any
//    arithmetic, fixed-order reduction);
//  * the remaining workgroups: the activations converted to fp16 and
//    permuted into the pair order of the unpacked codes (word w, pair p =
//    (x[w*CPW + p], x[w*CPW + p + CPW/2])), plus each 16-byte chunk's sum of
//    activations, so the backbone kernel only loads them.
template <int BITS>
__global__ __launch_bounds__(256) void decode_prep_kernel(const uint16_t* __restrict__ A,
                                                          const uint16_t* __restrict__ x,
                                                          float* __restrict__ t, f16x2* __restrict__ xp,
                                                          float* __restrict__ sx, int d_in, int rank, int T,
                                                          int act) {
    constexpr int CPW = 32 / BITS, HPW = CPW / 2, PPC = 4 * HPW;
    constexpr int KB = 4;                   // 16-byte loads per thread per batch
    constexpr int TB = 4;                   // tokens per pass over a row of A
    __shared__ float part[4][TB];
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int tid = threadIdx.x;
    if (static_cast<int>(blockIdx.x) < rank) {
        const int i = blockIdx.x;
        const uint16_t* ar = A + static_cast<size_t>(i) * d_in;
        for (int base = 0; base < d_in; base += 256 * 8 * KB) {
            u32x4 av[KB];
            int col[KB];
#pragma unroll
            for (int k = 0; k < KB; ++k) {
                col[k] = base + (tid + k * 256) * 8;
                av[k] = *reinterpret_cast<const u32x4*>(ar + (col[k] < d_in ? col[k] : 0));
            }
            for (int tb = 0; tb < T; tb += TB) {
                float acc[TB];
#pragma unroll
                for (int tk = 0; tk < TB; ++tk) {
                    acc[tk] = 0.f;
                    if (tb + tk >= T) continue;
                    const uint16_t* xr = x + static_cast<size_t>(tb + tk) * d_in;
#pragma unroll
                    for (int k = 0; k < KB; ++k) {
                        uint32_t xw[4];
                        load8_f16(xr + (col[k] < d_in ? col[k] : 0), act, xw);
                        float d = 0.f;
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            // copy the vector element to a scalar first: a bit_cast
                            // of a subscripted ext_vector reads element 0
                            const uint32_t ak = av[k][e], xk = xw[e];
                            d = dot2(__builtin_bit_cast(f16x2, ak), __builtin_bit_cast(f16x2, xk), d);
                        }
                        acc[tk] += col[k] < d_in ? d : 0.f;
                    }
                }
#pragma unroll
                for (int tk = 0; tk < TB; ++tk) {
                    const float v = wave_sum(acc[tk]);
                    if (lane == 0) part[wave][tk] = v;
                }
                __syncthreads();
                if (tid < TB && tb + tid < T) {
                    float* dst = t + static_cast<size_t>(tb + tid) * rank + i;
                    const float v = part[0][tid] + part[1][tid] + part[2][tid] + part[3][tid];
                    *dst = base == 0 ? v : *dst + v;
                }
                __syncthreads();
            }
        }
        return;
    }
    // activation preparation: one thread per (token, chunk)
    const int chunks = d_in / CPW / 4;
    const long long item = static_cast<long long>(blockIdx.x - rank) * 256 + tid;
    if (item >= static_cast<long long>(T) * chunks) return;
    const int tok = static_cast<int>(item / chunks);
    const int c = static_cast<int>(item % chunks);
    f16x2 v[PPC];
    load_chunk_x<BITS>(x + static_cast<size_t>(tok) * d_in, c, act, v);
    const f16x2 one = {static_cast<f16>(1.0f), static_cast<f16>(1.0f)};
    float sum = 0.f;
    f16x2* dst = xp + static_cast<size_t>(tok) * (d_in / 2) + static_cast<size_t>(c) * PPC;
#pragma unroll
    for (int p = 0; p < PPC; ++p) {
        sum = dot2(v[p], one, sum);
        dst[p] = v[p];
    }
    sx[static_cast<size_t>(tok) * chunks + c] = sum;
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

// sum of q * x * 2^-24 over the word(s): the per-scale accumulators with
// their power-of-two scales removed
template <int BITS>
__device__ __forceinline__ float combine(const float* d) {
    if (BITS == 4) return fmaf(d[1], 0.0625f, d[0]);
    return fmaf(d[3], 0.015625f, fmaf(d[2], 0.0625f, fmaf(d[1], 0.25f, d[0])));
}

// One batch of a wave: R rows x CPL chunks of packed codes, the matching
// scale/zero pairs and the rows' factor entries.
// Raw loads only: nothing may consume a value at load time, or the wave
// would stall on the prefetch it is meant to overlap.
template <int R, int CPL, int NB>
struct Batch {
    u32x4 q[R][CPL];
    uint16_t s[R][CPL];      // fp16 scale bits
    uint16_t z[R][CPL];      // fp16 zero-point bits
    uint16_t b[R][NB];       // B[row][i] for this lane's factor columns (NB >= 1)
};

// NB: factor columns of B per lane (rank <= NB * 64 * ks); 0 for rank 0.
template <int BITS, int NT, int CPL, int R, int NB>
__global__ __launch_bounds__(512) void decode_kernel(DecodeArgs a) {
    constexpr int CPW = 32 / BITS;    // codes per word
    constexpr int HPW = CPW / 2;      // fp16 pairs per word
    constexpr int CPC = 4 * CPW;      // codes per chunk
    constexpr int PPC = 4 * HPW;      // pairs per chunk
    constexpr int NACC = BITS == 4 ? 2 : 4;
    constexpr int NBA = NB > 0 ? NB : 1;
    constexpr bool XREG = NT * CPL * PPC <= 32;   // activations stay in registers

    __shared__ float red[2][8][R][NT];

    const int lane = threadIdx.x & 63;
    // wave-uniform values in scalar registers: row addressing stays scalar
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int waves = blockDim.x >> 6;
    const int words = a.d_in / CPW;
    const int chunks = words / 4;
    const int groups = a.d_in / a.G;
    const int ks = a.ks;
    const int rg_per_block = waves / ks;
    const int slice = wave % ks;
    const int rgw = wave / ks;
    const int rgroups = (a.d_out + R - 1) / R;
    const int nbatch = (rgroups + rg_per_block - 1) / rg_per_block;
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

    // activations of this lane's chunks (prepared: fp16, pair-permuted) and
    // their sums
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
    // this lane's entries of t = A x (factor columns lane + 64*(slice + ks*m))
    float tv[NT][NBA];
#pragma unroll
    for (int tk = 0; tk < NT; ++tk)
#pragma unroll
        for (int m = 0; m < NBA; ++m) {
            const int i = lane + 64 * (slice + ks * m);
            tv[tk][m] = (i < a.rank && a.tok0 + tk < a.T) ? a.t[static_cast<size_t>(tk) * a.rank + i] : 0.f;
        }

    auto load_batch = [&](Batch<R, CPL, NBA>& bt, int b) {
        const int row0 = (b * rg_per_block + rgw) * R;
        const int base = row0 < a.d_out ? row0 : 0;
        const int nrows = row0 < a.d_out ? min(R, a.d_out - row0) : 1;
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int row = base + (r < nrows ? r : 0);
            const u32x4* qr = reinterpret_cast<const u32x4*>(a.q + static_cast<size_t>(row) * words);
#pragma unroll
            for (int j = 0; j < CPL; ++j) bt.q[r][j] = __builtin_nontemporal_load(qr + cidx[j]);
#pragma unroll
            for (int j = 0; j < CPL; ++j) {
                const size_t gi = static_cast<size_t>(row) * groups + (cidx[j] * CPC) / a.G;
                bt.s[r][j] = a.s[gi];
                bt.z[r][j] = a.z[gi];
            }
#pragma unroll
            for (int m = 0; m < NB; ++m) {
                // columns past the rank read column 0 (valid data) and meet t = 0
                const int i = lane + 64 * (slice + ks * m);
                bt.b[r][m] = a.B[static_cast<size_t>(row) * a.r_max + (i < a.rank ? i : 0)];
            }
        }
    };

    auto compute_batch = [&](const Batch<R, CPL, NBA>& bt, int b, int buf) {
        const int row0 = (b * rg_per_block + rgw) * R;
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
                const f16x2* xp = XREG ? xv[XREG ? tk : 0][XREG ? j : 0] : xl;
#pragma unroll
                for (int r = 0; r < R; ++r) {
                    float d[NACC];
#pragma unroll
                    for (int k = 0; k < NACC; ++k) d[k] = 0.f;
#pragma unroll
                    for (int w = 0; w < 4; ++w) dot_word<BITS>(bt.q[r][j][w], xp + w * HPW, d);
                    const float sc = f16_bits_to_f32(bt.s[r][j]) * cmask[j];
                    const float zc = f16_bits_to_f32(bt.z[r][j]);
                    // s * (2^24 * sum q x - z * sum x): the codes were subnormals q * 2^-24
                    const float v = fmaf(combine<BITS>(d), 16777216.0f, -zc * sx[tk][j]);
                    acc[r][tk] = fmaf(sc, v, acc[r][tk]);
                }
            }
        }
        // rank-r up-projection: B[row, i] * t[i] over this lane's factor columns
#pragma unroll
        for (int r = 0; r < R; ++r)
#pragma unroll
            for (int m = 0; m < NB; ++m) {
                const float bv = f16_bits_to_f32(bt.b[r][m]);
#pragma unroll
                for (int tk = 0; tk < NT; ++tk) acc[r][tk] = fmaf(bv, tv[tk][m], acc[r][tk]);
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
                    if (row0 + rr < a.d_out && a.tok0 + tk < a.T)
                        store_out(a.y, static_cast<size_t>(a.tok0 + tk) * a.d_out + row0 + rr, tot, a.out);
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
            if (row < a.d_out && a.tok0 + tk < a.T) {
                float v = 0.f;
                for (int k = 0; k < ks; ++k) v += red[buf][wave + k][r][tk];
                store_out(a.y, static_cast<size_t>(a.tok0 + tk) * a.d_out + row, v, a.out);
            }
        }
    };

    // Persistent loop over batches with the next batch's loads in flight
    // during the current batch's arithmetic (two register sets, alternating
    // LDS buffers).  Every compute site has a single predecessor shape (next
    // batch issued, or this is the last batch) so the compiler's wait counts
    // let the prefetch stay in flight.
    const int stride = gridDim.x;
    int b = blockIdx.x;
    if (b >= nbatch) return;
    Batch<R, CPL, NBA> b0, b1;
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

struct Plan {
    int cpl, R, ks, cps, nt, nb, threads;
};

Plan plan(const QW& w, const LR& c, int T) {
    const int CPW = 32 / w.bits;
    const int chunks = w.d_in / CPW / 4;
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
    p.nb = c.rank == 0 ? 0 : (c.rank <= per ? 1 : (c.rank <= 2 * per ? 2 : 4));
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
    auto kern = decode_kernel<BITS, NT, CPL, R, NB>;
    // resident workgroups per CU for this instance (cached once per process)
    static int occ = 0;
    if (!occ) {
        int n = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kern, p.threads, 0) != hipSuccess || n <= 0) n = 1;
        occ = n;
    }
    const int rgroups = (a.d_out + R - 1) / R;
    const int rg_per_block = p.threads / 64 / p.ks;
    const int nbatch = (rgroups + rg_per_block - 1) / rg_per_block;
    // at most one resident wave of workgroups, each with the same number of
    // batches (no partial second wave)
    const int cap = occ * device_cus();
    const int per = (nbatch + cap - 1) / cap;
    const int blocks = (nbatch + per - 1) / per;
    hipLaunchKernelGGL(kern, dim3(blocks), dim3(p.threads), 0, st, a);
    return hipGetLastError();
}

template <int BITS, int NT, int CPL, int R>
hipError_t launch4(const DecodeArgs& a, const Plan& p, hipStream_t st) {
    switch (p.nb) {
        case 0: return launch5<BITS, NT, CPL, R, 0>(a, p, st);
        case 1: return launch5<BITS, NT, CPL, R, 1>(a, p, st);
        case 2: return launch5<BITS, NT, CPL, R, 2>(a, p, st);
        default: return launch5<BITS, NT, CPL, R, 4>(a, p, st);
    }
}

template <int BITS, int NT, int CPL>
hipError_t launch_r(const DecodeArgs& a, const Plan& p, hipStream_t st) {
    return launch4<BITS, NT, CPL, 4>(a, p, st);
}

template <int BITS, int NT>
hipError_t launch3(const DecodeArgs& a, const Plan& p, hipStream_t st) {
    return p.cpl == 2 ? launch_r<BITS, NT, 2>(a, p, st) : launch_r<BITS, NT, 1>(a, p, st);
}

template <int BITS>
hipError_t launch2(const DecodeArgs& a, const Plan& p, int nt, hipStream_t st) {
    if (nt == 1) return launch3<BITS, 1>(a, p, st);
    if (nt == 2) return launch3<BITS, 2>(a, p, st);
    return launch3<BITS, 4>(a, p, st);
}

}  // namespace

// Workspace: t [T][rank] float | xp [T][d_in/2] fp16 pairs | sx [T][chunks]
// float, each region 256-byte aligned.
struct WsLayout {
    size_t t, xp, sx, total;
};

WsLayout ws_layout(const QW& w, const LR& c, int T) {
    auto up = [](size_t n) { return (n + 255) / 256 * 256; };
    const size_t chunks = static_cast<size_t>(w.d_in) / (32 / w.bits) / 4;
    WsLayout l;
    l.t = 0;
    l.xp = up(static_cast<size_t>(c.rank) * T * sizeof(float));
    l.sx = l.xp + up(static_cast<size_t>(T) * w.d_in * 2);
    l.total = l.sx + up(static_cast<size_t>(T) * chunks * sizeof(float));
    return l;
}

size_t decode_workspace_bytes(const QW& w, const LR& c, int T) { return ws_layout(w, c, T).total; }

bool decode_fits(const QW& w, const LR&) {
    const int chunks = w.d_in / (32 / w.bits) / 4;
    return chunks <= 8 * 64 * 2;     // at most 8 K slices of 128 chunks
}

hipError_t launch_linear_decode(const QW& w, const LR& c, const void* x, int T, int act, void* y,
                                int out, void* ws, hipStream_t st) {
    const Plan p = plan(w, c, T);
    // the kernel is built for at most 8 waves (launch bounds, LDS arrays)
    if (p.ks > 8 || p.threads > 512 || p.threads % (64 * p.ks)) return hipErrorInvalidConfiguration;
    const WsLayout l = ws_layout(w, c, T);
    char* wsb = static_cast<char*>(ws);
    float* t = reinterpret_cast<float*>(wsb + l.t);
    f16x2* xp = reinterpret_cast<f16x2*>(wsb + l.xp);
    float* sx = reinterpret_cast<float*>(wsb + l.sx);
    const int chunks = w.d_in / (32 / w.bits) / 4;
    const long long items = static_cast<long long>(T) * chunks;
    const unsigned grid = static_cast<unsigned>(c.rank + (items + 255) / 256);
    const uint16_t* xs = static_cast<const uint16_t*>(x);
    if (w.bits == 4)
        hipLaunchKernelGGL(decode_prep_kernel<4>, dim3(grid), dim3(256), 0, st, c.A, xs, t, xp, sx, w.d_in, c.rank, T, act);
    else
        hipLaunchKernelGGL(decode_prep_kernel<2>, dim3(grid), dim3(256), 0, st, c.A, xs, t, xp, sx, w.d_in, c.rank, T, act);
    hipError_t e = hipGetLastError();
    DecodeArgs a;
    a.q = w.q; a.s = w.s; a.z = w.z; a.A = c.A; a.B = c.B;
    a.xp = xp; a.y = y;
    a.d_out = w.d_out; a.d_in = w.d_in; a.G = w.G; a.rank = c.rank; a.r_max = c.r_max;
    a.T = T; a.act = act; a.out = out;
    a.ks = p.ks; a.cps = p.cps;
    for (int tok0 = 0; tok0 < T && e == hipSuccess; tok0 += p.nt) {
        a.tok0 = tok0;
        a.t = t + static_cast<size_t>(tok0) * c.rank;
        a.sx = sx;
        e = w.bits == 4 ? launch2<4>(a, p, p.nt, st) : launch2<2>(a, p, p.nt, st);
    }
    return e;
}

}  // namespace cl
