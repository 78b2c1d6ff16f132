// Decode path of the error-compensated quantized linear (few tokens):
//
//     y[t] = deq(Q) x[t] + B[:, :r] (A[:r] x[t])          (Section 4.1)
//
// Two kernels on the caller's stream:
//   1. lowrank_down:  t[tok][i] = A[i] . x[tok]  (fp32, into the workspace)
//   2. decode_gemv:   streams the packed backbone once with 16-byte loads,
//      unpacks codes straight into fp16 lanes, runs v_dot2 against fp16
//      activations staged in LDS, applies each group's scale and zero point
//      in fp32, adds the rank-r up-projection B[o, :r] . t and rounds once.
//
// The backbone is HBM-bound (about half a byte per weight at 4 bits), so the
// kernel is organised around the memory stream: a wave owns ROWS consecutive
// rows and its 64 lanes sweep the row's 16-byte chunks side by side, so each
// load instruction reads ROWS fully coalesced 1 KiB segments; every lane keeps
// the activations of its chunk in registers and reuses them for all ROWS
// rows.  Small matrices split K over 2 or 4 waves of the workgroup (reduced
// through LDS in a fixed order, so results are bitwise reproducible).

#include "cl_device.h"
#include "cl_internal.h"

namespace cl {

namespace {

constexpr int kBlock = 256;   // 4 waves
constexpr int kMaxTok = 4;    // tokens per pass of the VALU kernel

struct DecodeArgs {
    const uint32_t* q;
    const uint16_t* s;
    const uint16_t* z;
    const uint16_t* B;
    const float* t;        // [T][rank] fp32, rank may be 0
    const uint16_t* x;     // [T][d_in] fp16/bf16 bits
    void* y;               // [T][d_out]
    int d_out, d_in, G, rank, r_max, T, tok0, act, out, ksplit;
};

// t[tok][i] = sum_c A[i][c] * x[tok][c]; one wave per (i), all tokens.
__global__ __launch_bounds__(kBlock) void lowrank_down_kernel(const uint16_t* __restrict__ A,
                                                              const uint16_t* __restrict__ x,
                                                              float* __restrict__ t, int d_in,
                                                              int rank, int T, int act) {
    const int lane = threadIdx.x & 63;
    const int i = blockIdx.x * (kBlock / 64) + (threadIdx.x >> 6);
    if (i >= rank) return;   // whole wave exits together; no barriers below
    const uint16_t* a = A + static_cast<size_t>(i) * d_in;
    for (int tok = 0; tok < T; ++tok) {
        const uint16_t* xr = x + static_cast<size_t>(tok) * d_in;
        float acc = 0.f;
        for (int c = lane * 8; c < d_in; c += 64 * 8) {
            const u32x4 av = *reinterpret_cast<const u32x4*>(a + c);
            const u32x4 xv = *reinterpret_cast<const u32x4*>(xr + c);
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const uint32_t aw = av[k], xw = xv[k];
                acc = fmaf(f16_bits_to_f32(aw & 0xffff), act_to_f32(xw & 0xffff, act), acc);
                acc = fmaf(f16_bits_to_f32(aw >> 16), act_to_f32(xw >> 16, act), acc);
            }
        }
        acc = wave_sum(acc);
        if (lane == 0) t[static_cast<size_t>(tok) * rank + i] = acc;
    }
}

template <int BITS, int NT, int ROWS>
__global__ __launch_bounds__(kBlock) void decode_gemv_kernel(DecodeArgs a) {
    constexpr int CPW = 32 / BITS;       // codes per 32-bit word
    constexpr int HPW = CPW / 2;         // fp16 pairs per word
    constexpr int CPC = 4 * CPW;         // codes per 16-byte chunk (32 or 64)
    constexpr int PPC = 4 * HPW;         // fp16 pairs per chunk (16 or 32)

    extern __shared__ uint32_t smem[];
    const int words = a.d_in / CPW;              // words per row
    const int chunks = words / 4;
    f16x2* xs = reinterpret_cast<f16x2*>(smem);  // [NT][d_in / 2], pair-permuted
    float* ts = reinterpret_cast<float*>(smem + NT * (a.d_in / 2));  // [NT][rank]
    float* red = ts + NT * a.rank;               // [4 waves][ROWS][NT]

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;

    // Stage this pass's activations as the (q_p, q_{p+HPW}) pair order of the
    // unpacked codes: word w, pair p holds (x[w*CPW + p], x[w*CPW + p + HPW]).
    for (int idx = tid; idx < NT * words; idx += kBlock) {
        const int tk = idx / words, w = idx - tk * words;
        if (a.tok0 + tk >= a.T) continue;
        const uint16_t* src = a.x + static_cast<size_t>(a.tok0 + tk) * a.d_in + static_cast<size_t>(w) * CPW;
        uint16_t v[CPW];
#pragma unroll
        for (int j = 0; j < CPW; j += 8) {
            const u32x4 u = *reinterpret_cast<const u32x4*>(src + j);
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                v[j + 2 * k] = static_cast<uint16_t>(u[k] & 0xffff);
                v[j + 2 * k + 1] = static_cast<uint16_t>(u[k] >> 16);
            }
        }
#pragma unroll
        for (int p = 0; p < HPW; ++p) {
            f16x2 pr;
            pr.x = act_to_f16(v[p], a.act);
            pr.y = act_to_f16(v[p + HPW], a.act);
            xs[static_cast<size_t>(tk) * (a.d_in / 2) + w * HPW + p] = pr;
        }
    }
    for (int idx = tid; idx < NT * a.rank; idx += kBlock) {
        const int tk = idx / a.rank;
        ts[idx] = (a.tok0 + tk < a.T) ? a.t[static_cast<size_t>(a.tok0) * a.rank + idx] : 0.f;
    }
    __syncthreads();

    const int sets = kBlock / 64 / a.ksplit;
    const int set = blockIdx.x * sets + wave / a.ksplit;
    const int kpart = wave % a.ksplit;
    const int row0 = set * ROWS;
    const int groups = a.d_in / a.G;
    const int lanes = 64 * a.ksplit;

    float acc[ROWS][NT];
#pragma unroll
    for (int r = 0; r < ROWS; ++r)
#pragma unroll
        for (int tk = 0; tk < NT; ++tk) acc[r][tk] = 0.f;

    if (row0 < a.d_out) {
        const int nrows = min(ROWS, a.d_out - row0);
        for (int c = lane + 64 * kpart; c < chunks; c += lanes) {
            u32x4 qv[ROWS];
#pragma unroll
            for (int r = 0; r < ROWS; ++r) {
                const int row = row0 + (r < nrows ? r : 0);
                qv[r] = __builtin_nontemporal_load(
                    reinterpret_cast<const u32x4*>(a.q + static_cast<size_t>(row) * words) + c);
            }
            const int g = (c * CPC) / a.G;
            float sc[ROWS], sz[ROWS];
#pragma unroll
            for (int r = 0; r < ROWS; ++r) {
                const int row = row0 + (r < nrows ? r : 0);
                const float s = f16_bits_to_f32(a.s[static_cast<size_t>(row) * groups + g]);
                const float zz = f16_bits_to_f32(a.z[static_cast<size_t>(row) * groups + g]);
                sc[r] = s * 16777216.0f;   // undo the 2^-24 of the subnormal codes
                sz[r] = s * zz;
            }
#pragma unroll
            for (int tk = 0; tk < NT; ++tk) {
                const f16x2* xp = xs + static_cast<size_t>(tk) * (a.d_in / 2) + static_cast<size_t>(c) * PPC;
                f16x2 xv[PPC];
#pragma unroll
                for (int p = 0; p < PPC; ++p) xv[p] = xp[p];
                const f16x2 one = {static_cast<f16>(1.0f), static_cast<f16>(1.0f)};
                float sx = 0.f;
#pragma unroll
                for (int p = 0; p < PPC; ++p) sx = dot2(xv[p], one, sx);
#pragma unroll
                for (int r = 0; r < ROWS; ++r) {
                    float d = 0.f;
#pragma unroll
                    for (int wd = 0; wd < 4; ++wd)
#pragma unroll
                        for (int p = 0; p < HPW; ++p)
                            d = dot2(code_pair<BITS>(qv[r][wd], p), xv[wd * HPW + p], d);
                    acc[r][tk] = fmaf(sc[r], d, fmaf(-sz[r], sx, acc[r][tk]));
                }
            }
        }
        // rank-r up-projection, split over the lanes of the row set
        if (a.rank > 0) {
            for (int r = 0; r < nrows; ++r) {
                const uint16_t* br = a.B + static_cast<size_t>(row0 + r) * a.r_max;
                for (int i = lane + 64 * kpart; i < a.rank; i += lanes) {
                    const float b = f16_bits_to_f32(br[i]);
#pragma unroll
                    for (int tk = 0; tk < NT; ++tk) acc[r][tk] = fmaf(b, ts[tk * a.rank + i], acc[r][tk]);
                }
            }
        }
    }
#pragma unroll
    for (int r = 0; r < ROWS; ++r)
#pragma unroll
        for (int tk = 0; tk < NT; ++tk) {
            const float v = wave_sum(acc[r][tk]);
            if (lane == 0) red[(wave * ROWS + r) * NT + tk] = v;
        }
    __syncthreads();
    if (kpart == 0 && lane < ROWS * NT) {
        const int r = lane / NT, tk = lane - r * NT;
        const int row = row0 + r;
        if (row < a.d_out && a.tok0 + tk < a.T) {
            float v = 0.f;
            for (int k = 0; k < a.ksplit; ++k) v += red[((wave + k) * ROWS + r) * NT + tk];
            store_out(a.y, static_cast<size_t>(a.tok0 + tk) * a.d_out + row, v, a.out);
        }
    }
}

constexpr size_t kMaxLds = 65536;

size_t lds_bytes(int d_in, int rank, int nt, int rows) {
    return static_cast<size_t>(nt) * (static_cast<size_t>(d_in) / 2 * 4 + static_cast<size_t>(rank) * 4) +
           static_cast<size_t>(4) * rows * nt * 4;
}

template <int BITS, int NT, int ROWS>
hipError_t launch_gemv(const DecodeArgs& a, hipStream_t st) {
    const int sets = (a.d_out + ROWS - 1) / ROWS;
    const int sets_per_block = kBlock / 64 / a.ksplit;
    const unsigned grid = static_cast<unsigned>((sets + sets_per_block - 1) / sets_per_block);
    const size_t lds = lds_bytes(a.d_in, a.rank, NT, ROWS);
    hipLaunchKernelGGL((decode_gemv_kernel<BITS, NT, ROWS>), dim3(grid), dim3(kBlock), lds, st, a);
    return hipGetLastError();
}

template <int BITS>
hipError_t launch_bits(DecodeArgs a, hipStream_t st) {
    constexpr int ROWS = 4;
    // split K across waves when there are too few row sets to fill the chip
    const int sets = (a.d_out + ROWS - 1) / ROWS;
    a.ksplit = sets >= 4096 ? 1 : (sets >= 2048 ? 2 : 4);
    // tokens per pass: as many as the staged activations leave room for
    int per_pass = kMaxTok;
    while (per_pass > 1 && lds_bytes(a.d_in, a.rank, per_pass, ROWS) > kMaxLds) per_pass >>= 1;
    hipError_t e = hipSuccess;
    for (a.tok0 = 0; a.tok0 < a.T && e == hipSuccess; a.tok0 += per_pass) {
        const int n = min(per_pass, a.T - a.tok0);
        if (n == 1) e = launch_gemv<BITS, 1, ROWS>(a, st);
        else if (n == 2) e = launch_gemv<BITS, 2, ROWS>(a, st);
        else e = launch_gemv<BITS, 4, ROWS>(a, st);
    }
    return e;
}

}  // namespace

size_t decode_workspace_bytes(const QW&, const LR& c, int T) {
    return static_cast<size_t>(c.rank) * T * sizeof(float);
}

bool decode_fits(const QW& w, const LR& c) { return lds_bytes(w.d_in, c.rank, 1, 4) <= kMaxLds; }

hipError_t launch_linear_decode(const QW& w, const LR& c, const void* x, int T, int act, void* y,
                                int out, void* ws, hipStream_t st) {
    float* t = static_cast<float*>(ws);
    if (c.rank > 0) {
        const unsigned grid = static_cast<unsigned>((c.rank + 3) / 4);
        hipLaunchKernelGGL(lowrank_down_kernel, dim3(grid), dim3(kBlock), 0, st, c.A,
                           static_cast<const uint16_t*>(x), t, w.d_in, c.rank, T, act);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    DecodeArgs a;
    a.q = w.q; a.s = w.s; a.z = w.z; a.B = c.B; a.t = t;
    a.x = static_cast<const uint16_t*>(x); a.y = y;
    a.d_out = w.d_out; a.d_in = w.d_in; a.G = w.G; a.rank = c.rank; a.r_max = c.r_max;
    a.T = T; a.tok0 = 0; a.act = act; a.out = out; a.ksplit = 1;
    return w.bits == 4 ? launch_bits<4>(a, st) : launch_bits<2>(a, st);
}

}  // namespace cl
