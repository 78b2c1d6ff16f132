// Compensation factors from the quantization error, on the GPU, in fp64.
//
// The paper takes the compensation factors from the singular value
// decomposition of the residual E = W - W_hat (Section 4.1) and relies on the
// truncated SVD being the best rank-r approximation, its squared Frobenius
// error being the sum of the squared tail singular values (Appendix B.2,
// Eckart-Young-Mirsky).  With E = U diag(sigma) V^T, sigma descending:
//
//     A = diag(sqrt(sigma[:r_max])) V^T[:r_max]        (r_max x d_in)
//     B = U[:, :r_max] diag(sqrt(sigma[:r_max]))       (d_out x r_max)
//
// so B[:, :r] A[:r] is the rank-r truncation for every r <= r_max; the sign of
// each singular pair makes the largest-magnitude entry of the U column
// positive (first index on ties).
//
// Steps (all fp64, one stream, the host waits once per Jacobi sweep):
//  1. E = W - s (q - z) elementwise.
//  2. The Gram matrix over the smaller side, C = E^T E (d_in <= d_out) or
//     C = E E^T, with a tiled fp64 GEMM (64 x 64 tiles through LDS).
//  3. Eigen-decomposition C = X diag(lambda) X^T by the parallel cyclic
//     Jacobi method: a sweep visits every index pair once in n-1 rounds of
//     n/2 disjoint pairs (round-robin order); per round one kernel computes
//     the n/2 rotations that zero C[p][q] and one applies them all at once,
//     C <- J^T C J (each thread owns a 2 x 2 block, so the update is in place)
//     and X <- X J.  Pairs with |C[p][q]| below 1e-14 trace(C)/n are skipped;
//     a sweep with no rotation ends the iteration.
//  4. sigma = sqrt(lambda) sorted descending; the top r_max eigenvectors are
//     gathered.  If X holds right vectors V: A = sqrt(sigma) V^T and
//     B = E V / sqrt(sigma) (= U sqrt(sigma)); if it holds left vectors U:
//     B = U sqrt(sigma) and A = U^T E / sqrt(sigma).
//  5. Sign fix on the U column, rounding to fp16 (one rounding from fp64).
//
// The Gram route squares the condition number: singular values far below
// sqrt(eps) * sigma_max carry absolute, not relative, accuracy.  The factors
// only use the leading ones.

#include "cl_device.h"
#include "cl_internal.h"

namespace cl {

namespace {

constexpr int kMaxSweeps = 40;
constexpr double kJacobiTol = 1e-14;

size_t up256(size_t n) { return (n + 255) / 256 * 256; }

struct CompLayout {
    size_t E, C, X, rot, lam, order, count, delta, sign, Xr, P, total;
};

CompLayout comp_layout(int d_out, int d_in, int r_max) {
    const size_t n = static_cast<size_t>(d_in <= d_out ? d_in : d_out);
    const size_t N = n + (n & 1);
    const size_t big = static_cast<size_t>(d_in > d_out ? d_in : d_out);
    CompLayout l;
    l.E = 0;
    l.C = l.E + up256(static_cast<size_t>(d_out) * d_in * 8);
    l.X = l.C + up256(n * n * 8);
    l.rot = l.X + up256(n * n * 8);
    l.lam = l.rot + up256(N / 2 * 2 * 8);
    l.order = l.lam + up256(n * 8);
    l.count = l.order + up256(n * 4);
    l.delta = l.count + up256(kMaxSweeps * 4);
    l.sign = l.delta + 256;
    l.Xr = l.sign + up256(static_cast<size_t>(r_max) * 8 + 8);
    l.P = l.Xr + up256(static_cast<size_t>(r_max) * n * 8 + 8);
    l.total = l.P + up256(static_cast<size_t>(r_max) * big * 8 + 8);
    return l;
}

__device__ __forceinline__ double h2d(uint16_t h) {
    return static_cast<double>(f16_bits_to_f32(h));
}

// E[o][c] = W[o][c] - s (q - z), one thread per element
__global__ __launch_bounds__(256) void residual_kernel(const float* __restrict__ W, QW w, double* __restrict__ E) {
    const size_t idx = static_cast<size_t>(blockIdx.x) * 256 + threadIdx.x;
    const size_t total = static_cast<size_t>(w.d_out) * w.d_in;
    if (idx >= total) return;
    const int o = static_cast<int>(idx / w.d_in);
    const int c = static_cast<int>(idx - static_cast<size_t>(o) * w.d_in);
    // code c: bits bits * c .. of the row's bit string (3-bit codes can
    // straddle two words)
    const uint32_t* row = w.q + static_cast<size_t>(o) * (static_cast<size_t>(w.d_in) * w.bits / 32);
    const int bp = w.bits * c;
    uint64_t two = row[bp >> 5];
    if ((bp & 31) + w.bits > 32) two |= static_cast<uint64_t>(row[(bp >> 5) + 1]) << 32;
    const uint32_t code = static_cast<uint32_t>(two >> (bp & 31)) & ((1u << w.bits) - 1u);
    const size_t gi = static_cast<size_t>(o) * (w.d_in / w.G) + c / w.G;
    const double what = h2d(w.s[gi]) * (static_cast<double>(code) - h2d(w.z[gi]));
    E[idx] = static_cast<double>(W[idx]) - what;
}

// out[i * ldo + j] = sum_k X[i * xi + k * xk] * Y[j * yj + k * yk]  (fp64)
// 64 x 64 output tile per 256-thread workgroup, 4 x 4 per thread, k in steps
// of 16 through LDS.  XK1 / YK1: the operand is contiguous along k (else along
// i / j), which decides the load order so that loads coalesce.
template <bool XK1, bool YK1>
__global__ __launch_bounds__(256) void gemm_nt_f64(const double* __restrict__ X, size_t xi, size_t xk,
                                                   const double* __restrict__ Y, size_t yj, size_t yk, int I, int J,
                                                   int K, double* __restrict__ out, size_t ldo) {
    constexpr int BT = 64, BK = 16;
    __shared__ double xs[BK][BT + 1];
    __shared__ double ys[BK][BT + 1];
    const int tid = threadIdx.x;
    const int tx = tid & 15, ty = tid >> 4;
    const int i0 = blockIdx.y * BT, j0 = blockIdx.x * BT;
    double acc[4][4] = {};
    for (int k0 = 0; k0 < K; k0 += BK) {
#pragma unroll
        for (int l = 0; l < 4; ++l) {
            const int e = tid + 256 * l;
            int ii, kk;
            if (XK1) { kk = e & (BK - 1); ii = e / BK; } else { ii = e & (BT - 1); kk = e / BT; }
            const int gi = i0 + ii, gk = k0 + kk;
            xs[kk][ii] = (gi < I && gk < K) ? X[gi * xi + gk * xk] : 0.0;
            int jj, kj;
            if (YK1) { kj = e & (BK - 1); jj = e / BK; } else { jj = e & (BT - 1); kj = e / BT; }
            const int gj = j0 + jj, gkj = k0 + kj;
            ys[kj][jj] = (gj < J && gkj < K) ? Y[gj * yj + gkj * yk] : 0.0;
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < BK; ++kk) {
            double a[4], b[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                a[u] = xs[kk][ty + 16 * u];
                b[u] = ys[kk][tx + 16 * u];
            }
#pragma unroll
            for (int u = 0; u < 4; ++u)
#pragma unroll
                for (int v = 0; v < 4; ++v) acc[u][v] = fma(a[u], b[v], acc[u][v]);
        }
        __syncthreads();
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const int gi = i0 + ty + 16 * u;
        if (gi >= I) continue;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int gj = j0 + tx + 16 * v;
            if (gj < J) out[gi * ldo + gj] = acc[u][v];
        }
    }
}

// X = identity, sweep counters zero, lam[i] = C[i][i]; workgroup 0 then
// derives the skip threshold from the trace.
__global__ __launch_bounds__(256) void jacobi_init_kernel(const double* __restrict__ C, double* __restrict__ Xm, int n,
                                                          int* __restrict__ count, double* __restrict__ delta) {
    const size_t idx = static_cast<size_t>(blockIdx.x) * 256 + threadIdx.x;
    const size_t nn = static_cast<size_t>(n) * n;
    if (idx < nn) Xm[idx] = (idx / n == idx % n) ? 1.0 : 0.0;
    if (blockIdx.x == 0) {
        __shared__ double part[256];
        if (threadIdx.x < kMaxSweeps) count[threadIdx.x] = 0;
        double t = 0.0;
        for (int i = threadIdx.x; i < n; i += 256) t += C[static_cast<size_t>(i) * n + i];
        part[threadIdx.x] = t;
        __syncthreads();
        for (int s = 128; s > 0; s >>= 1) {
            if (threadIdx.x < s) part[threadIdx.x] += part[threadIdx.x + s];
            __syncthreads();
        }
        if (threadIdx.x == 0) *delta = kJacobiTol * part[0] / n;
    }
}

// Round r of the round-robin order over N (even) indices: pair 0 is
// (r, N-1), pair i >= 1 is ((r + i) mod (N-1), (r - i) mod (N-1)).  Over
// r = 0..N-2 every unordered pair occurs exactly once; within a round the N/2
// pairs are disjoint.  Index N-1 == n (odd n) is a placeholder.
__device__ __forceinline__ void round_pair(int N, int r, int i, int& p, int& q) {
    const int M = N - 1;
    if (i == 0) { p = r; q = M; return; }
    p = (r + i) % M;
    q = (r - i + M) % M;
}

// One rotation per pair: zero C[p][q] with J = [[c, s], [-s, c]] on (p, q):
// tau = (C_qq - C_pp) / (2 C_pq), t the smaller root of t^2 + 2 tau t - 1 = 0,
// c = 1 / sqrt(1 + t^2), s = t c  (the symmetric Schur decomposition of the
// 2 x 2 block).
__global__ __launch_bounds__(256) void jacobi_rot_kernel(const double* __restrict__ C, int n, int N, int r,
                                                         const double* __restrict__ delta, double2* __restrict__ rot,
                                                         int* __restrict__ count) {
    const int i = blockIdx.x * 256 + threadIdx.x;
    bool did = false;
    if (i < N / 2) {
        int p, q;
        round_pair(N, r, i, p, q);
        double c = 1.0, s = 0.0;
        if (p < n && q < n) {
            const double apq = C[static_cast<size_t>(p) * n + q];
            if (fabs(apq) > *delta) {
                const double app = C[static_cast<size_t>(p) * n + p];
                const double aqq = C[static_cast<size_t>(q) * n + q];
                const double tau = (aqq - app) / (2.0 * apq);
                double t;
                if (fabs(tau) > 1e150) t = 0.5 / tau;
                else t = (tau >= 0.0 ? 1.0 : -1.0) / (fabs(tau) + sqrt(1.0 + tau * tau));
                c = 1.0 / sqrt(1.0 + t * t);
                s = t * c;
                did = s != 0.0;
            }
        }
        rot[i] = make_double2(c, s);
    }
    const unsigned long long b = __ballot(did);
    if ((threadIdx.x & 63) == 0 && b) atomicAdd(count, __popcll(b));
}

// Apply the round's rotations.  Rows blockIdx.y < N/2: the C blocks of row
// pair a = blockIdx.y with column pairs b = thread index,
// C_ab <- J_a^T C_ab J_b.  Rows beyond: row i of X, columns of pair b,
// X_b <- X_b J_b.  Blocks whose two rotations are the identity are left alone.
__global__ __launch_bounds__(256) void jacobi_apply_kernel(double* __restrict__ C, double* __restrict__ Xm, int n,
                                                           int N, int r, const double2* __restrict__ rot) {
    const int b = blockIdx.x * 256 + threadIdx.x;
    const int half = N / 2;
    if (b >= half) return;
    int pb, qb;
    round_pair(N, r, b, pb, qb);
    const double2 jb = rot[b];
    const bool vpb = pb < n, vqb = qb < n;
    if (static_cast<int>(blockIdx.y) < half) {
        const int a = blockIdx.y;
        const double2 ja = rot[a];
        if (ja.y == 0.0 && jb.y == 0.0) return;
        int pa, qa;
        round_pair(N, r, a, pa, qa);
        const bool vpa = pa < n, vqa = qa < n;
        const size_t rp = static_cast<size_t>(pa) * n, rq = static_cast<size_t>(qa) * n;
        const double x00 = (vpa && vpb) ? C[rp + pb] : 0.0;
        const double x01 = (vpa && vqb) ? C[rp + qb] : 0.0;
        const double x10 = (vqa && vpb) ? C[rq + pb] : 0.0;
        const double x11 = (vqa && vqb) ? C[rq + qb] : 0.0;
        // (C J_b): columns p, q
        const double y00 = jb.x * x00 - jb.y * x01, y01 = jb.y * x00 + jb.x * x01;
        const double y10 = jb.x * x10 - jb.y * x11, y11 = jb.y * x10 + jb.x * x11;
        // J_a^T (C J_b): rows p, q
        double z00 = ja.x * y00 - ja.y * y10, z01 = ja.x * y01 - ja.y * y11;
        double z10 = ja.y * y00 + ja.x * y10, z11 = ja.y * y01 + ja.x * y11;
        if (a == b && ja.y != 0.0) { z01 = 0.0; z10 = 0.0; }   // the entry the rotation annihilates
        if (vpa && vpb) C[rp + pb] = z00;
        if (vpa && vqb) C[rp + qb] = z01;
        if (vqa && vpb) C[rq + pb] = z10;
        if (vqa && vqb) C[rq + qb] = z11;
    } else {
        if (jb.y == 0.0) return;
        const size_t row = static_cast<size_t>(blockIdx.y - half) * n;
        const double x0 = vpb ? Xm[row + pb] : 0.0;
        const double x1 = vqb ? Xm[row + qb] : 0.0;
        if (vpb) Xm[row + pb] = jb.x * x0 - jb.y * x1;
        if (vqb) Xm[row + qb] = jb.y * x0 + jb.x * x1;
    }
}

// Descending order of the eigenvalues (ties by index); sigma = sqrt(max(0,
// lambda)) in that order.
__global__ __launch_bounds__(256) void eig_sort_kernel(const double* __restrict__ C, int n, double* __restrict__ lam,
                                                       int* __restrict__ order, float* __restrict__ sigma) {
    const int i = blockIdx.x * 256 + threadIdx.x;
    if (i >= n) return;
    const double li = C[static_cast<size_t>(i) * n + i];
    int rank = 0;
    for (int j = 0; j < n; ++j) {
        const double lj = C[static_cast<size_t>(j) * n + j];
        rank += (lj > li) || (lj == li && j < i);
    }
    order[rank] = i;
    lam[rank] = li;
    if (sigma) sigma[rank] = static_cast<float>(sqrt(li > 0.0 ? li : 0.0));
}

// Xr[j][i] = X[i][order[j]] for the leading r_max eigenvectors.
__global__ __launch_bounds__(256) void gather_kernel(const double* __restrict__ Xm, int n, const int* __restrict__ order,
                                                     int r_max, double* __restrict__ Xr) {
    const size_t idx = static_cast<size_t>(blockIdx.x) * 256 + threadIdx.x;
    if (idx >= static_cast<size_t>(r_max) * n) return;
    const int j = static_cast<int>(idx / n), i = static_cast<int>(idx % n);
    Xr[idx] = Xm[static_cast<size_t>(i) * n + order[j]];
}

// sign[j] = +-1 so that the largest-magnitude entry (first index on ties) of
// U column j, u[i * stride + j * jstride] for i < len, becomes positive.
__global__ __launch_bounds__(256) void sign_kernel(const double* __restrict__ u, size_t stride, size_t jstride, int len,
                                                   double* __restrict__ sign) {
    __shared__ double bv[256];
    __shared__ int bi[256];
    const int j = blockIdx.x;
    double best = -1.0, val = 0.0;
    int bidx = 0x7fffffff;
    for (int i = threadIdx.x; i < len; i += 256) {
        const double x = u[i * stride + j * jstride];
        if (fabs(x) > best) { best = fabs(x); bidx = i; val = x; }
    }
    bv[threadIdx.x] = best;
    bi[threadIdx.x] = bidx;
    __shared__ double vv[256];
    vv[threadIdx.x] = val;
    __syncthreads();
    for (int s = 128; s > 0; s >>= 1) {
        if (threadIdx.x < s) {
            const double o = bv[threadIdx.x + s];
            const int oi = bi[threadIdx.x + s];
            if (o > bv[threadIdx.x] || (o == bv[threadIdx.x] && oi < bi[threadIdx.x])) {
                bv[threadIdx.x] = o;
                bi[threadIdx.x] = oi;
                vv[threadIdx.x] = vv[threadIdx.x + s];
            }
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) sign[j] = vv[0] < 0.0 ? -1.0 : 1.0;
}

// fp16 factors.  right: X held right vectors (Xr = V^T rows, P = E V);
// otherwise left vectors (Xr = U^T rows, P = U^T E).
__global__ __launch_bounds__(256) void factor_a_kernel(const double* __restrict__ Xr, const double* __restrict__ P,
                                                       const double* __restrict__ lam, const double* __restrict__ sign,
                                                       int r_max, int d_in, bool right, uint16_t* __restrict__ A) {
    const size_t idx = static_cast<size_t>(blockIdx.x) * 256 + threadIdx.x;
    if (idx >= static_cast<size_t>(r_max) * d_in) return;
    const int j = static_cast<int>(idx / d_in);
    const double sg = sqrt(lam[j] > 0.0 ? lam[j] : 0.0);
    const double root = sqrt(sg);
    double v;
    if (right) v = root * Xr[idx];
    else v = sg > 0.0 ? P[idx] / root : 0.0;
    A[idx] = f64_to_f16_rne(sign[j] * v);
}

__global__ __launch_bounds__(256) void factor_b_kernel(const double* __restrict__ Xr, const double* __restrict__ P,
                                                       const double* __restrict__ lam, const double* __restrict__ sign,
                                                       int r_max, int d_out, bool right, uint16_t* __restrict__ B) {
    const size_t idx = static_cast<size_t>(blockIdx.x) * 256 + threadIdx.x;
    if (idx >= static_cast<size_t>(d_out) * r_max) return;
    const int o = static_cast<int>(idx / r_max), j = static_cast<int>(idx % r_max);
    const double sg = sqrt(lam[j] > 0.0 ? lam[j] : 0.0);
    const double root = sqrt(sg);
    double v;
    if (right) v = sg > 0.0 ? P[idx] / root : 0.0;                 // P is [d_out][r_max]
    else v = root * Xr[static_cast<size_t>(j) * d_out + o];
    B[idx] = f64_to_f16_rne(sign[j] * v);
}

unsigned grid1(size_t n) { return static_cast<unsigned>((n + 255) / 256); }

template <bool XK1, bool YK1>
void gemm(const double* X, size_t xi, size_t xk, const double* Y, size_t yj, size_t yk, int I, int J, int K,
          double* out, size_t ldo, hipStream_t st) {
    dim3 grid((J + 63) / 64, (I + 63) / 64);
    hipLaunchKernelGGL((gemm_nt_f64<XK1, YK1>), grid, dim3(256), 0, st, X, xi, xk, Y, yj, yk, I, J, K, out, ldo);
}

}  // namespace

bool comp_fits(int d_out, int d_in) {
    const int n = d_in <= d_out ? d_in : d_out;
    return n <= 8192 && static_cast<long long>(d_out) * d_in <= (1ll << 31);
}

size_t comp_workspace_bytes(int d_out, int d_in, int r_max) {
    return comp_layout(d_out, d_in, r_max).total;
}

hipError_t launch_build_compensation(const float* W, const QW& w, int r_max, uint16_t* A, uint16_t* B, float* sigma,
                                     void* ws, hipStream_t st, int* sweeps_out) {
    const int d_out = w.d_out, d_in = w.d_in;
    const bool right = d_in <= d_out;              // Gram over d_in: eigenvectors are V
    const int n = right ? d_in : d_out;
    const int N = n + (n & 1);
    const CompLayout l = comp_layout(d_out, d_in, r_max);
    char* b = static_cast<char*>(ws);
    double* E = reinterpret_cast<double*>(b + l.E);
    double* C = reinterpret_cast<double*>(b + l.C);
    double* Xm = reinterpret_cast<double*>(b + l.X);
    double2* rot = reinterpret_cast<double2*>(b + l.rot);
    double* lam = reinterpret_cast<double*>(b + l.lam);
    int* order = reinterpret_cast<int*>(b + l.order);
    int* count = reinterpret_cast<int*>(b + l.count);
    double* delta = reinterpret_cast<double*>(b + l.delta);
    double* sign = reinterpret_cast<double*>(b + l.sign);
    double* Xr = reinterpret_cast<double*>(b + l.Xr);
    double* P = reinterpret_cast<double*>(b + l.P);
    hipError_t e;

    const size_t total = static_cast<size_t>(d_out) * d_in;
    hipLaunchKernelGGL(residual_kernel, dim3(grid1(total)), dim3(256), 0, st, W, w, E);
    // Gram: C[i][j] = sum_k E_k,i E_k,j over the larger side
    if (right) gemm<false, false>(E, 1, d_in, E, 1, d_in, n, n, d_out, C, n, st);
    else gemm<true, true>(E, d_in, 1, E, d_in, 1, n, n, d_in, C, n, st);
    hipLaunchKernelGGL(jacobi_init_kernel, dim3(grid1(static_cast<size_t>(n) * n)), dim3(256), 0, st, C, Xm, n, count,
                       delta);
    if ((e = hipGetLastError()) != hipSuccess) return e;

    int sweeps = 0;
    for (; sweeps < kMaxSweeps; ++sweeps) {
        for (int r = 0; r < N - 1; ++r) {
            hipLaunchKernelGGL(jacobi_rot_kernel, dim3(grid1(N / 2)), dim3(256), 0, st, C, n, N, r, delta, rot,
                               count + sweeps);
            hipLaunchKernelGGL(jacobi_apply_kernel, dim3(grid1(N / 2), N / 2 + n), dim3(256), 0, st, C, Xm, n, N, r,
                               rot);
        }
        if ((e = hipGetLastError()) != hipSuccess) return e;
        int rotations = 0;
        if ((e = hipMemcpyAsync(&rotations, count + sweeps, sizeof(int), hipMemcpyDeviceToHost, st)) != hipSuccess)
            return e;
        if ((e = hipStreamSynchronize(st)) != hipSuccess) return e;
        if (rotations == 0) break;
    }
    if (sweeps_out) *sweeps_out = sweeps;
    if (sweeps == kMaxSweeps) return hipErrorNotReady;       // did not converge (reported by the caller)

    hipLaunchKernelGGL(eig_sort_kernel, dim3(grid1(n)), dim3(256), 0, st, C, n, lam, order, sigma);
    if (r_max > 0) {
        hipLaunchKernelGGL(gather_kernel, dim3(grid1(static_cast<size_t>(r_max) * n)), dim3(256), 0, st, Xm, n,
                           order, r_max, Xr);
        if (right) {
            // P[o][j] = sum_c E[o][c] V[c][j]
            gemm<true, true>(E, d_in, 1, Xr, d_in, 1, d_out, r_max, d_in, P, r_max, st);
            hipLaunchKernelGGL(sign_kernel, dim3(r_max), dim3(256), 0, st, P, static_cast<size_t>(r_max),
                               static_cast<size_t>(1), d_out, sign);
        } else {
            // P[j][c] = sum_o U[o][j] E[o][c]
            gemm<true, false>(Xr, d_out, 1, E, 1, d_in, r_max, d_in, d_out, P, d_in, st);
            hipLaunchKernelGGL(sign_kernel, dim3(r_max), dim3(256), 0, st, Xr, static_cast<size_t>(1),
                               static_cast<size_t>(d_out), d_out, sign);
        }
        hipLaunchKernelGGL(factor_a_kernel, dim3(grid1(static_cast<size_t>(r_max) * d_in)), dim3(256), 0, st, Xr, P,
                           lam, sign, r_max, d_in, right, A);
        hipLaunchKernelGGL(factor_b_kernel, dim3(grid1(static_cast<size_t>(d_out) * r_max)), dim3(256), 0, st, Xr, P,
                           lam, sign, r_max, d_out, right, B);
    }
    return hipGetLastError();
}

}  // namespace cl
