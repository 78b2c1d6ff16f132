// Expert-gathered compensated linear for a MoE layer (decode):
//
//     y[t][j] = deq(Q_e) x + B_e[:, :r_e] (A_e[:r_e] x),   e = ids[t][j]
//
// with x = x[t] (shared by a token's slots, e.g. gate/up) or x[t][j] (the
// slot's own input, e.g. down).  The paper regroups the same projection of
// all activated experts into one step (Section 4.2.2, Cross-Expert Pipeline
// Reorganization; Appendix A.1, MoE Layer); here that is one pair of launches
// over every routed expert, and only routed experts' codes, scales, zeros and
// factors are read.
//
// A call covers a window of up to 4 linears over the same routing and input
// (e.g. a layer's gate and up); a single linear is the window of one.
//
//  * moe_prep_kernel: workgroup (linear, j, q), j < min(E, T*k), reads the
//    routing table -- so no workgroup ever waits for another -- counts slots
//    per expert, scans the counts and takes e = the j-th routed expert in
//    ascending id order (none: it exits).  Each of its four waves computes
//    t[slot][i] = A_e[i] . x_slot for one rank row i = 4q + wave of its
//    linear over all of e's slots (four slots per pass).  Workgroup
//    (0, j, 0) also writes entry j of the active-expert table and e's slots,
//    in slot order, into the sorted slot list, and (linear, j, 0) that
//    linear's rank of e; workgroups (linear, 0, 0) write the number of
//    routed experts and zero rows for slots whose id is out of range.  The
//    remaining workgroups prepare the activations (fp16, pair-permuted,
//    per-chunk sums) exactly as the dense decode does.
//  * moe_kernel: one workgroup per (linear, active expert, row batch); the
//    grid is sized for the most experts T*k slots can reach and surplus
//    workgroups exit on the device-side count.  Each wave loads its slice
//    (4 rows for 4-bit codes, 2 for 2-bit, per row set of LG lanes; one
//    16-byte chunk per lane) of the expert's backbone and factor entries
//    once and applies it to every slot routed to that expert.  Same
//    arithmetic as the dense decode kernel: mask-only unpack into subnormal
//    fp16 lanes, v_dot2, per-chunk scale and zero in fp32, B t in the same
//    partial sums, transposing butterfly, fixed-order K-slice reduction.
//  * moe_mfma_kernel: with several slots per expert (4-bit codes), the
//    expert's rows against its slots on MFMA (slots as the columns).

#include "cl_device.h"
#include "cl_internal.h"
#include "gemv_common.h"
#include "mfma_common.h"

namespace cl {

// Routing-error record of this device: zero, or bit 63 set with the slot
// (bits 32..62) and the id (bits 0..31) of an out-of-range routing entry seen
// by a MoE call since the record was last read.  Each device holds its own
// copy for the life of the process.
__device__ unsigned long long moe_routing_error;

namespace {

// rows per wave batch: 4 for 4-bit codes, 2 for 2-bit (twice the
// activation registers per chunk)
constexpr int rows_per_wave(int bits) { return bits == 4 ? 4 : 2; }
constexpr int kMaxSlots = 1024;      // T * k
constexpr int kMaxExperts = 1024;
constexpr int kTab = 8;              // ints per active-expert table entry
constexpr int kMaxMoeWin = 4;        // linears per window
// Direct path (moe_direct_kernel): at most this many slots; row batches per
// wave counted for 4 waves of 4 rows per row set of LG lanes (64 rows per
// workgroup, 32 with two chunks per lane; the launch splits them over 8
// waves)
constexpr int kDirectMaxSlots = 8;
constexpr int direct_batches(int lg, int cpl) { return cpl == 2 ? 2 : (lg == 64 ? 4 : 2); }
// MFMA path: 16-row tiles per workgroup and K blocks in flight per wave.
// Measured on the 48-layer T = 64 step with the workgroup's loads issued in
// need order (scales and zeros, slot ids, code blocks): 8 x 1 166 us per
// layer, 4 x 2 191, 8 x 2 229, 12 x 1 230, 16 x 1 227 (with the code loads
// issued after the scale/zero copy: 4 x 2 213 us; one tile of 16 rows had
// taken 389, every workgroup re-reading its slots' activations).  Once the
// pipeline's tail stopped re-reading code blocks: 4 x 1 143.7 us, 8 x 1
// 150.5, 2 x 1 153.0, 6 x 1 161.7, 4 x 2 ~160 (165 VGPRs at 4 x 1: three
// waves per SIMD against two).
constexpr int kMoeTpw = 4;
constexpr int kMoeNbuf = 1;

// One linear of a window: its stacked experts and its share of the grids.
struct MoeLin {
    const uint32_t* q;
    const uint16_t* s;
    const uint16_t* z;
    const uint16_t* A;
    const uint16_t* B;
    const int32_t* ranks;
    const int32_t* slot_rank;  // [T*k] per-slot ranks (clamped to 0..r_max), or null: ranks[e]
    void* y;
    float* t;                // [T*k][r_max] (workspace)
    size_t q_stride, sz_stride, a_stride, b_stride;   // elements per expert
    int d_out, r_max;
    int rq;                  // preparation workgroups per expert (4 rank rows each)
    int bpe;                 // backbone batches per expert
    int prep_end;            // rank workgroups of linears 0 .. this one (prefix sum)
    int blk_end;             // backbone workgroups of linears 0 .. this one (prefix sum)
    int nrb;                 // direct path: row blocks per slot
};

// A window of n linears over the same routing and activations (one linear
// is the window n = 1).
struct MoeArgs {
    MoeLin lin[kMaxMoeWin];
    int n;
    const int32_t* ids;
    const uint16_t* x;
    const uint16_t* u;       // gated input: the activations are SiLU(x) u elementwise (null: x)
    int E, T, k, d_in, G, act, out, x_per_slot;
    // workspace
    int* n_active;
    int* table;              // [max_active][kTab]: expert, first sorted index, slot count, first slot,
                             // then each linear's rank
    int* sorted;             // [T*k] slot ids grouped by expert, slot order within
    f16x2* xp;               // [rows][d_in/2]
    float* sx;               // [rows][chunks]
    int ks, cps;             // K slices, chunks per slice
    int rb;                  // direct path: rows per workgroup
    int nrbm;                // direct path: row blocks per (linear, slot) unit (the largest linear's)
};

template <int BITS>
__global__ __launch_bounds__(256) void moe_prep_kernel(MoeArgs a) {
    constexpr int CPW = 32 / BITS, HPW = CPW / 2, PPC = 4 * HPW;
    // sids[S], mys[S] (this expert's slots, in slot order), hist[E] (slots
    // per expert), rk[E] (the experts' ranks): sized by the call, so more
    // workgroups fit a CU
    extern __shared__ int prep_lds[];
    __shared__ int wsum[4][2];
    __shared__ int wcnt[4];
    __shared__ int sel, sel_lt, sel_n, srank;
    __shared__ u32x4 xsh[4][256];          // a pass's activations, 4 slots x 2048 columns
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int S = a.T * a.k;
    const int blk = blockIdx.x;
    int* const sids = prep_lds;
    int* const mys = sids + S;
    int* const hist = mys + S;
    int* const rk = hist + a.E;

    if (blk < a.lin[a.n - 1].prep_end) {
        // workgroup (linear li, j, quad): the j-th routed expert (ascending
        // id), its rank rows 4 quad .. 4 quad + 3 of linear li; every
        // workgroup derives the routing itself
        int li = 0;
        while (blk >= a.lin[li].prep_end) ++li;
        const MoeLin& L = a.lin[li];
        const int local = blk - (li ? a.lin[li - 1].prep_end : 0);
        const int j = local / L.rq;
        const int quad = local - j * L.rq;
        // The experts' ranks, the routing ids and the per-slot ranks are
        // loaded in one round trip: every load is unconditional (clamped
        // index, out-of-range values replaced afterwards), so none waits at
        // a branch for the ones before it.  The histogram is cleared
        // meanwhile.
        for (int i = tid; i < a.E; i += 256) hist[i] = 0;
        if (tid == 0) sel = -1;
        constexpr int kPer = kMaxExperts / 256;       // experts and slots per thread, at most
        const bool dyn = L.slot_rank != nullptr;
        const int32_t* rsrc = L.r_max > 0 ? L.ranks : a.ids;    // ranks may be null when r_max is 0
        const int32_t* ssrc = dyn ? L.slot_rank : a.ids;
        int rkv[kPer], idv[kPer], srv[kPer];
#pragma unroll
        for (int u = 0; u < kPer; ++u) {
            const int i = tid + 256 * u;
            rkv[u] = rsrc[min(i, a.E - 1)];
            idv[u] = a.ids[min(i, S - 1)];
            srv[u] = ssrc[min(i, S - 1)];
        }
        __syncthreads();
#pragma unroll
        for (int u = 0; u < kPer; ++u) {
            const int i = tid + 256 * u;
            if (i < a.E) rk[i] = L.r_max > 0 ? rkv[u] : 0;
            if (i < S) {
                sids[i] = idv[u];
                if (idv[u] >= 0 && idv[u] < a.E) atomicAdd(&hist[idv[u]], 1);
            }
        }
        __syncthreads();
        // block scan over the experts (thread t owns experts 4 t .. 4 t + 3):
        // the first sorted slot of each expert and its index among the
        // routed experts; expert e with index j is this workgroup's
        int c[4], cs = 0, fs = 0;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int ex = 4 * tid + q;
            c[q] = ex < a.E ? hist[ex] : 0;
            cs += c[q];
            fs += c[q] > 0;
        }
        int ic = cs, ifl = fs;                   // inclusive scan within the wave
        for (int off = 1; off < 64; off <<= 1) {
            const int tc = __shfl_up(ic, off, 64), tf = __shfl_up(ifl, off, 64);
            if (lane >= off) { ic += tc; ifl += tf; }
        }
        if (lane == 63) { wsum[wave][0] = ic; wsum[wave][1] = ifl; }
        __syncthreads();
        int pc = ic - cs, pf = ifl - fs;
        for (int w2 = 0; w2 < wave; ++w2) { pc += wsum[w2][0]; pf += wsum[w2][1]; }
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            if (c[q] > 0) {
                if (pf == j) { sel = 4 * tid + q; sel_lt = pc; sel_n = c[q]; }
                pc += c[q];
                pf += 1;
            }
        }
        if (li == 0 && j == 0 && quad == 0 && tid == 0)
            *a.n_active = wsum[0][1] + wsum[1][1] + wsum[2][1] + wsum[3][1];
        __syncthreads();
        if (j == 0 && quad == 0) {
            // out-of-range ids: their output rows are zero.  One parallel
            // check first (valid routing skips the rest), then each wave
            // zeroes the rows of its share of the slots.
            int bad = 0;
            for (int sl = tid; sl < S; sl += 256) bad |= !(sids[sl] >= 0 && sids[sl] < a.E);
            if (__syncthreads_or(bad)) {
                for (int sl = wave; sl < S; sl += 4) {
                    const int id = sids[sl];
                    if (id >= 0 && id < a.E) continue;
                    // the device's routing-error record (reported by
                    // cl_moe_status): a flag bit, the slot and the id
                    if (li == 0 && lane == 0)
                        __hip_atomic_store(&moe_routing_error,
                                           (1ull << 63) | (static_cast<unsigned long long>(sl) << 32) |
                                               static_cast<uint32_t>(id),
                                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    for (int o = lane; o < L.d_out; o += 64)
                        store_out(L.y, static_cast<size_t>(sl) * L.d_out + o, 0.f, a.out);
                }
            }
        }
        const int e = sel;
        if (e < 0) return;                      // fewer than j + 1 routed experts
        const int ne = sel_n, cnt_lt = sel_lt;
        int rank = rk[e];
        rank = rank < 0 ? 0 : (rank > L.r_max ? L.r_max : rank);
        // per-slot ranks: the expert's rank here is the largest of its slots'
        // (A_e x is computed that far; each slot reads its own prefix)
        if (dyn && tid == 0) srank = 0;
        // this expert's slots in slot order (ballots, 256 slots per pass)
        int base_pos = 0;
#pragma unroll
        for (int u = 0; u < kPer; ++u) {
            if (256 * u >= S) break;
            const int sl = 256 * u + tid;
            const bool mine = sl < S && sids[sl] == e;
            const unsigned long long m = __ballot(mine);
            if (lane == 0) wcnt[wave] = __popcll(m);
            __syncthreads();
            int off = base_pos;
            for (int w2 = 0; w2 < wave; ++w2) off += wcnt[w2];
            if (mine) {
                const int pos = off + __popcll(m & ((1ull << lane) - 1ull));
                if (li == 0 && quad == 0) {
                    a.sorted[cnt_lt + pos] = sl;
                    if (pos == 0) a.table[kTab * j + 3] = sl;
                }
                mys[pos] = sl;
                if (dyn) {
                    const int rs = srv[u];
                    atomicMax(&srank, rs < 0 ? 0 : (rs > L.r_max ? L.r_max : rs));
                }
            }
            base_pos += wcnt[0] + wcnt[1] + wcnt[2] + wcnt[3];
            __syncthreads();
        }
        if (dyn) rank = srank;
        if (quad == 0 && tid == 0) {
            if (li == 0) {
                a.table[kTab * j + 0] = e;
                a.table[kTab * j + 1] = cnt_lt;
                a.table[kTab * j + 2] = ne;
            }
            a.table[kTab * j + 4 + li] = rank;
        }
        // t[slot][i] = A_e[i] . x_slot: wave w takes rank row i = 4 quad + w;
        // each pass's activations (4 slots x 2048 columns) go into LDS once
        // for the workgroup's four waves
        const int i = 4 * quad + wave;
        if (4 * quad >= rank) return;
        const bool has = i < rank;
        const uint16_t* ar = L.A + static_cast<size_t>(e) * L.a_stride + static_cast<size_t>(has ? i : 4 * quad) * a.d_in;
        for (int j0 = 0; j0 < ne; j0 += 4) {
            const uint16_t* xr[4];
            int sl4[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                sl4[u] = mys[j0 + u < ne ? j0 + u : j0];
                const int xrow = a.x_per_slot ? sl4[u] : sl4[u] / a.k;
                xr[u] = a.x + static_cast<size_t>(xrow) * a.d_in;
            }
            float acc[4] = {0.f, 0.f, 0.f, 0.f};
            for (int c0 = 0; c0 < a.d_in; c0 += 4 * 512) {
                u32x4 av[4], xl[4];
                const int cx = c0 + 8 * tid;
#pragma unroll
                for (int u = 0; u < 4; ++u) xl[u] = *reinterpret_cast<const u32x4*>(xr[u] + (cx < a.d_in ? cx : 0));
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int c = c0 + 512 * q + 8 * lane;
                    av[q] = *reinterpret_cast<const u32x4*>(ar + (c < a.d_in ? c : 0));
                }
                __syncthreads();                 // the previous pass's reads are done
#pragma unroll
                for (int u = 0; u < 4; ++u)
                    xsh[u][tid] = cx < a.d_in ? act8_to_f16(xl[u], a.act) : u32x4{0u, 0u, 0u, 0u};
                __syncthreads();
                if (has) {
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
#pragma unroll
                        for (int u = 0; u < 4; ++u) {
                            const u32x4 xw = xsh[u][64 * q + lane];
                            float d = 0.f;
#pragma unroll
                            for (int h = 0; h < 4; ++h) {
                                const uint32_t ae = av[q][h], xe = xw[h];
                                d = dot2(__builtin_bit_cast(f16x2, ae), __builtin_bit_cast(f16x2, xe), d);
                            }
                            acc[u] += d;
                        }
                    }
                }
            }
            if (has) {
                const float tot = wave_sum_multi<4>(acc);      // lane l: slot j0 + l / 16
                const int u = lane >> 4;
                if ((lane & 15) == 0 && j0 + u < ne) L.t[static_cast<size_t>(sl4[u]) * L.r_max + i] = tot;
            }
        }
        return;
    }
    // activation preparation, one thread per (row, chunk)
    const int rows = a.x_per_slot ? S : a.T;
    const int chunks = a.d_in / CPW / 4;
    const long long item = static_cast<long long>(blk - a.lin[a.n - 1].prep_end) * 256 + tid;
    if (item >= static_cast<long long>(rows) * chunks) return;
    const int row = static_cast<int>(item / chunks);
    const int c = static_cast<int>(item % chunks);
    f16x2 v[PPC];
    load_chunk_x<BITS>(a.x + static_cast<size_t>(row) * a.d_in, c, a.act, v);
    const f16x2 one = {static_cast<f16>(1.0f), static_cast<f16>(1.0f)};
    float sum = 0.f;
    f16x2* dst = a.xp + static_cast<size_t>(row) * (a.d_in / 2) + static_cast<size_t>(c) * PPC;
#pragma unroll
    for (int p = 0; p < PPC; ++p) {
        sum = dot2(v[p], one, sum);
        dst[p] = v[p];
    }
    a.sx[static_cast<size_t>(row) * chunks + c] = sum;
}

// NB: factor columns per lane (r_max <= NB * 64 * ks); 0 when r_max is 0.
// HOIST: unpack the codes once into fp16 lanes held in registers (for
// experts that meet several slots); otherwise unpack per slot.
// Sum R values over each group of LG consecutive lanes (LG = 16, 32 or 64,
// a power of two >= R, R <= 16) with a transposing butterfly; on return lane
// l holds the total of value index (l % LG) / (LG / R) of its group.
template <int R, int LG>
__device__ __forceinline__ float group_sum_multi(float (&v)[R]) {
    const int lane = threadIdx.x & 63;
    float a[R];
#pragma unroll
    for (int i = 0; i < R; ++i) a[i] = v[i];
    int n = R;
    int bit = LG / 2;
#pragma unroll
    for (int step = 0; step < 4; ++step) {
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

// Without the hoisted unpack the kernel keeps no next-slot prefetch (it
// cost 19 VGPRs) and the 4-bit, one-factor-column instance is held to 128
// VGPRs (4 waves per SIMD): measured on MI355X, the 48-layer T = 1 and
// T = 8 steps went from 39.3 and 102.9 us to 37.3 and 94.1 us.  The
// 64-lane instance then keeps one register in scratch (one store and one
// load per wave); held to 168 VGPRs instead (3 waves per SIMD) it has none,
// but the T = 8 step takes 79.7 us against 75.1.
//
// LG: lanes per row set.  Rows of at least 64 chunks use the whole wave
// (LG = 64); shorter rows (the 768-wide down projection: 24 chunks) give
// each group of LG = 32 or 16 lanes its own R rows, so a wave covers
// 64 / LG row sets and fewer lanes idle (24 of 64 lanes were busy).
template <int BITS, int CPL, int NB, bool HOIST, int LG>
__global__ __launch_bounds__(512)
__attribute__((amdgpu_waves_per_eu(!HOIST && BITS == 4 && NB <= 1 ? 4 : 1)))
void moe_kernel(MoeArgs a) {
    constexpr int R = rows_per_wave(BITS);
    constexpr int CPW = 32 / BITS;
    constexpr int HPW = CPW / 2;
    constexpr int CPC = 4 * CPW;
    constexpr int PPC = 4 * HPW;
    constexpr int NACC = BITS == 4 ? 2 : 4;
    constexpr int NBA = NB > 0 ? NB : 1;
    __shared__ float red[8][R];

    // the active-expert count and this entry are read together (the entry
    // exists for every ae below min(E, T k); it is used only if ae is active)
    // workgroup -> (linear li, active expert ae, row batch)
    const int blk = blockIdx.x;
    int li = 0;
    while (blk >= a.lin[li].blk_end) ++li;
    const MoeLin& L = a.lin[li];
    const int local = blk - (li ? a.lin[li - 1].blk_end : 0);
    const int ae = local / L.bpe;
    const int n_active = *a.n_active;
    const int* ent = a.table + kTab * ae;
    const int e = ent[0], sbeg = ent[1], scnt = ent[2], slot0 = ent[3], rank = ent[4 + li];
    if (ae >= n_active) return;                     // whole workgroup: no routed expert here
    const int batch = local - ae * L.bpe;

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int waves = blockDim.x >> 6;
    const int ks = a.ks;
    const int rg_per_block = waves / ks;
    const int slice = wave % ks;
    const int rgw = wave / ks;
    const int words = a.d_in / CPW;
    const int chunks = words / 4;
    const int groups = a.d_in / a.G;
    const int c_begin = slice * a.cps;
    const int c_end = min(chunks, c_begin + a.cps);
    constexpr int SETS = 64 / LG;                  // row sets per wave
    const int lg = lane % LG;                      // lane within its row set
    const int row0 = ((batch * rg_per_block + rgw) * SETS + lane / LG) * R;
    const bool active = row0 < L.d_out;
    const int base = active ? row0 : 0;
    const int nrows = active ? min(R, L.d_out - row0) : 1;

    int cidx[CPL];
    float cmask[CPL];
#pragma unroll
    for (int j = 0; j < CPL; ++j) {
        cidx[j] = c_begin + lg + LG * j;
        const bool valid = cidx[j] < c_end;
        cmask[j] = valid ? 1.f : 0.f;
        if (!valid) cidx[j] = c_begin;
    }

    // this expert's rows: codes, scales, zeros, factor entries (loaded once)
    const uint32_t* qe = L.q + static_cast<size_t>(e) * L.q_stride;
    const uint16_t* se = L.s + static_cast<size_t>(e) * L.sz_stride;
    const uint16_t* ze = L.z + static_cast<size_t>(e) * L.sz_stride;
    u32x4 qv[R][CPL];
    float sc[R][CPL], zc[R][CPL];
    float bv[R][NBA];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int row = base + (r < nrows ? r : 0);
        const u32x4* qr = reinterpret_cast<const u32x4*>(qe + static_cast<size_t>(row) * words);
#pragma unroll
        for (int j = 0; j < CPL; ++j) {
            qv[r][j] = __builtin_nontemporal_load(qr + cidx[j]);
            const size_t gi = static_cast<size_t>(row) * groups + (cidx[j] * CPC) / a.G;
            sc[r][j] = f16_bits_to_f32(se[gi]) * cmask[j];
            zc[r][j] = f16_bits_to_f32(ze[gi]);
        }
#pragma unroll
        for (int m = 0; m < NB; ++m) {
            const int i = lg + LG * (slice + ks * m);
            const uint16_t* Be = L.B + static_cast<size_t>(e) * L.b_stride;
            bv[r][m] = i < rank ? f16_bits_to_f32(Be[static_cast<size_t>(row) * L.r_max + i]) : 0.f;
        }
    }

    // The expert's slot ids, 64 at a time in the lanes (read back with a
    // shuffle); with the hoisted unpack each slot's activations are loaded
    // one slot ahead, otherwise at the slot itself.
    auto load_x = [&](int sl, f16x2 (&xv)[PPC], float& sxv, float (&tv)[NBA]) {
        const int xrow = a.x_per_slot ? sl : sl / a.k;
        // this slot's rank: its own (per-slot ranks) or the expert's
        int rs = rank;
        if (L.slot_rank) {
            const int v = L.slot_rank[sl];
            rs = v < 0 ? 0 : (v > L.r_max ? L.r_max : v);
        }
        const u32x4* src = reinterpret_cast<const u32x4*>(a.xp + static_cast<size_t>(xrow) * (a.d_in / 2) +
                                                          static_cast<size_t>(cidx[0]) * PPC);
#pragma unroll
        for (int p4 = 0; p4 < PPC / 4; ++p4) {
            const u32x4 u = src[p4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const uint32_t uq = u[q];
                xv[4 * p4 + q] = __builtin_bit_cast(f16x2, uq);
            }
        }
        sxv = a.sx[static_cast<size_t>(xrow) * chunks + cidx[0]];
#pragma unroll
        for (int m = 0; m < NB; ++m) {
            const int i = lg + LG * (slice + ks * m);
            tv[m] = i < rs ? L.t[static_cast<size_t>(sl) * L.r_max + i] : 0.f;
        }
    };
    // the unpacked codes (HOIST), from the raw loads above
    constexpr int UPW = BITS == 4 ? 4 : 8;       // fp16 pairs per word
    f16x2 un[HOIST ? R : 1][HOIST ? 4 * UPW : 1];
    if constexpr (HOIST) {
#pragma unroll
        for (int rr0 = 0; rr0 < R; ++rr0)
#pragma unroll
            for (int w = 0; w < 4; ++w) {
                const uint32_t qw = qv[rr0][0][w];
                unpack_word<BITS>(qw, &un[rr0][w * UPW]);
            }
    }
    // the first slot comes with the table entry, so its activations load
    // together with the codes; the rest of the slot ids are read meanwhile
    int lane_slot = lane < scnt ? a.sorted[sbeg + lane] : 0;
    f16x2 xn[HOIST ? PPC : 1];
    float sxn = 0.f, tn[HOIST ? NBA : 1];
    if constexpr (HOIST) load_x(slot0, xn, sxn, tn);
    for (int jslot = 0; jslot < scnt; ++jslot) {
        if constexpr (!HOIST) {
            if (jslot > 0 && (jslot & 63) == 0) {
                const int j = jslot + lane;
                lane_slot = j < scnt ? a.sorted[sbeg + j] : 0;
            }
        }
        const int sl = __shfl(lane_slot, jslot & 63, 64);
        f16x2 xv[PPC];
        float tv[NBA];
        float sxv;
        if constexpr (HOIST) {
#pragma unroll
            for (int p = 0; p < PPC; ++p) xv[p] = xn[p];
            sxv = sxn;
#pragma unroll
            for (int m = 0; m < NBA; ++m) tv[m] = tn[m];
            if (jslot + 1 < scnt) {
                if (((jslot + 1) & 63) == 0) {
                    const int j = jslot + 1 + lane;
                    lane_slot = j < scnt ? a.sorted[sbeg + j] : 0;
                }
                load_x(__shfl(lane_slot, (jslot + 1) & 63, 64), xn, sxn, tn);
            }
        } else {
            load_x(jslot == 0 ? slot0 : sl, xv, sxv, tv);
        }
        float acc[R];
#pragma unroll
        for (int r = 0; r < R; ++r) {
            float d[NACC];
#pragma unroll
            for (int q = 0; q < NACC; ++q) d[q] = 0.f;
#pragma unroll
            for (int w = 0; w < 4; ++w) {
                if constexpr (HOIST) dot_unpacked<BITS>(&un[r][w * UPW], xv + w * HPW, d);
                else dot_word<BITS>(qv[r][0][w], xv + w * HPW, d);
            }
            const float v = fmaf(combine<BITS>(d), 16777216.0f, -zc[r][0] * sxv);
            acc[r] = sc[r][0] * v;
        }
#pragma unroll
        for (int m = 0; m < NB; ++m)
#pragma unroll
            for (int r = 0; r < R; ++r) acc[r] = fmaf(bv[r][m], tv[m], acc[r]);
        const float tot = group_sum_multi<R, LG>(acc);
        constexpr int SPAN = LG / R;
        const int rr = (lg / SPAN) & (R - 1);
        if (ks == 1 || LG < 64) {               // short rows always have one K slice
            if ((lane & (SPAN - 1)) == 0 && active && row0 + rr < L.d_out)
                store_out(L.y, static_cast<size_t>(sl) * L.d_out + row0 + rr, tot, a.out);
        } else {
            if ((lane & (SPAN - 1)) == 0) red[wave][rr] = tot;
            __syncthreads();
            if (slice == 0 && lane < R && active && row0 + lane < L.d_out) {
                float v = 0.f;
                for (int kk = 0; kk < ks; ++kk) v += red[wave + kk][lane];
                store_out(L.y, static_cast<size_t>(sl) * L.d_out + row0 + lane, v, a.out);
            }
            __syncthreads();
        }
    }
}

// Few slots, 4-bit codes: one launch and no preparation.  Workgroup =
// (linear, slot, block of a.rb rows), the row blocks of one (linear, slot)
// unit on one XCD (48-layer T = 1 step 18.8 -> 18.5 us).  It reads the slot's expert id, forms
// the slot's activations in registers (the same fp16 pairs and chunk sums the
// preparation writes), computes t = A_e[:r] x itself (each of its NWV waves
// takes rows i = wave + NWV p below the rank, UR rows with all their loads in flight,
// one butterfly sum per row; the slot's other workgroups repeat this small
// product, r x d_in multiply-adds over A_e rows that L2 serves after the
// first), and then applies its rows' codes with the arithmetic of
// moe_kernel: row batches of 4 rows per row set of LG lanes, CPL chunks per
// lane.  Every load of the workgroup's NBW batches per wave is issued right
// after the id arrives, before the A_e x product: with one batch in flight
// per wave the layer waited one memory round trip per batch.  At one
// token with 8 routed experts this replaces the preparation launch and its
// dependent memory round trips (ids, A_e rows, then the backbone's reads of
// t and the activations).
// The gated activations h = SiLU(g) u of every slot, 8 per thread, as fp16:
// the input of the preparation and backbone kernels for a gated call.
__global__ __launch_bounds__(256) void moe_gate_kernel(const uint16_t* g, const uint16_t* u, uint16_t* h, size_t n8,
                                                       int act) {
    const size_t i = static_cast<size_t>(blockIdx.x) * 256 + threadIdx.x;
    if (i >= n8) return;
    reinterpret_cast<u32x4*>(h)[i] =
        gated8_to_f16(reinterpret_cast<const u32x4*>(g)[i], reinterpret_cast<const u32x4*>(u)[i], act);
}

template <int LG, int CPL, int NB, int QX, int NBW, bool GATED, int NWV>
__global__ __launch_bounds__(64 * NWV) void moe_direct_kernel(MoeArgs a) {
    constexpr int R = 4, CPC = 32, PPC = 16, HPW = 4, NACC = 2;
    constexpr int SETS = 64 / LG;
    constexpr int NBA = NB > 0 ? NB : 1;
    constexpr int UR = (QX > 4 || NWV > 4) ? 4 : 8;   // rank rows per wave in flight
    __shared__ float tsh[NBA * LG];                // t of the slot, zero past its rank
    __shared__ int rks[256];                       // the experts' ranks (E <= 256)
    // unit u = (linear u / S, slot u % S); workgroup i runs on XCD i % 8, so
    // the row blocks of unit u go to XCD u % 8: its A_e rows and activations
    // stay in one L2
    const int blk = blockIdx.x;
    const int S = a.T * a.k;
    const int nrbm = a.nrbm;
    const int j = blk / 8;
    const int u = blk % 8 + 8 * (j / nrbm);
    const int rbi = j % nrbm;
    if (u >= a.n * S) return;
    const int li = u / S;
    const int sl = u - li * S;
    const MoeLin& L = a.lin[li];
    if (rbi >= L.nrb) return;
    const int rfirst = rbi * a.rb;
    const int rend = min(L.d_out, rfirst + a.rb);
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lg = lane % LG;
    const int chunks = a.d_in / CPC;
    const int words = a.d_in / 8;
    const int groups = a.d_in / a.G;

    const int e = a.ids[sl];
    const int xrow = a.x_per_slot ? sl : sl / a.k;
    const uint16_t* xr = a.x + static_cast<size_t>(xrow) * a.d_in;
    // activations of this lane's chunks (unpack pair order) and their sums
    int cidx[CPL];
    float cmask[CPL];
#pragma unroll
    for (int j = 0; j < CPL; ++j) {
        cidx[j] = lg + LG * j;
        cmask[j] = cidx[j] < chunks ? 1.f : 0.f;
        if (cidx[j] >= chunks) cidx[j] = 0;
    }
    // raw loads here; the conversion (load_chunk_x's pairs and the chunk
    // sums) waits until the other loads are out
    u32x4 xraw[CPL][4];
#pragma unroll
    for (int j = 0; j < CPL; ++j)
#pragma unroll
        for (int w = 0; w < 4; ++w) xraw[j][w] = *reinterpret_cast<const u32x4*>(xr + (cidx[j] * 4 + w) * 8);
    // gated input: the up rows beside the gate rows, SiLU(g) u formed at
    // the conversions below
    const uint16_t* ur = GATED ? a.u + static_cast<size_t>(xrow) * a.d_in : xr;
    u32x4 uraw[GATED ? CPL : 1][4];
    if constexpr (GATED) {
#pragma unroll
        for (int j = 0; j < CPL; ++j)
#pragma unroll
            for (int w = 0; w < 4; ++w) uraw[j][w] = *reinterpret_cast<const u32x4*>(ur + (cidx[j] * 4 + w) * 8);
    }
    // the rank comes with the id: per-slot ranks one word, static ranks the
    // whole table (thread i its expert i, E <= 256) for an LDS lookup once e
    // is known; both loads unconditional from selected pointers (a load
    // under a branch is waited for where the branches meet)
    const bool rtab = L.r_max > 0 && !L.slot_rank && a.E <= 256;
    const int rk_tab = (rtab ? L.ranks : a.ids)[rtab ? min(tid, a.E - 1) : 0];
    const int rk_slot = (L.slot_rank ? L.slot_rank : a.ids)[sl];
    if (e < 0 || e >= a.E) {
        // out-of-range id: this slot's rows are zero, and the device's
        // routing-error record notes it (as the preparation does)
        if (li == 0 && rbi == 0 && tid == 0)
            __hip_atomic_store(&moe_routing_error,
                               (1ull << 63) | (static_cast<unsigned long long>(sl) << 32) | static_cast<uint32_t>(e),
                               __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        for (int o = rfirst + tid; o < rend; o += 64 * NWV)
            store_out(L.y, static_cast<size_t>(sl) * L.d_out + o, 0.f, a.out);
        return;
    }

    // row batches: batch b covers rows rfirst + b R SETS .. + R SETS - 1, a
    // row set of LG lanes R consecutive rows; wave w takes b = w, w + NWV, ...
    const uint32_t* qe = L.q + static_cast<size_t>(e) * L.q_stride;
    const uint16_t* se = L.s + static_cast<size_t>(e) * L.sz_stride;
    const uint16_t* ze = L.z + static_cast<size_t>(e) * L.sz_stride;
    const uint16_t* Be = L.B + static_cast<size_t>(e) * L.b_stride;
    const int nbatch = (rend - rfirst + R * SETS - 1) / (R * SETS);
    // scales, zeros and factor entries one per register: 16-bit loads into
    // register halves make each load wait for the one before
    struct Bt {
        u32x4 q[R][CPL];
        uint32_t s[R][CPL], z[R][CPL], b[R][NBA];
    };
    auto row_of = [&](int b, int& row0, int& nrows) {
        row0 = rfirst + b * R * SETS + (lane / LG) * R;
        nrows = row0 < rend ? min(R, rend - row0) : 0;
    };
    auto load_batch = [&](int b, Bt& bt) {
        int row0, nrows;
        row_of(b, row0, nrows);
        const int base = nrows > 0 ? row0 : rfirst;
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int row = base + (r < nrows ? r : 0);
#pragma unroll
            for (int j = 0; j < CPL; ++j) {
                bt.q[r][j] = __builtin_nontemporal_load(
                    reinterpret_cast<const u32x4*>(qe + static_cast<size_t>(row) * words) + cidx[j]);
                const size_t gi = static_cast<size_t>(row) * groups + (cidx[j] * CPC) / a.G;
                bt.s[r][j] = se[gi];
                bt.z[r][j] = ze[gi];
            }
#pragma unroll
            for (int m = 0; m < NB; ++m) {
                const int i = lg + LG * m;
                bt.b[r][m] = Be[static_cast<size_t>(row) * L.r_max + (i < L.r_max ? i : 0)];
            }
        }
    };
    // all of this wave's batches (b = wave + NWV u) load before the t product,
    // unconditionally (a batch past the last reads the last one's rows): a
    // load under a branch is waited for where the branches meet
    Bt bts[NBW];
#pragma unroll
    for (int u = 0; u < NBW; ++u) load_batch(min(wave + NWV * u, nbatch - 1), bts[u]);

    // t = A_e[:rank] x: x as fp16 runs, lane l and pass q holding columns
    // 512 q + 8 l .. + 7
    // raw loads now, the conversion after the A loads are out
    u32x4 xw[QX], uw[GATED ? QX : 1];
#pragma unroll
    for (int q = 0; q < QX; ++q) {
        const int c = 512 * q + 8 * lane;
        xw[q] = *reinterpret_cast<const u32x4*>(xr + (c < a.d_in ? c : 0));
        if constexpr (GATED) uw[q] = *reinterpret_cast<const u32x4*>(ur + (c < a.d_in ? c : 0));
    }
    bool xconv = false;
    // the slot's rank (the batches' loads are out; the A rows wait for it)
    if (tid < 256) rks[tid] = rk_tab;
    __syncthreads();
    int rank = L.slot_rank ? rk_slot : (rtab ? rks[e] : (L.r_max > 0 ? L.ranks[e] : 0));
    rank = L.r_max == 0 ? 0 : (rank < 0 ? 0 : (rank > L.r_max ? L.r_max : rank));
    const uint16_t* Ae = L.A + static_cast<size_t>(e) * L.a_stride;
    // rows below the rank only
    for (int p0 = 0; wave + NWV * p0 < rank; p0 += UR) {
        // clamped addresses and selects: the loads carry no branches
        u32x4 av[UR][QX];
#pragma unroll
        for (int u = 0; u < UR; ++u) {
            const int i = wave + NWV * (p0 + u);
            const int ic = i < rank ? i : wave;
#pragma unroll
            for (int q = 0; q < QX; ++q) {
                const int c = 512 * q + 8 * lane;
                av[u][q] = *reinterpret_cast<const u32x4*>(Ae + static_cast<size_t>(ic) * a.d_in + (c < a.d_in ? c : 0));
            }
        }
        // keep the value work below the loads above (hoisted, it waited for
        // earlier loads before these were issued)
        __builtin_amdgcn_sched_barrier(0);
        if (!xconv) {
#pragma unroll
            for (int q = 0; q < QX; ++q) {
                u32x4 v;
                if constexpr (GATED) v = gated8_to_f16(xw[q], uw[q], a.act);
                else v = act8_to_f16(xw[q], a.act);
                xw[q] = 512 * q + 8 * lane < a.d_in ? v : u32x4{0u, 0u, 0u, 0u};
            }
            xconv = true;
        }
        float d[UR];
#pragma unroll
        for (int u = 0; u < UR; ++u) {
            d[u] = 0.f;
#pragma unroll
            for (int q = 0; q < QX; ++q)
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    // copy the vector elements to scalars first: a bit_cast
                    // of a subscripted ext_vector reads element 0
                    const uint32_t ak = av[u][q][k], xk = xw[q][k];
                    d[u] = dot2(__builtin_bit_cast(f16x2, ak), __builtin_bit_cast(f16x2, xk), d[u]);
                }
        }
        // lane l holds the total of row p0 + l / (64 / UR)
        const float tot = wave_sum_multi<UR>(d);
        const int u = lane / (64 / UR);
        const int i = wave + NWV * (p0 + u);
        if (lane % (64 / UR) == 0 && i < rank) tsh[i] = tot;
    }
    for (int i = rank + tid; i < NBA * LG; i += 64 * NWV) tsh[i] = 0.f;
    __syncthreads();
    // the activations of this lane's chunks in the unpack's pair order,
    // (x[w 8 + p], x[w 8 + p + 4]) for word w and pair p, and their sums
    f16x2 xv[CPL][PPC];
    float sxv[CPL];
    const f16x2 one = {static_cast<f16>(1.0f), static_cast<f16>(1.0f)};
#pragma unroll
    for (int j = 0; j < CPL; ++j) {
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            u32x4 u;
            if constexpr (GATED) u = gated8_to_f16(xraw[j][w], uraw[j][w], a.act);
            else u = act8_to_f16(xraw[j][w], a.act);
#pragma unroll
            for (int pp = 0; pp < 4; ++pp) {
                const uint32_t lo = u[pp / 2], hi = u[(pp + 4) / 2];
                const uint32_t va = (pp & 1) ? (lo >> 16) : (lo & 0xffff);
                const uint32_t vb = (pp & 1) ? (hi & 0xffff0000u) : (hi << 16);
                xv[j][w * HPW + pp] = __builtin_bit_cast(f16x2, va | vb);
            }
        }
        float sum = 0.f;
#pragma unroll
        for (int p = 0; p < PPC; ++p) sum = dot2(xv[j][p], one, sum);
        sxv[j] = sum;
    }
    float tv[NBA];
#pragma unroll
    for (int m = 0; m < NBA; ++m) tv[m] = NB > 0 ? tsh[lg + LG * m] : 0.f;

#pragma unroll
    for (int u = 0; u < NBW; ++u) {
        const int b = wave + NWV * u;
        if (b >= nbatch) break;
        const Bt& cur = bts[u];
        int row0, nrows;
        row_of(b, row0, nrows);
        float acc[R];
#pragma unroll
        for (int r = 0; r < R; ++r) {
            acc[r] = 0.f;
#pragma unroll
            for (int j = 0; j < CPL; ++j) {
                float d[NACC];
#pragma unroll
                for (int q = 0; q < NACC; ++q) d[q] = 0.f;
#pragma unroll
                for (int w = 0; w < 4; ++w) dot_word<4>(cur.q[r][j][w], xv[j] + w * HPW, d);
                const float v = fmaf(combine<4>(d), 16777216.0f, -f16_bits_to_f32(cur.z[r][j]) * sxv[j]);
                acc[r] = fmaf(f16_bits_to_f32(cur.s[r][j]) * cmask[j], v, acc[r]);
            }
#pragma unroll
            for (int m = 0; m < NB; ++m) {
                const float bvm = lg + LG * m < rank ? f16_bits_to_f32(cur.b[r][m]) : 0.f;
                acc[r] = fmaf(bvm, tv[m], acc[r]);
            }
        }
        const float tot = group_sum_multi<R, LG>(acc);
        constexpr int SPAN = LG / R;
        const int rr = (lg / SPAN) & (R - 1);
        if ((lane & (SPAN - 1)) == 0 && rr < nrows)
            store_out(L.y, static_cast<size_t>(sl) * L.d_out + row0 + rr, tot, a.out);
    }
}

// Many slots per expert, 4-bit codes: the expert's rows against its slots on
// MFMA (v_mfma_f32_16x16x32_f16), so the per-slot VALU work of the kernel
// above (every slot's dot products on every lane) becomes MFMA rows.
// Workgroup = (linear, active expert, TPW tiles of 16 rows); its four waves
// split the 128-code blocks of K (wave w takes blocks w, w + 4, ..., NBUF in
// flight); the expert's slots go in passes of 16.  Per block a lane loads,
// for each tile, 16 bytes of codes of row r = lane % 16, and once for all
// tiles the matching four 16-byte words of prepared activations of its
// pass's slot r.  The activations are the MFMA's A operand and the codes its
// B operand, so lane (g, r) accumulates slots 4 g .. 4 g + 3 of the pass for
// weight row r.  As in the many-token dense decode the codes become the
// exact fp16 integers q - z and each quantization group's steps run into a
// fresh fp32 partial that the group's scale multiplies in fp32 (GPB groups
// per 128-code block; with more than one the code words are transposed
// across the lane groups first).  The rank term is extra MFMA steps over
// [t | B_e] (t split into fp16 hi and lo parts, one step each); the waves'
// tiles are summed through LDS in a fixed order; one rounding to the output
// dtype.
template <int TPW, int NBUF, int GPB>
__global__ __launch_bounds__(256) void moe_mfma_kernel(MoeArgs a) {
    __shared__ f32x4 red[4][TPW][64];
    extern __shared__ uint16_t szl[];             // [2][16 TPW][szl_stride(groups)]: the rows' scales, then zeros
    const int blk = blockIdx.x;
    int li = 0;
    while (blk >= a.lin[li].blk_end) ++li;
    const MoeLin& L = a.lin[li];
    const int local = blk - (li ? a.lin[li - 1].blk_end : 0);
    const int ae = local / L.bpe;                 // bpe: workgroups (16 TPW rows) per expert
    const int n_active = *a.n_active;
    const int* ent = a.table + kTab * ae;
    const int e = ent[0], sbeg = ent[1], scnt = ent[2], rank = ent[4 + li];
    if (ae >= n_active) return;                   // whole workgroup: no routed expert here
    const int row0 = (local - ae * L.bpe) * 16 * TPW;
    const int lane = threadIdx.x & 63;
    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int g = lane >> 4, r = lane & 15;
    int row[TPW];
    bool rowv[TPW];
#pragma unroll
    for (int j = 0; j < TPW; ++j) {
        rowv[j] = row0 + 16 * j + r < L.d_out;
        row[j] = rowv[j] ? row0 + 16 * j + r : L.d_out - 1;
    }
    const int K = a.d_in;
    const int nkb = (K + 127) / 128;
    const int words_row = K / 8;
    const int groups = K / a.G;
    const uint32_t* qe = L.q + static_cast<size_t>(e) * L.q_stride;
    const uint16_t* se = L.s + static_cast<size_t>(e) * L.sz_stride;
    const uint16_t* ze = L.z + static_cast<size_t>(e) * L.sz_stride;
    const uint16_t* Be = L.B + static_cast<size_t>(e) * L.b_stride;
    const uint32_t mlo = __builtin_amdgcn_readfirstlane(0x000F000Fu);
    const uint32_t mhi = __builtin_amdgcn_readfirstlane(0x00F000F0u);
    const uint32_t bias = 0x64006400u;
    const u32x4 zero = {0u, 0u, 0u, 0u};

    struct Blk {
        u32x4 w[TPW];
        u32x4 x[4];
    };
    // codes of block kb for this lane's tiles, and the activations of the
    // words it feeds to MFMA step t: 4 g + t of the block, or 4 t + g once
    // the codes are transposed (a word past K reads word g, met by a zero
    // scale).  Loads are unconditional (clamped addresses) and nothing
    // consumes a loaded value before compute.  A block past the last one
    // (the pipeline's tail) reads one line, the expert's first 16 bytes, on
    // every lane: reloading a block already computed fetched its lines from
    // HBM a second time (the streamed code lines have left L2 by then; the
    // down linear's 6 blocks on 4 waves had fetched 2.25 times its bytes).
    auto load_w = [&](int kb, Blk& b) {
        const bool live = kb < nkb;
        const int wi = min(kb * 16 + 4 * g, words_row - 4);
#pragma unroll
        for (int j = 0; j < TPW; ++j)
            b.w[j] = __builtin_nontemporal_load(
                live ? reinterpret_cast<const u32x4*>(qe + static_cast<size_t>(row[j]) * words_row + wi)
                     : reinterpret_cast<const u32x4*>(qe));
    };
    auto load_x = [&](int kb, Blk& b, const u32x4* xr) {
        const int wi = min(kb * 16 + 4 * g, words_row - 4);
#pragma unroll
        for (int t = 0; t < 4; ++t)
            b.x[t] = xr[GPB == 1 ? wi + t : (kb * 128 + 32 * t < K ? kb * 16 + 4 * t + g : g)];
    };
    // rank-term operands of the step at factor column kr: this lane's slot's
    // t (8 floats, zero past its rank) and the tiles' B entries
    struct RankOp {
        float t[8];
        uint32_t bw[TPW][4];
    };
    // 16-byte loads when every row of t and B starts 16-byte aligned (r_max a
    // multiple of 8: t rows of r_max floats in the 256-byte aligned
    // workspace, B rows of r_max halves); a step past r_max reads column 0
    const bool rvec = (L.r_max & 7) == 0 && (reinterpret_cast<uintptr_t>(L.B) & 15) == 0;
    auto rank_load = [&](int kr, int sl, RankOp& o) {
        const int k = kr + 8 * g;
        const float* trow = L.t + static_cast<size_t>(sl) * L.r_max;
        if (rvec) {
            const int kk = k + 8 <= L.r_max ? k : 0;
            const f32x4 t0 = *reinterpret_cast<const f32x4*>(trow + kk);
            const f32x4 t1 = *reinterpret_cast<const f32x4*>(trow + kk + 4);
#pragma unroll
            for (int q = 0; q < 4; ++q) { o.t[q] = t0[q]; o.t[4 + q] = t1[q]; }
#pragma unroll
            for (int j = 0; j < TPW; ++j) {
                const u32x4 v = *reinterpret_cast<const u32x4*>(Be + static_cast<size_t>(row[j]) * L.r_max + kk);
#pragma unroll
                for (int q = 0; q < 4; ++q) { const uint32_t vq = v[q]; o.bw[j][q] = vq; }
            }
            return;
        }
#pragma unroll
        for (int q = 0; q < 8; ++q) o.t[q] = trow[k + q < L.r_max ? k + q : 0];
#pragma unroll
        for (int j = 0; j < TPW; ++j) {
            const uint16_t* brow = Be + static_cast<size_t>(row[j]) * L.r_max;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int k0 = k + 2 * q, k1 = k0 + 1;
                const uint32_t lo = brow[k0 < L.r_max ? k0 : 0];
                const uint32_t hi = brow[k1 < L.r_max ? k1 : 0];
                o.bw[j][q] = lo | (hi << 16);
            }
        }
    };

    // What is needed first is issued first (vector loads complete in issue
    // order): the scales and zeros of the workgroup's rows, then this lane's
    // slot of the first pass, then the first round of code blocks; the LDS
    // copy of the scales and zeros then waits only for them, and the code
    // loads stay in flight across the barrier.  (Issued after the copy, the
    // code loads had one more dependent round trip per workgroup.)
    const int nval = min(16 * TPW, L.d_out - row0) * groups;
    const uint16_t* ssrc = se + static_cast<size_t>(row0) * groups;
    const uint16_t* zsrc = ze + static_cast<size_t>(row0) * groups;
    const int RS = szl_stride(groups);            // padded row stride of the tables
    uint16_t* zl = szl + 16 * TPW * RS;
    const bool al = ((reinterpret_cast<uintptr_t>(ssrc) | reinterpret_cast<uintptr_t>(zsrc)) & 15) == 0;
    const int n16 = al ? nval / 8 : 0;
    // table entry of the run's value i (row i / groups, column i % groups;
    // the identity on an unpadded table, where pieces may span rows)
    auto tix = [&](int i) { return RS == groups ? i : i / groups * RS + i % groups; };
    // first 16-byte piece of each array per thread (a valid aligned address
    // when this thread has none)
    const u32x4* s16p = n16 ? reinterpret_cast<const u32x4*>(ssrc) + min(tid, n16 - 1)
                            : reinterpret_cast<const u32x4*>(a.table);
    const u32x4* z16p = n16 ? reinterpret_cast<const u32x4*>(zsrc) + min(tid, n16 - 1)
                            : reinterpret_cast<const u32x4*>(a.table);
    const u32x4 s_first = *s16p, z_first = *z16p;
    int sl = a.sorted[sbeg + (r < scnt ? r : 0)];
    constexpr int SPAN = 4 * NBUF;
    const int rounds = (nkb + SPAN - 1) / SPAN;
    Blk b[NBUF];
#pragma unroll
    for (int j = 0; j < NBUF; ++j) load_w(wave + 4 * j, b[j]);
    if (tid < n16) {
        *reinterpret_cast<u32x4*>(szl + tix(8 * tid)) = s_first;
        *reinterpret_cast<u32x4*>(zl + tix(8 * tid)) = z_first;
    }
    for (int i = tid + 256; i < n16; i += 256) {           // rows with more than 32 groups
        *reinterpret_cast<u32x4*>(szl + tix(8 * i)) = reinterpret_cast<const u32x4*>(ssrc)[i];
        *reinterpret_cast<u32x4*>(zl + tix(8 * i)) = reinterpret_cast<const u32x4*>(zsrc)[i];
    }
    for (int i = 8 * n16 + tid; i < nval; i += 256) {      // misaligned runs, the last few values
        szl[tix(i)] = ssrc[i];
        zl[tix(i)] = zsrc[i];
    }
    __syncthreads();

    for (int p0 = 0; p0 < scnt; p0 += 16) {
        if (p0 > 0) {
            // a later pass of 16 slots: its slots and its first code round
            sl = a.sorted[sbeg + (p0 + r < scnt ? p0 + r : 0)];
#pragma unroll
            for (int j = 0; j < NBUF; ++j) load_w(wave + 4 * j, b[j]);
        }
        // this lane's slot (MFMA row r of the activations); absent slots read
        // a present one and are masked to zero
        const bool sv = p0 + r < scnt;
        const int xrow = a.x_per_slot ? sl : sl / a.k;
        const u32x4* xr = reinterpret_cast<const u32x4*>(a.xp + static_cast<size_t>(xrow) * (K / 2));
#pragma unroll
        for (int j = 0; j < NBUF; ++j) load_x(wave + 4 * j < nkb ? wave + 4 * j : 0, b[j], xr);
        // this lane's slot's rank: its own (per-slot ranks) or the expert's
        int rs = rank;
        if (L.slot_rank) {
            const int v = L.slot_rank[sl];
            rs = v < 0 ? 0 : (v > L.r_max ? L.r_max : v);
        }
        f32x4 acc[TPW];
#pragma unroll
        for (int j = 0; j < TPW; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
        auto compute = [&](int kb, const Blk& bk) {
            // per group: MFMA steps into a fresh partial of sum (q - z) x,
            // then acc += s * partial in fp32; past K, past the matrix or a
            // padding block the scale is 0
            constexpr int SPG = 4 / GPB;
            u32x4 xv[4];
#pragma unroll
            for (int t = 0; t < 4; ++t) xv[t] = sv ? bk.x[t] : zero;
#pragma unroll
            for (int j = 0; j < TPW; ++j) {
                uint32_t w[4];
#pragma unroll
                for (int t = 0; t < 4; ++t) { const uint32_t v = bk.w[j][t]; w[t] = v; }
                if constexpr (GPB > 1) transpose_words(w);
#pragma unroll
                for (int q = 0; q < GPB; ++q) {
                    const int kc = kb * 128 + 32 * SPG * q;
                    const bool on = kb < nkb && kc < K && rowv[j];
                    const int lr = (16 * j + r) * RS + (on ? kc / a.G : 0);
                    const Zq zq = make_zq(szl[16 * TPW * RS + lr]);
                    f32x4 pp = mfma(xv[SPG * q], codes_minus_zero(w[SPG * q], zq, mlo, mhi, bias),
                                    f32x4{0.f, 0.f, 0.f, 0.f});
#pragma unroll
                    for (int t = SPG * q + 1; t < SPG * q + SPG; ++t)
                        pp = mfma(xv[t], codes_minus_zero(w[t], zq, mlo, mhi, bias), pp);
                    acc[j] = fma4(on ? f16_bits_to_f32(szl[lr]) : 0.f, pp, acc[j]);
                }
            }
        };
        for (int rd = 0; rd < rounds; ++rd) {
#pragma unroll
            for (int j = 0; j < NBUF; ++j) {
                const int kb = wave + SPAN * rd + 4 * j;
                compute(kb, b[j]);
                const int kn = kb + SPAN;
                load_w(kn, b[j]);
                load_x(kn < nkb ? kn : 0, b[j], xr);
            }
        }
        // rank-r term: 32 factor columns per step, wave w taking steps w, w + 4
        // (t as fp16 hi + lo parts, two MFMA steps; entries past the slot's
        // rank, past the expert's rank or of absent slots and rows are zero)
        auto rank_mma = [&](int kr, const RankOp& o) {
            const int k = kr + 8 * g;
            uint32_t tw[4], tlo[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int k0 = k + 2 * q, k1 = k0 + 1;
                split_f16x2((sv && k0 < rs) ? o.t[2 * q] : 0.f, (sv && k1 < rs) ? o.t[2 * q + 1] : 0.f, tw[q],
                            tlo[q]);
            }
#pragma unroll
            for (int j = 0; j < TPW; ++j) {
                uint32_t aw[4];
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int k0 = k + 2 * q, k1 = k0 + 1;
                    const uint32_t lo = (rowv[j] && k0 < rank) ? (o.bw[j][q] & 0xffffu) : 0u;
                    const uint32_t hi = (rowv[j] && k1 < rank) ? (o.bw[j][q] >> 16) : 0u;
                    aw[q] = lo | (hi << 16);
                }
                const u32x4 bop = {aw[0], aw[1], aw[2], aw[3]};
                acc[j] = mfma(u32x4{tw[0], tw[1], tw[2], tw[3]}, bop, acc[j]);
                acc[j] = mfma(u32x4{tlo[0], tlo[1], tlo[2], tlo[3]}, bop, acc[j]);
            }
        };
        // (prefetching the first step's operands ahead of the K loop kept
        // them live through it: 256 VGPRs plus 72 AGPRs, one wave per SIMD)
        for (int kr = 32 * wave; kr < rank; kr += 128) {
            RankOp o2;
            rank_load(kr, sl, o2);
            rank_mma(kr, o2);
        }
#pragma unroll
        for (int j = 0; j < TPW; ++j) red[wave][j][lane] = acc[j];
        __syncthreads();
        // wave w sums and stores tiles w, w + 4, ... in a fixed order;
        // v[e] = y[slot of pass row 4 g + e][row0 + 16 j + r]
        int osl[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) osl[q] = __shfl(sl, 4 * g + q, 64);
#pragma unroll
        for (int j = 0; j < TPW; ++j) {
            if (j % 4 != wave || !rowv[j]) continue;
            const f32x4 v = red[0][j][lane] + red[1][j][lane] + red[2][j][lane] + red[3][j][lane];
#pragma unroll
            for (int q = 0; q < 4; ++q)
                if (p0 + 4 * g + q < scnt) store_out(L.y, static_cast<size_t>(osl[q]) * L.d_out + row[j], v[q], a.out);
        }
        __syncthreads();                           // red is reused by the next pass
    }
}

size_t up256(size_t n) { return (n + 255) / 256 * 256; }

struct MoeLayout {
    size_t n_active, table, sorted, t[kMaxMoeWin], xp, sx, h, total;
};

MoeLayout moe_layout(int n, const QW* w, const int* r_max, int E, int T, int k, int x_per_slot) {
    const int S = T * k;
    const int max_active = S < E ? S : E;
    const int rows = x_per_slot ? S : T;
    const size_t chunks = static_cast<size_t>(w[0].d_in) / (32 / w[0].bits) / 4;
    MoeLayout l;
    l.n_active = 0;
    l.table = 256;
    l.sorted = l.table + up256(static_cast<size_t>(max_active) * kTab * sizeof(int));
    size_t off = l.sorted + up256(static_cast<size_t>(S) * sizeof(int));
    for (int i = 0; i < n; ++i) {
        l.t[i] = off;
        off += up256(static_cast<size_t>(S) * r_max[i] * sizeof(float));
    }
    l.xp = off;
    l.sx = l.xp + up256(static_cast<size_t>(rows) * w[0].d_in * 2);
    l.h = l.sx + up256(static_cast<size_t>(rows) * chunks * sizeof(float));
    // gated per-slot input (x_per_slot 2): SiLU(g) u of every slot in fp16
    l.total = l.h + (x_per_slot == 2 ? up256(static_cast<size_t>(S) * w[0].d_in * 2) : 0);
    return l;
}

template <int BITS, int CPL, int NB, int LG>
hipError_t launch_moe4(const MoeArgs& a, bool hoist, int blocks, int threads, hipStream_t st) {
    if (hoist)
        hipLaunchKernelGGL((moe_kernel<BITS, CPL, NB, true, LG>), dim3(blocks), dim3(threads), 0, st, a);
    else
        hipLaunchKernelGGL((moe_kernel<BITS, CPL, NB, false, LG>), dim3(blocks), dim3(threads), 0, st, a);
    return hipGetLastError();
}

template <int BITS, int LG>
hipError_t launch_moe3(const MoeArgs& a, int nb, bool hoist, int blocks, int threads, hipStream_t st) {
    switch (nb) {
        case 0: return launch_moe4<BITS, 1, 0, LG>(a, hoist, blocks, threads, st);
        case 1: return launch_moe4<BITS, 1, 1, LG>(a, hoist, blocks, threads, st);
        case 2: return launch_moe4<BITS, 1, 2, LG>(a, hoist, blocks, threads, st);
        default: return launch_moe4<BITS, 1, 4, LG>(a, hoist, blocks, threads, st);
    }
}

template <int BITS>
hipError_t launch_moe2(const MoeArgs& a, int lg, int nb, bool hoist, int blocks, int threads, hipStream_t st) {
    if (lg == 16) return launch_moe3<BITS, 16>(a, nb, hoist, blocks, threads, st);
    if (lg == 32) return launch_moe3<BITS, 32>(a, nb, hoist, blocks, threads, st);
    return launch_moe3<BITS, 64>(a, nb, hoist, blocks, threads, st);
}

// Eight waves per workgroup, each with half the row batches of four (the
// rows per workgroup unchanged): two waves per SIMD where four held one,
// and the t product's rank rows spread over twice the waves (48-layer
// T = 1 step 18.9 -> 16.7 us).  The gated instance keeps four: every wave
// forms SiLU(g) u for the whole activation row it converts, so eight
// waves doubled that work (down 9.4 -> 11.2 us).
template <int LG, int CPL, int QX, bool G>
hipError_t launch_direct4(const MoeArgs& a, int nb, int blocks, hipStream_t st) {
    constexpr int NWV = G ? 4 : 8;
    constexpr int NBW = direct_batches(LG, CPL) * 4 / NWV;
    const dim3 th(64 * NWV);
    if (nb == 0) hipLaunchKernelGGL((moe_direct_kernel<LG, CPL, 0, QX, NBW, G, NWV>), dim3(blocks), th, 0, st, a);
    else if (nb == 1) hipLaunchKernelGGL((moe_direct_kernel<LG, CPL, 1, QX, NBW, G, NWV>), dim3(blocks), th, 0, st, a);
    else hipLaunchKernelGGL((moe_direct_kernel<LG, CPL, 2, QX, NBW, G, NWV>), dim3(blocks), th, 0, st, a);
    return hipGetLastError();
}

template <int LG, int CPL, int QX>
hipError_t launch_direct3(const MoeArgs& a, int nb, int blocks, hipStream_t st) {
    return a.u ? launch_direct4<LG, CPL, QX, true>(a, nb, blocks, st)
               : launch_direct4<LG, CPL, QX, false>(a, nb, blocks, st);
}

// (LG, CPL, QX) instances: 24-32 chunk rows (d_in <= 1024), 64-chunk rows
// (d_in <= 2048), 128-chunk rows (d_in <= 4096)
hipError_t launch_direct(const MoeArgs& a, int lg, int cpl, int nb, int qx, int blocks, hipStream_t st) {
    if (lg == 32) return launch_direct3<32, 1, 2>(a, nb, blocks, st);
    if (cpl == 1 && qx <= 4) return launch_direct3<64, 1, 4>(a, nb, blocks, st);
    return launch_direct3<64, 2, 8>(a, nb, blocks, st);
}

}  // namespace

bool moe_fits(const QW& w, int E, int T, int k) {
    // one chunk per lane over at most 8 K slices: d_in <= 16384 (4-bit), 32768 (2-bit)
    const int chunks = w.d_in / (32 / w.bits) / 4;
    return chunks <= 8 * 64 && E <= kMaxExperts && T * k <= kMaxSlots;
}

size_t moe_workspace_bytes(int n, const QW* w, const int* r_max, int E, int T, int k, int x_per_slot) {
    return moe_layout(n, w, r_max, E, T, k, x_per_slot).total;
}

hipError_t launch_moe_decode(int n, const QW* w, const uint16_t* const* A, const uint16_t* const* B,
                             const int* r_max, const int32_t* const* ranks, const int32_t* const* slot_ranks,
                             int E, const void* x, const void* u, int x_per_slot,
                             const int32_t* ids, int T, int k, int act, void* const* y, int out, void* ws,
                             hipStream_t st) {
    if (n < 1 || n > kMaxMoeWin) return hipErrorInvalidConfiguration;
    const MoeLayout l = moe_layout(n, w, r_max, E, T, k, x_per_slot);
    char* wsb = static_cast<char*>(ws);
    const int d_in = w[0].d_in, bits = w[0].bits;
    MoeArgs a{};
    a.n = n;
    a.ids = ids;
    a.x = static_cast<const uint16_t*>(x);
    a.u = static_cast<const uint16_t*>(u);
    a.E = E; a.T = T; a.k = k; a.d_in = d_in; a.G = w[0].G;
    a.act = act; a.out = out; a.x_per_slot = x_per_slot ? 1 : 0;
    a.n_active = reinterpret_cast<int*>(wsb + l.n_active);
    a.table = reinterpret_cast<int*>(wsb + l.table);
    a.sorted = reinterpret_cast<int*>(wsb + l.sorted);
    a.xp = reinterpret_cast<f16x2*>(wsb + l.xp);
    a.sx = reinterpret_cast<float*>(wsb + l.sx);
    // K split as in the dense decode: one chunk per lane, a power-of-two
    // number of slices (at most 8, which moe_fits guarantees)
    const int chunks = d_in / (32 / bits) / 4;
    int ks = (chunks + 63) / 64;
    while (ks & (ks - 1)) ++ks;
    a.ks = ks;
    a.cps = (chunks + a.ks - 1) / a.ks;
    // lanes per row set: rows shorter than 64 chunks share a wave between
    // 2 or 4 row sets (one K slice)
    int rmax = 0;
    for (int i = 0; i < n; ++i) rmax = max(rmax, r_max[i]);
    int lg = chunks <= 16 ? 16 : (chunks <= 32 ? 32 : 64);
    if (rmax > 4 * lg) lg = 64;                    // at most 4 factor columns per lane
    const int sets = 64 / lg;
    const int threads = 64 * (a.ks > 4 ? a.ks : 4);
    if (a.ks > 8 || threads > 512 || threads % (64 * a.ks)) return hipErrorInvalidConfiguration;
    if (lg < 64 && a.ks != 1) return hipErrorInvalidConfiguration;
    const int rg_per_block = threads / 64 / a.ks * sets;
    const int S = T * k;
    const int max_active = S < E ? S : E;
    // experts meeting two or more slots on average: 4-bit codes go to MFMA
    // (tiles of 16 rows), 2-bit codes are unpacked once per batch
    const bool many = S >= 2 * max_active;
    const bool on_mfma = many && bits == 4;
    int prep_end = 0, blk_end = 0;
    for (int i = 0; i < n; ++i) {
        MoeLin& L = a.lin[i];
        L.q = w[i].q; L.s = w[i].s; L.z = w[i].z; L.A = A[i]; L.B = B[i]; L.ranks = ranks[i];
        L.slot_rank = slot_ranks ? slot_ranks[i] : nullptr;
        L.y = y[i];
        L.t = reinterpret_cast<float*>(wsb + l.t[i]);
        L.q_stride = static_cast<size_t>(w[i].d_out) * (d_in / (32 / bits));
        L.sz_stride = static_cast<size_t>(w[i].d_out) * (d_in / w[i].G);
        L.a_stride = static_cast<size_t>(r_max[i]) * d_in;
        L.b_stride = static_cast<size_t>(w[i].d_out) * r_max[i];
        L.d_out = w[i].d_out;
        L.r_max = r_max[i];
        L.rq = r_max[i] > 0 ? (r_max[i] + 3) / 4 : 1;
        const int rgroups = (w[i].d_out + rows_per_wave(bits) - 1) / rows_per_wave(bits);
        L.bpe = on_mfma ? (w[i].d_out + 16 * kMoeTpw - 1) / (16 * kMoeTpw)
                        : (rgroups + rg_per_block - 1) / rg_per_block;
        prep_end += max_active * L.rq;
        blk_end += max_active * L.bpe;
        L.prep_end = prep_end;
        L.blk_end = blk_end;
    }
    // few slots, 4-bit codes, rows of at most 4096 codes: the direct path
    // (one launch, no preparation, no workspace)
    const int dlg = chunks <= 32 ? 32 : 64;
    const int dcpl = (chunks + dlg - 1) / dlg;
    if (bits == 4 && S <= kDirectMaxSlots && dcpl <= 2 && rmax <= 2 * dlg) {
        a.rb = 16 * (64 / dlg) * direct_batches(dlg, dcpl);
        int nrbm = 0;
        for (int i = 0; i < n; ++i) {
            MoeLin& L = a.lin[i];
            L.nrb = (w[i].d_out + a.rb - 1) / a.rb;
            nrbm = max(nrbm, L.nrb);
        }
        a.nrbm = nrbm;
        const int dblk = 8 * ((n * S + 7) / 8) * nrbm;
        const int dnb = rmax == 0 ? 0 : (rmax <= dlg ? 1 : 2);
        const int qx = d_in <= 1024 ? 2 : (d_in <= 2048 ? 4 : 8);
        return launch_direct(a, dlg, dcpl, dnb, qx, dblk, st);
    }
    const int per = lg * a.ks;                     // factor columns per lane pass
    const int nb = rmax == 0 ? 0 : (rmax <= per ? 1 : (rmax <= 2 * per ? 2 : 4));
    if (rmax > 4 * per) return hipErrorInvalidConfiguration;

    if (a.u) {
        // gated input off the one-launch path: SiLU(g) u once for every slot
        // (each preparation workgroup forming it for its slots had repeated
        // the exponentials once per rank row: 52 against 11 us at 512 slots),
        // then the plain path on it
        uint16_t* h = reinterpret_cast<uint16_t*>(wsb + l.h);
        const size_t n8 = static_cast<size_t>(S) * d_in / 8;
        hipLaunchKernelGGL(moe_gate_kernel, dim3(static_cast<unsigned>((n8 + 255) / 256)), dim3(256), 0, st, a.x, a.u,
                           h, n8, a.act);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        a.x = h;
        a.u = nullptr;
        a.act = DT_FP16;
    }
    const int rows = x_per_slot ? S : T;
    const long long items = static_cast<long long>(rows) * chunks;
    const unsigned pgrid = static_cast<unsigned>(prep_end + (items + 255) / 256);
    const size_t plds = static_cast<size_t>(2 * S + 2 * E) * sizeof(int);
    if (bits == 4)
        hipLaunchKernelGGL(moe_prep_kernel<4>, dim3(pgrid), dim3(256), plds, st, a);
    else
        hipLaunchKernelGGL(moe_prep_kernel<2>, dim3(pgrid), dim3(256), plds, st, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (on_mfma) {
        const size_t lds = static_cast<size_t>(2) * 16 * kMoeTpw * szl_stride(d_in / w[0].G) * 2;
        // quantization groups a 128-code block can meet (see the kernel)
        const int G = w[0].G;
        if (G % 128 == 0)
            hipLaunchKernelGGL((moe_mfma_kernel<kMoeTpw, kMoeNbuf, 1>), dim3(blk_end), dim3(256), lds, st, a);
        else if (G % 64 == 0)
            hipLaunchKernelGGL((moe_mfma_kernel<kMoeTpw, 1, 2>), dim3(blk_end), dim3(256), lds, st, a);
        else
            hipLaunchKernelGGL((moe_mfma_kernel<kMoeTpw, 1, 4>), dim3(blk_end), dim3(256), lds, st, a);
        return hipGetLastError();
    }
    return bits == 4 ? launch_moe2<4>(a, lg, nb, many, blk_end, threads, st)
                     : launch_moe2<2>(a, lg, nb, many, blk_end, threads, st);
}

hipError_t moe_take_routing_error(hipStream_t st, unsigned long long* word) {
    unsigned long long v = 0;
    hipError_t e = hipMemcpyFromSymbolAsync(&v, HIP_SYMBOL(moe_routing_error), sizeof(v), 0,
                                            hipMemcpyDeviceToHost, st);
    if (e == hipSuccess) e = hipStreamSynchronize(st);
    if (e == hipSuccess && v) {
        const unsigned long long zero = 0;
        e = hipMemcpyToSymbolAsync(HIP_SYMBOL(moe_routing_error), &zero, sizeof(zero), 0, hipMemcpyHostToDevice,
                                   st);
        if (e == hipSuccess) e = hipStreamSynchronize(st);
    }
    *word = v;
    return e;
}

}  // namespace cl
