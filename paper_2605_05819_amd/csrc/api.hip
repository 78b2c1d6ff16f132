// C ABI of the compensated quantized linear: argument validation, workspace
// sizing, error reporting and dispatch to the gfx950 kernels.  Nothing here
// touches the HIP runtime before every argument has been checked, so invalid
// calls return an error without enqueuing work (and without needing a GPU).

#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <mutex>

#include "../../include/cl.h"
#include "cl_internal.h"

namespace {

thread_local char g_err[512] = "no error";
// Jacobi sweeps of the calling thread's last cl_build_compensation call
thread_local int g_last_sweeps = 0;

cl_status fail(cl_status code, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof(g_err), fmt, ap);
    va_end(ap);
    return code;
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

cl_status check_shape(int d_out, int d_in, int bits, int G, const char* who) {
    if (bits != 2 && bits != 3 && bits != 4)
        return fail(CL_EUNSUPPORTED, "%s: bits must be 2, 3 or 4 (got %d)", who, bits);
    if (d_out <= 0 || d_in <= 0) return fail(CL_EINVAL, "%s: d_out and d_in must be positive", who);
    // codes of one run never straddle two groups: a 16-byte run at 2 and 4
    // bits, a 3-word run of 32 codes at 3 bits
    const int run = bits == 3 ? 32 : 128 / bits;
    if (G <= 0 || G % run) return fail(CL_EINVAL, "%s: group_size must be a positive multiple of %d for %d-bit codes (got %d)", who, run, bits, G);
    if (d_in % G) return fail(CL_EINVAL, "%s: d_in (%d) must be a multiple of group_size (%d)", who, d_in, G);
    // rows of 3-bit codes stay 16-byte aligned: d_in * 3 / 8 bytes per row
    if (bits == 3 && d_in % 128)
        return fail(CL_EINVAL, "%s: d_in must be a multiple of 128 for 3-bit codes (got %d)", who, d_in);
    return CL_OK;
}

cl_status check_qweight(const cl_qweight* w, cl::QW* out, const char* who) {
    if (!w) return fail(CL_EINVAL, "%s: null weight descriptor", who);
    cl_status st = check_shape(w->d_out, w->d_in, w->bits, w->group_size, who);
    if (st) return st;
    if (!w->q || !w->scales || !w->zeros) return fail(CL_EINVAL, "%s: null q/scales/zeros pointer", who);
    if (!aligned(w->q, 16)) return fail(CL_EINVAL, "%s: q must be 16-byte aligned", who);
    if (!aligned(w->scales, 2) || !aligned(w->zeros, 2)) return fail(CL_EINVAL, "%s: scales/zeros must be 2-byte aligned", who);
    *out = {w->q, w->scales, w->zeros, w->d_out, w->d_in, w->bits, w->group_size};
    return CL_OK;
}

cl_status check_lowrank(const cl_lowrank* c, const cl::QW& w, cl::LR* out, const char* who) {
    *out = {nullptr, nullptr, 0, 0};
    if (!c) return CL_OK;   // no compensation
    if (c->rank < 0 || c->r_max < 0 || c->rank > c->r_max || c->r_max > 256)
        return fail(CL_EINVAL, "%s: need 0 <= rank <= r_max <= 256 (rank %d, r_max %d)", who, c->rank, c->r_max);
    if (c->rank == 0) return CL_OK;
    if (!c->A || !c->B) return fail(CL_EINVAL, "%s: null A or B with rank %d", who, c->rank);
    if (!aligned(c->A, 16)) return fail(CL_EINVAL, "%s: A must be 16-byte aligned", who);
    if (!aligned(c->B, 2)) return fail(CL_EINVAL, "%s: B must be 2-byte aligned", who);
    (void)w;
    *out = {c->A, c->B, c->r_max, c->rank};
    return CL_OK;
}

cl_status hip_status(hipError_t e, const char* who) {
    if (e == hipSuccess) return CL_OK;
    return fail(CL_EHIP, "%s: HIP error %d (%s)", who, static_cast<int>(e), hipGetErrorString(e));
}

}  // namespace

extern "C" {

const char* cl_last_error(void) { return g_err; }

cl_status cl_quantize_pack(const float* W, int32_t d_out, int32_t d_in, int32_t bits, int32_t group_size,
                           uint32_t* q, uint16_t* scales, uint16_t* zeros, void* stream) {
    const char* who = "cl_quantize_pack";
    cl_status st = check_shape(d_out, d_in, bits, group_size, who);
    if (st) return st;
    if (!W || !q || !scales || !zeros) return fail(CL_EINVAL, "%s: null pointer argument", who);
    if (!aligned(W, 4) || !aligned(q, 16) || !aligned(scales, 2) || !aligned(zeros, 2))
        return fail(CL_EINVAL, "%s: misaligned buffer (W 4, q 16, scales/zeros 2 bytes)", who);
    return hip_status(cl::launch_quantize_pack(W, d_out, d_in, bits, group_size, q, scales, zeros,
                                               static_cast<hipStream_t>(stream)), who);
}

cl_status cl_dequantize(const cl_qweight* w, float* W_hat, void* stream) {
    const char* who = "cl_dequantize";
    cl::QW qw;
    cl_status st = check_qweight(w, &qw, who);
    if (st) return st;
    if (!W_hat || !aligned(W_hat, 4)) return fail(CL_EINVAL, "%s: null or misaligned output", who);
    return hip_status(cl::launch_dequantize(qw, W_hat, static_cast<hipStream_t>(stream)), who);
}

int32_t cl_build_compensation_sweeps(void) { return g_last_sweeps; }

size_t cl_build_compensation_workspace(int32_t d_out, int32_t d_in, int32_t r_max) {
    const int n = d_in <= d_out ? d_in : d_out;
    if (d_out < 1 || d_in < 1 || r_max < 0 || r_max > 256 || r_max > n || !cl::comp_fits(d_out, d_in)) return 0;
    return cl::comp_workspace_bytes(d_out, d_in, r_max);
}

cl_status cl_build_compensation(const float* W, const cl_qweight* w, int32_t r_max, uint16_t* A, uint16_t* B,
                                float* sigma, void* ws, size_t ws_bytes, void* stream) {
    const char* who = "cl_build_compensation";
    cl::QW qw;
    cl_status st = check_qweight(w, &qw, who);
    if (st) return st;
    const int n = qw.d_in <= qw.d_out ? qw.d_in : qw.d_out;
    if (!cl::comp_fits(qw.d_out, qw.d_in))
        return fail(CL_EUNSUPPORTED, "%s: min(d_out, d_in) must be <= 8192 and d_out * d_in <= 2^31", who);
    if (r_max < 0 || r_max > 256 || r_max > n)
        return fail(CL_EINVAL, "%s: r_max must be in 0..min(256, d_out, d_in) (got %d)", who, r_max);
    if (!W || !aligned(W, 4)) return fail(CL_EINVAL, "%s: null or misaligned W", who);
    if (r_max > 0 && (!A || !B || !aligned(A, 2) || !aligned(B, 2)))
        return fail(CL_EINVAL, "%s: null or misaligned A or B", who);
    if (sigma && !aligned(sigma, 4)) return fail(CL_EINVAL, "%s: misaligned sigma", who);
    const size_t need = cl::comp_workspace_bytes(qw.d_out, qw.d_in, r_max);
    if (!ws || ws_bytes < need)
        return fail(CL_EWORKSPACE, "%s: workspace of %zu bytes needed (got %zu)", who, need, ws ? ws_bytes : 0);
    if (!aligned(ws, 256)) return fail(CL_EINVAL, "%s: workspace must be 256-byte aligned", who);
    int sweeps = 0;
    const hipError_t e = cl::launch_build_compensation(W, qw, r_max, A, B, sigma, ws,
                                                       static_cast<hipStream_t>(stream), &sweeps);
    // the loop stops at the first sweep without rotations: count it
    g_last_sweeps = e == hipSuccess ? sweeps + 1 : sweeps;
    if (e == hipErrorNotReady)
        return fail(CL_EUNSUPPORTED, "%s: the Jacobi eigensolver did not converge in %d sweeps", who, sweeps);
    return hip_status(e, who);
}

}  // extern "C"

namespace {

// Validate a window of n linears (c may be NULL: no compensation anywhere).
cl_status check_window(int32_t n, const cl_qweight* w, const cl_lowrank* c, cl::QW* qw, cl::LR* lr,
                       const char* who) {
    if (n < 1 || n > 8) return fail(CL_EINVAL, "%s: a window holds 1..8 linears (got %d)", who, n);
    if (!w) return fail(CL_EINVAL, "%s: null weight descriptor array", who);
    for (int i = 0; i < n; ++i) {
        cl_status st = check_qweight(&w[i], &qw[i], who);
        if (st) return st;
        if (qw[i].d_in != qw[0].d_in || qw[i].bits != qw[0].bits || qw[i].G != qw[0].G)
            return fail(CL_EINVAL, "%s: linears of one window must share d_in, bits and group_size", who);
        st = check_lowrank(c ? &c[i] : nullptr, qw[i], &lr[i], who);
        if (st) return st;
    }
    if (!cl::decode_fits(qw[0]))
        return fail(CL_EUNSUPPORTED, "%s: d_in %d exceeds the decode kernel's limit", who, qw[0].d_in);
    return CL_OK;
}

// Scratch of the no-allocation decode entry point: one array per device,
// held until the process ends.  In host code `scratch` names a host-side
// stand-in, not device memory: its device address comes from
// hipGetSymbolAddress, once per device with that device current, and only
// that address is ever handed to a kernel.
constexpr int kMaxDevices = 64;
static __device__ __align__(256) unsigned char scratch[CL_NOALLOC_SCRATCH_BYTES];
std::mutex g_scratch_mu;
void* g_scratch_dev[kMaxDevices];

hipError_t scratch_address(void** out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_dev[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        g_scratch_dev[dev] = p;
    }
    *out = g_scratch_dev[dev];
    return hipSuccess;
}

// ws == nullptr with noalloc: the call runs on the device's scratch array
cl_status decode_common(int32_t n, const cl_qweight* w, const cl_lowrank* c, const void* x, int32_t T,
                        int32_t act_dtype, void* const* y, int32_t out_dtype, void* ws, size_t ws_bytes,
                        void* stream, const char* who, bool glu = false, bool noalloc = false) {
    cl::QW qw[8];
    cl::LR lr[8];
    cl_status st = check_window(n, w, c, qw, lr, who);
    if (st) return st;
    if (glu && qw[0].d_out != qw[1].d_out)
        return fail(CL_EINVAL, "%s: gate and up differ in d_out (%d, %d)", who, qw[0].d_out, qw[1].d_out);
    if (T < 1 || T > 64) return fail(CL_EINVAL, "%s: T must be in 1..64 (got %d)", who, T);
    if (act_dtype != CL_FP16 && act_dtype != CL_BF16)
        return fail(CL_EINVAL, "%s: act_dtype must be CL_FP16 or CL_BF16", who);
    if (out_dtype != CL_FP16 && out_dtype != CL_BF16 && out_dtype != CL_FP32)
        return fail(CL_EINVAL, "%s: out_dtype must be CL_FP16, CL_BF16 or CL_FP32", who);
    const char* out = glu ? "h" : "y";
    if (!x || !y) return fail(CL_EINVAL, "%s: null x or %s", who, out);
    if (!aligned(x, 16)) return fail(CL_EINVAL, "%s: x must be 16-byte aligned", who);
    for (int i = 0; i < n; ++i) {
        if (!y[i]) return fail(CL_EINVAL, "%s: null %s", who, out);
        if (!aligned(y[i], out_dtype == CL_FP32 ? 4 : 2)) return fail(CL_EINVAL, "%s: misaligned %s", who, out);
    }
    const size_t need = cl::decode_workspace_bytes(n, qw, lr, T);
    if (noalloc) {
        if (need > CL_NOALLOC_SCRATCH_BYTES)
            return fail(CL_EWORKSPACE, "%s: this call needs %zu bytes of scratch; the no-allocation entry point "
                        "holds %zu per device (use cl_linear_decode with a workspace)", who, need,
                        static_cast<size_t>(CL_NOALLOC_SCRATCH_BYTES));
        const hipError_t e = scratch_address(&ws);
        if (e != hipSuccess) return hip_status(e, who);
    } else {
        if (!ws || ws_bytes < need)
            return fail(CL_EWORKSPACE, "%s: workspace of %zu bytes needed (got %zu)", who, need, ws ? ws_bytes : 0);
        if (!aligned(ws, 256)) return fail(CL_EINVAL, "%s: workspace must be 256-byte aligned", who);
    }
    return hip_status(cl::launch_linear_decode(n, qw, lr, x, T, act_dtype, y, out_dtype, ws,
                                               static_cast<hipStream_t>(stream), glu), who);
}

size_t window_workspace(int32_t n, const cl_qweight* w, const cl_lowrank* c, int32_t tokens) {
    char saved[sizeof(g_err)];
    memcpy(saved, g_err, sizeof(g_err));
    cl::QW qw[8];
    cl::LR lr[8];
    size_t bytes = 0;
    if (tokens >= 1 && tokens <= 64 && check_window(n, w, c, qw, lr, "") == CL_OK)
        bytes = cl::decode_workspace_bytes(n, qw, lr, tokens);
    memcpy(g_err, saved, sizeof(g_err));   // a size query leaves the last error alone
    return bytes;
}

}  // namespace

extern "C" {

size_t cl_linear_workspace(const cl_qweight* w, const cl_lowrank* c, int32_t tokens) {
    return window_workspace(1, w, c, tokens);
}

size_t cl_linear_window_workspace(int32_t n, const cl_qweight* w, const cl_lowrank* c, int32_t tokens) {
    return window_workspace(n, w, c, tokens);
}

cl_status cl_linear_decode(const cl_qweight* w, const cl_lowrank* c, const void* x, int32_t T,
                           int32_t act_dtype, void* y, int32_t out_dtype, void* ws, size_t ws_bytes,
                           void* stream) {
    void* ys[1] = {y};
    return decode_common(1, w, c, x, T, act_dtype, y ? ys : nullptr, out_dtype, ws, ws_bytes, stream,
                         "cl_linear_decode");
}

cl_status cl_linear_decode_noalloc(const cl_qweight* w, const cl_lowrank* c, const void* x, int32_t T,
                                   int32_t act_dtype, void* y, int32_t out_dtype, void* stream) {
    void* ys[1] = {y};
    return decode_common(1, w, c, x, T, act_dtype, y ? ys : nullptr, out_dtype, nullptr, 0, stream,
                         "cl_linear_decode_noalloc", false, true);
}

size_t cl_prefill_workspace(const cl_qweight* w, const cl_lowrank* c, int32_t M) {
    char saved[sizeof(g_err)];
    memcpy(saved, g_err, sizeof(g_err));
    cl::QW qw;
    cl::LR lr;
    size_t bytes = 0;
    if (M >= 1 && check_qweight(w, &qw, "") == CL_OK && check_lowrank(c, qw, &lr, "") == CL_OK)
        bytes = cl::prefill_workspace_bytes(qw, lr, M);
    memcpy(g_err, saved, sizeof(g_err));
    return bytes;
}

cl_status cl_linear_prefill(const cl_qweight* w, const cl_lowrank* c, const void* X, int32_t M, int32_t act_dtype,
                            void* Y, int32_t out_dtype, void* ws, size_t ws_bytes, void* stream) {
    const char* who = "cl_linear_prefill";
    cl::QW qw;
    cl::LR lr;
    cl_status st = check_qweight(w, &qw, who);
    if (st) return st;
    st = check_lowrank(c, qw, &lr, who);
    if (st) return st;
    if (qw.d_in % 64) return fail(CL_EUNSUPPORTED, "%s: d_in must be a multiple of 64 (got %d)", who, qw.d_in);
    if (M < 1) return fail(CL_EINVAL, "%s: M must be >= 1 (got %d)", who, M);
    if (static_cast<long long>(M) * qw.d_in > (1ll << 31) - 1)
        return fail(CL_EUNSUPPORTED, "%s: M * d_in must be below 2^31 (split the tokens)", who);
    if (act_dtype != CL_FP16 && act_dtype != CL_BF16)
        return fail(CL_EINVAL, "%s: act_dtype must be CL_FP16 or CL_BF16", who);
    if (out_dtype != CL_FP16 && out_dtype != CL_BF16 && out_dtype != CL_FP32)
        return fail(CL_EINVAL, "%s: out_dtype must be CL_FP16, CL_BF16 or CL_FP32", who);
    if (!X || !Y) return fail(CL_EINVAL, "%s: null X or Y", who);
    if (!aligned(X, 16)) return fail(CL_EINVAL, "%s: X must be 16-byte aligned", who);
    if (!aligned(Y, out_dtype == CL_FP32 ? 4 : 2)) return fail(CL_EINVAL, "%s: misaligned Y", who);
    const size_t need = cl::prefill_workspace_bytes(qw, lr, M);
    if (need > 0 && (!ws || ws_bytes < need))
        return fail(CL_EWORKSPACE, "%s: workspace of %zu bytes needed (got %zu)", who, need, ws ? ws_bytes : 0);
    if (need > 0 && !aligned(ws, 256)) return fail(CL_EINVAL, "%s: workspace must be 256-byte aligned", who);
    return hip_status(cl::launch_linear_prefill(qw, lr, X, M, act_dtype, Y, out_dtype, ws,
                                                static_cast<hipStream_t>(stream)), who);
}

}  // extern "C"

namespace {

// Shared validation of the MoE entry points: n linears over one routing and
// one activation tensor (same d_in, bits and group size).
cl_status moe_common(int32_t n, const cl_qweight* w, const uint16_t* const* A, const uint16_t* const* B,
                     const int32_t* r_max, const int32_t* const* ranks, const int32_t* const* slot_ranks,
                     int32_t num_experts, const void* x, const void* u,
                     int32_t x_per_slot, const int32_t* topk_ids, int32_t T, int32_t k, int32_t act_dtype,
                     void* const* y, int32_t out_dtype, void* ws, size_t ws_bytes, void* stream, const char* who) {
    if (n < 1 || n > 4) return fail(CL_EINVAL, "%s: n must be in 1..4 (got %d)", who, n);
    if (!w || !A || !B || !r_max || !ranks || !y) return fail(CL_EINVAL, "%s: null argument array", who);
    cl::QW qw[4];
    int rm[4];
    for (int i = 0; i < n; ++i) {
        cl_status st = check_qweight(&w[i], &qw[i], who);
        if (st) return st;
        if (qw[i].d_in != qw[0].d_in || qw[i].bits != qw[0].bits || qw[i].G != qw[0].G)
            return fail(CL_EINVAL, "%s: the linears of a window must share d_in, bits and group size", who);
        if (qw[i].bits == 3) return fail(CL_EUNSUPPORTED, "%s: 3-bit codes run on the dense decode entry points only", who);
        if (r_max[i] < 0 || r_max[i] > 256) return fail(CL_EINVAL, "%s: r_max must be in 0..256", who);
        if (r_max[i] > 0) {
            if (!A[i] || !B[i] || !ranks[i]) return fail(CL_EINVAL, "%s: null A, B or ranks with r_max %d", who, r_max[i]);
            if (!aligned(A[i], 16) || !aligned(B[i], 2) || !aligned(ranks[i], 4))
                return fail(CL_EINVAL, "%s: A must be 16-byte, B 2-byte, ranks 4-byte aligned", who);
        }
        if (slot_ranks && slot_ranks[i] && !aligned(slot_ranks[i], 4))
            return fail(CL_EINVAL, "%s: slot_ranks must be 4-byte aligned", who);
        if (!y[i]) return fail(CL_EINVAL, "%s: null y", who);
        if (!aligned(y[i], out_dtype == CL_FP32 ? 4 : 2)) return fail(CL_EINVAL, "%s: misaligned y", who);
        rm[i] = r_max[i];
    }
    if (num_experts < 1) return fail(CL_EINVAL, "%s: num_experts must be >= 1", who);
    if (T < 1 || T > 64) return fail(CL_EINVAL, "%s: T must be in 1..64 (got %d)", who, T);
    if (k < 1) return fail(CL_EINVAL, "%s: k must be >= 1", who);
    if (!cl::moe_fits(qw[0], num_experts, T, k))
        return fail(CL_EUNSUPPORTED, "%s: at most 1024 experts, 1024 slots (T*k) and d_in <= 8192 * bits", who);
    if (!topk_ids || !aligned(topk_ids, 4)) return fail(CL_EINVAL, "%s: null or misaligned topk_ids", who);
    if (act_dtype != CL_FP16 && act_dtype != CL_BF16)
        return fail(CL_EINVAL, "%s: act_dtype must be CL_FP16 or CL_BF16", who);
    if (out_dtype != CL_FP16 && out_dtype != CL_BF16 && out_dtype != CL_FP32)
        return fail(CL_EINVAL, "%s: out_dtype must be CL_FP16, CL_BF16 or CL_FP32", who);
    if (!x) return fail(CL_EINVAL, "%s: null x", who);
    if (!aligned(x, 16)) return fail(CL_EINVAL, "%s: x must be 16-byte aligned", who);
    if (u && !aligned(u, 16)) return fail(CL_EINVAL, "%s: u must be 16-byte aligned", who);
    const int xs = u ? 2 : (x_per_slot ? 1 : 0);       // 2: gated per-slot input
    const size_t need = cl::moe_workspace_bytes(n, qw, rm, num_experts, T, k, xs);
    if (!ws || ws_bytes < need)
        return fail(CL_EWORKSPACE, "%s: workspace of %zu bytes needed (got %zu)", who, need, ws ? ws_bytes : 0);
    if (!aligned(ws, 256)) return fail(CL_EINVAL, "%s: workspace must be 256-byte aligned", who);
    return hip_status(cl::launch_moe_decode(n, qw, A, B, rm, ranks, slot_ranks, num_experts, x, u, xs, topk_ids, T, k,
                                            act_dtype,
                                            y, out_dtype, ws, static_cast<hipStream_t>(stream)),
                      who);
}

size_t moe_ws(int32_t n, const cl_qweight* w, const int32_t* r_max, int32_t num_experts, int32_t T, int32_t k,
              int32_t x_per_slot) {
    char saved[sizeof(g_err)];
    memcpy(saved, g_err, sizeof(g_err));
    size_t bytes = 0;
    cl::QW qw[4];
    int rm[4];
    bool ok = n >= 1 && n <= 4 && w && r_max && num_experts >= 1 && T >= 1 && T <= 64 && k >= 1;
    for (int i = 0; ok && i < n; ++i) {
        ok = check_qweight(&w[i], &qw[i], "") == CL_OK && qw[i].bits != 3 && r_max[i] >= 0 && r_max[i] <= 256 &&
             qw[i].d_in == qw[0].d_in && qw[i].bits == qw[0].bits && qw[i].G == qw[0].G;
        rm[i] = ok ? r_max[i] : 0;
    }
    if (ok && cl::moe_fits(qw[0], num_experts, T, k))
        bytes = cl::moe_workspace_bytes(n, qw, rm, num_experts, T, k, x_per_slot);
    memcpy(g_err, saved, sizeof(g_err));
    return bytes;
}

}  // namespace

extern "C" {

size_t cl_moe_workspace(const cl_qweight* w_expert0, int32_t r_max, int32_t num_experts, int32_t T, int32_t k,
                        int32_t x_per_slot) {
    return moe_ws(1, w_expert0, &r_max, num_experts, T, k, x_per_slot ? 1 : 0);
}

size_t cl_moe_gated_workspace(const cl_qweight* w_expert0, int32_t r_max, int32_t num_experts, int32_t T,
                              int32_t k) {
    return moe_ws(1, w_expert0, &r_max, num_experts, T, k, 2);
}

size_t cl_moe_window_workspace(int32_t n, const cl_qweight* w_expert0, const int32_t* r_max, int32_t num_experts,
                               int32_t T, int32_t k, int32_t x_per_slot) {
    return moe_ws(n, w_expert0, r_max, num_experts, T, k, x_per_slot ? 1 : 0);
}

cl_status cl_moe_linear_decode(const cl_qweight* w_expert0, const uint16_t* A, const uint16_t* B, int32_t r_max,
                               const int32_t* ranks, int32_t num_experts, const void* x, int32_t x_per_slot,
                               const int32_t* topk_ids, int32_t T, int32_t k, int32_t act_dtype, void* y,
                               int32_t out_dtype, void* ws, size_t ws_bytes, void* stream) {
    return moe_common(1, w_expert0, &A, &B, &r_max, &ranks, nullptr, num_experts, x, nullptr, x_per_slot, topk_ids,
                      T, k, act_dtype, &y, out_dtype, ws, ws_bytes, stream, "cl_moe_linear_decode");
}

cl_status cl_moe_linear_decode_gated(const cl_qweight* w_expert0, const uint16_t* A, const uint16_t* B,
                                     int32_t r_max, const int32_t* ranks, const int32_t* slot_ranks,
                                     int32_t num_experts, const void* g, const void* u, const int32_t* topk_ids,
                                     int32_t T, int32_t k, int32_t act_dtype, void* y, int32_t out_dtype, void* ws,
                                     size_t ws_bytes, void* stream) {
    const char* who = "cl_moe_linear_decode_gated";
    if (!g || !u) return fail(CL_EINVAL, "%s: null g or u", who);
    return moe_common(1, w_expert0, &A, &B, &r_max, &ranks, &slot_ranks, num_experts, g, u, 1, topk_ids, T, k,
                      act_dtype, &y, out_dtype, ws, ws_bytes, stream, who);
}

cl_status cl_moe_linear_decode_window(int32_t n, const cl_qweight* w_expert0, const uint16_t* const* A,
                                      const uint16_t* const* B, const int32_t* r_max, const int32_t* const* ranks,
                                      const int32_t* const* slot_ranks, int32_t num_experts, const void* x,
                                      int32_t x_per_slot,
                                      const int32_t* topk_ids, int32_t T, int32_t k, int32_t act_dtype,
                                      void* const* y, int32_t out_dtype, void* ws, size_t ws_bytes, void* stream) {
    return moe_common(n, w_expert0, A, B, r_max, ranks, slot_ranks, num_experts, x, nullptr, x_per_slot, topk_ids,
                      T, k, act_dtype, y, out_dtype, ws, ws_bytes, stream, "cl_moe_linear_decode_window");
}

cl_status cl_linear_decode_window(int32_t n, const cl_qweight* w, const cl_lowrank* c, const void* x,
                                  int32_t T, int32_t act_dtype, void* const* y, int32_t out_dtype, void* ws,
                                  size_t ws_bytes, void* stream) {
    return decode_common(n, w, c, x, T, act_dtype, y, out_dtype, ws, ws_bytes, stream,
                         "cl_linear_decode_window");
}

cl_status cl_allocate_ranks(int32_t n, const float* const* sigma, const int32_t* len, const double* sens,
                            double layer_score, double r_std, const int32_t* levels, int32_t nlevels, int32_t r_max,
                            double tau, int32_t* ranks) {
    const char* who = "cl_allocate_ranks";
    if (n < 1 || n > cl::kMaxRankWin) return fail(CL_EINVAL, "%s: n must be in 1..%d (got %d)", who, cl::kMaxRankWin, n);
    if (!sigma || !len || !sens || !levels || !ranks) return fail(CL_EINVAL, "%s: null argument", who);
    if (!(layer_score >= 0.0) || !isfinite(layer_score) || !(r_std >= 0.0) || !isfinite(r_std))
        return fail(CL_EINVAL, "%s: layer_score and r_std must be finite and >= 0", who);
    if (!(tau >= 0.0) || !isfinite(tau)) return fail(CL_EINVAL, "%s: tau must be finite and >= 0", who);
    if (r_max < 0) return fail(CL_EINVAL, "%s: r_max must be >= 0", who);
    if (nlevels < 1 || nlevels > 64 || levels[0] != 0)
        return fail(CL_EINVAL, "%s: levels must hold 1..64 values starting with 0", who);
    for (int l = 1; l < nlevels; ++l)
        if (levels[l] <= levels[l - 1]) return fail(CL_EINVAL, "%s: levels must be strictly increasing", who);
    for (int i = 0; i < n; ++i) {
        if (!sigma[i] || len[i] < 1) return fail(CL_EINVAL, "%s: spectrum %d is null or empty", who, i);
        if (!(sens[i] >= 0.0) || !isfinite(sens[i]))
            return fail(CL_EINVAL, "%s: sensitivity %d must be finite and >= 0", who, i);
        for (int j = 0; j < len[i]; ++j)
            if (!(sigma[i][j] >= 0.0f) || !isfinite(sigma[i][j]) || (j > 0 && sigma[i][j] > sigma[i][j - 1]))
                return fail(CL_EINVAL, "%s: spectrum %d must be finite, >= 0 and descending (index %d)", who, i, j);
    }
    int lens[cl::kMaxRankWin], lv[64], out[cl::kMaxRankWin];
    for (int i = 0; i < n; ++i) lens[i] = len[i];
    for (int l = 0; l < nlevels; ++l) lv[l] = levels[l];
    cl::allocate_window_ranks(n, sigma, lens, sens, layer_score, r_std, lv, nlevels, r_max, tau, out, nullptr);
    for (int i = 0; i < n; ++i) ranks[i] = out[i];
    return CL_OK;
}

cl_status cl_moe_status(void* stream) {
    const char* who = "cl_moe_status";
    unsigned long long v = 0;
    const hipError_t e = cl::moe_take_routing_error(static_cast<hipStream_t>(stream), &v);
    if (e != hipSuccess) return hip_status(e, who);
    if (v)
        return fail(CL_EINVAL, "%s: a MoE call met routing id %d in slot %d (outside 0..num_experts-1); "
                    "that slot's output row was written as zeros", who, static_cast<int32_t>(v & 0xffffffffu),
                    static_cast<int>((v >> 32) & 0x7fffffffu));
    return CL_OK;
}

cl_status cl_layer_sensitivity(int32_t L, const double* D, int32_t K, double* S) {
    const char* who = "cl_layer_sensitivity";
    if (L < 1 || L > cl::kMaxLayers) return fail(CL_EINVAL, "%s: L must be in 1..%d (got %d)", who, cl::kMaxLayers, L);
    if (K < 1 || K > L) return fail(CL_EINVAL, "%s: K must be in 1..L (got %d)", who, K);
    if (!D || !S) return fail(CL_EINVAL, "%s: null argument", who);
    for (int l = 0; l < L; ++l)
        if (!(D[l] >= 0.0) || !isfinite(D[l])) return fail(CL_EINVAL, "%s: D[%d] must be finite and >= 0", who, l);
    cl::layer_sensitivity(L, D, K, S);
    return CL_OK;
}

cl_status cl_linear_decode_glu(const cl_qweight* w, const cl_lowrank* c, const void* x, int32_t T,
                               int32_t act_dtype, void* h, int32_t out_dtype, void* ws, size_t ws_bytes,
                               void* stream) {
    void* hs[2] = {h, h};
    return decode_common(2, w, c, x, T, act_dtype, h ? hs : nullptr, out_dtype, ws, ws_bytes, stream,
                         "cl_linear_decode_glu", true);
}

}  // extern "C"
