// Host-side launchers shared between the ABI layer (api.hip) and the kernel
// translation units.  Arguments reaching these functions are already
// validated; each returns the hipError_t of its launch.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace cl {

struct QW {                    // packed backbone, validated
    const uint32_t* q;
    const uint16_t* s;
    const uint16_t* z;
    int d_out, d_in, bits, G;
};

struct LR {                    // compensation factors, validated (rank may be 0)
    const uint16_t* A;
    const uint16_t* B;
    int r_max, rank;
};

hipError_t launch_quantize_pack(const float* W, int d_out, int d_in, int bits, int G, uint32_t* q,
                                uint16_t* s, uint16_t* z, hipStream_t st);
hipError_t launch_dequantize(const QW& w, float* out, hipStream_t st);

// Decode of a window of n (1..8) linears sharing d_in, bits, group size and
// the activations x; arguments already validated.  glu: n = 2 linears of the
// same d_out (gate, up) and one output y[0] = SiLU(gate x) * (up x).
size_t decode_workspace_bytes(int n, const QW* w, const LR* c, int T);
bool decode_fits(const QW& w);   // d_in within the kernel's K-slice limit
hipError_t launch_linear_decode(int n, const QW* w, const LR* c, const void* x, int T, int act,
                                void* const* y, int out, void* ws, hipStream_t st, bool glu = false);

// Prefill: T = X A^T into the workspace, then the MFMA GEMM with the rank
// fold; d_in must be a multiple of 64.
size_t prefill_workspace_bytes(const QW& w, const LR& c, int M);
hipError_t launch_linear_prefill(const QW& w, const LR& c, const void* X, int M, int act, void* Y, int out,
                                 void* ws, hipStream_t st);

// Compensation factors from the SVD of W - deq(Q) (fp64 Gram + Jacobi);
// synchronizes the stream once per Jacobi sweep.  hipErrorNotReady: no
// convergence within the sweep limit.
bool comp_fits(int d_out, int d_in);
size_t comp_workspace_bytes(int d_out, int d_in, int r_max);
hipError_t launch_build_compensation(const float* W, const QW& w, int r_max, uint16_t* A, uint16_t* B, float* sigma,
                                     void* ws, hipStream_t st, int* sweeps_out);

// MoE decode over stacked experts (expert e's arrays at e times one expert's
// size) for a window of n <= 4 linears sharing the routing and activations;
// arguments already validated.
bool moe_fits(const QW& w, int E, int T, int k);
size_t moe_workspace_bytes(int n, const QW* w, const int* r_max, int E, int T, int k, int x_per_slot);
hipError_t launch_moe_decode(int n, const QW* w, const uint16_t* const* A, const uint16_t* const* B,
                             const int* r_max, const int32_t* const* ranks, const int32_t* const* slot_ranks,
                             int E, const void* x, const void* u, int x_per_slot,
                             const int32_t* ids, int T, int k, int act, void* const* y, int out, void* ws,
                             hipStream_t st);

// The current device's routing-error record (see moe.hip): waits for the
// stream, returns the record in *word (0: none) and clears it.
hipError_t moe_take_routing_error(hipStream_t st, unsigned long long* word);

// Rank allocation (host code, ranks.hip): salient-set size and salience
// ratio of one descending spectrum; ranks of one compensation window (cont,
// if not null, receives the continuous ranks before alignment); layer scores
// from layer-level sensitivities.  Arguments already validated.
constexpr int kMaxRankWin = 64;
constexpr int kMaxLayers = 4096;
int salient_count(const float* sigma, int n, double tau, double* phi);
void allocate_window_ranks(int n, const float* const* sigma, const int* len, const double* sens, double layer_score,
                           double r_std, const int* levels, int nlevels, int r_max, double tau, int* ranks,
                           double* cont);
void layer_sensitivity(int L, const double* D, int K, double* S);

}  // namespace cl
