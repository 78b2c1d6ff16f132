/*
 * cl.h -- C ABI of the error-compensated quantized linear layer for AMD
 * MI355X (gfx950).
 *
 * The layer (HCInfer, arXiv 2605.05819, Section 4.1, Theoretical Framework)
 * replaces a linear layer by a low-bit backbone plus a low-rank correction of
 * its quantization error.  With column vectors and the weight stored
 * d_out x d_in, every token x computes
 *
 *     y = deq(Q, scales, zeros) x + B[:, :r] (A[:r, :] x)
 *
 * where deq(Q, s, z)[o][c] = s[o][c/G] * (q[o][c] - z[o][c/G]) and A, B are
 * the leading factors of the SVD of W - deq(Q) (sorted by descending singular
 * value, so every prefix rank r <= r_max is the optimal rank-r correction).
 *
 * Conventions for every entry point
 * ---------------------------------
 *  - Pointers marked "device" point to device memory of the current HIP
 *    device; the caller allocates and frees all of it.  The library allocates
 *    nothing on these calls and keeps no pointer after returning.
 *  - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *    Calls only enqueue work and return; buffers must stay alive until the
 *    stream has executed it.
 *  - Descriptor structs are read during the call and may be reused at once.
 *  - Arrays are row-major and densely packed.
 *  - Arguments are validated before anything is enqueued.  On a non-zero
 *    status nothing was enqueued and cl_last_error() describes the problem.
 *    No call aborts or throws.
 *
 * Packed backbone layout (cl_qweight)
 * -----------------------------------
 *  q       uint32 [d_out][d_in * bits / 32].  2 and 4 bits: the code of
 *          column c is in word c / (32/bits) of its row at bit offset
 *          bits * (c % (32/bits)) (LSB first).  3 bits: columns 32 j ..
 *          32 j + 31 fill words 3 j .. 3 j + 2 of the row, column 32 j + i at
 *          bit offset 3 i of those 96 bits (little-endian).  16-byte aligned.
 *  scales  fp16   [d_out][d_in / group_size], the group's step size.
 *  zeros   fp16   [d_out][d_in / group_size], integer zero point 0..2^bits-1.
 *  bits in {2, 3, 4}; group_size a multiple of 128/bits at 2 and 4 bits (a
 *  16-byte run of codes never straddles two groups) and of 32 at 3 bits;
 *  d_in a multiple of group_size, and of 128 at 3 bits.
 *
 * Compensation factors (cl_lowrank)
 * ---------------------------------
 *  A  fp16 [r_max][d_in]   (rows 0..rank-1 are used)
 *  B  fp16 [d_out][r_max]  (columns 0..rank-1 of every row are used)
 *  0 <= rank <= r_max <= 256.  With rank == 0, A and B may be NULL.
 */
#ifndef CL_H_
#define CL_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t cl_status;
enum {
    CL_OK = 0,
    CL_EINVAL = 1,        /* bad argument: null pointer, bad size, misalignment */
    CL_EUNSUPPORTED = 2,  /* well-formed but not implemented (e.g. bits = 5)    */
    CL_EWORKSPACE = 3,    /* workspace missing or smaller than required         */
    CL_EHIP = 4           /* the HIP runtime reported an error at launch        */
};

/* Element types of activations and outputs. */
enum { CL_FP16 = 1, CL_BF16 = 2, CL_FP32 = 3 };

typedef struct cl_qweight {
    const uint32_t* q;        /* device */
    const uint16_t* scales;   /* device, fp16 bits */
    const uint16_t* zeros;    /* device, fp16 bits */
    int32_t d_out;
    int32_t d_in;
    int32_t bits;
    int32_t group_size;
} cl_qweight;

typedef struct cl_lowrank {
    const uint16_t* A;        /* device, fp16 bits, [r_max][d_in]  */
    const uint16_t* B;        /* device, fp16 bits, [d_out][r_max] */
    int32_t r_max;
    int32_t rank;
} cl_lowrank;

/*
 * cl_quantize_pack -- quantize a float32 weight group-wise and pack it.
 *
 * Section 5.1 quantizes the backbone with GPTQ; without calibration data GPTQ
 * is round-to-nearest on an asymmetric per-group min/max grid, computed here in
 * fp64 and bit-exact with that definition:
 *   lo = min(min w, 0), hi = max(max w, 0); an all-equal group uses [-1, 1];
 *   s16 = fp16(round-to-nearest-even((hi - lo) / (2^bits - 1))), kept within
 *         [2^-24, 65504];
 *   z = clamp(rint(-lo / s16), 0, 2^bits - 1);
 *   q = clamp(rint(w / s16) + z, 0, 2^bits - 1)   (rint: ties to even).
 *
 *  W       device float32 [d_out][d_in] (input, finite values)
 *  q       device uint32  [d_out][d_in*bits/32] (output, 16-byte aligned)
 *  scales, zeros  device fp16 [d_out][d_in/group_size] (outputs)
 * Errors: CL_EINVAL for null pointers, non-positive sizes, misaligned q or a
 * group_size / d_in that breaks the layout rules above; CL_EUNSUPPORTED for
 * bits other than 2, 3 and 4.
 */
cl_status cl_quantize_pack(const float* W, int32_t d_out, int32_t d_in, int32_t bits,
                           int32_t group_size, uint32_t* q, uint16_t* scales, uint16_t* zeros,
                           void* stream);

/*
 * cl_dequantize -- W_hat[o][c] = s[o][c/G] * (q[o][c] - z[o][c/G]) as float32
 * (exact: an fp16 step times a small integer fits float32).
 *  W_hat   device float32 [d_out][d_in] (output)
 * Errors: as cl_quantize_pack.
 */
cl_status cl_dequantize(const cl_qweight* w, float* W_hat, void* stream);

/*
 * cl_build_compensation -- compensation factors from the quantization error
 * (Section 4.1: SVD of the residual; Appendix B.2: the truncated SVD is the
 * best rank-r approximation, error = the tail singular values).  With
 * E = W - deq(q, scales, zeros) = U diag(sigma) V^T, sigma descending:
 *     A = diag(sqrt(sigma[:r_max])) V^T[:r_max],   B = U[:, :r_max] diag(sqrt(sigma[:r_max])),
 * each singular pair signed so that the largest-magnitude entry of its U
 * column is positive (first index on ties); rounded once to fp16.  Any prefix
 * rank r <= r_max of the stored factors is the optimal rank-r truncation.
 *
 *  W      device fp32 [d_out][d_in], the weight w was quantized from
 *  w      its packed backbone (as for cl_linear_decode)
 *  r_max  0..min(256, d_out, d_in)
 *  A      device fp16 [r_max][d_in] (output; may be NULL when r_max = 0)
 *  B      device fp16 [d_out][r_max] (output; may be NULL when r_max = 0)
 *  sigma  device fp32 [min(d_out, d_in)], every singular value, descending
 *         (output; may be NULL)
 *  ws     device workspace of cl_build_compensation_workspace(...) bytes,
 *         256-byte aligned (fp64 residual, Gram matrix and eigenvectors)
 * Computed in fp64 from the Gram matrix of E over its smaller side with a
 * parallel cyclic Jacobi eigensolver; singular values far below
 * 1e-8 * sigma[0] have absolute accuracy only.  An offline step: the call
 * waits on the stream once per Jacobi sweep and returns when the factors are
 * enqueued.  Limits: min(d_out, d_in) <= 8192, d_out * d_in <= 2^31
 * (CL_EUNSUPPORTED beyond); CL_EUNSUPPORTED also if the eigensolver does not
 * converge in 40 sweeps.
 */
cl_status cl_build_compensation(const float* W, const cl_qweight* w, int32_t r_max, uint16_t* A, uint16_t* B,
                                float* sigma, void* ws, size_t ws_bytes, void* stream);

/* Workspace bytes for cl_build_compensation (0 for rejected sizes). */
size_t cl_build_compensation_workspace(int32_t d_out, int32_t d_in, int32_t r_max);

/*
 * Jacobi sweeps the calling thread's last cl_build_compensation call ran
 * (including the final sweep without rotations; 0 before any call).  A
 * report of the eigensolver's work, for timing and tuning.
 */
int32_t cl_build_compensation_sweeps(void);

/*
 * cl_linear_workspace -- bytes of device workspace that cl_linear_decode needs
 * for this weight, factor set (NULL for none) and token count.  Returns 0 for
 * arguments cl_linear_decode would reject.
 */
size_t cl_linear_workspace(const cl_qweight* w, const cl_lowrank* c, int32_t tokens);

/*
 * cl_linear_decode -- compensated linear for a few decode tokens (Section 4.1):
 *     y[t] = deq(Q) x[t] + B[:, :rank] (A[:rank] x[t]),   t = 0..T-1.
 * Two kernels are enqueued: a small one that forms A[:rank] x and the
 * activations in the layout the backbone consumes (in the workspace), then
 * one memory-bound kernel that unpacks, dequantizes and multiplies the
 * backbone and folds in the rank-r up-projection B t.  Accumulation is
 * float32; the result is rounded once to out_dtype.  t = A x is float32 for
 * one and two tokens; from three tokens (the MFMA backbone) it enters the
 * contraction as an fp16 pair hi + lo (about 2^-22 relative), so |A x| must
 * stay below 65504, and below 2^-14 it keeps fp16's subnormal resolution
 * (2^-25 absolute).
 *
 *  w, c       the packed backbone and its factors (c may be NULL for rank 0)
 *  x          device [T][d_in] of act_dtype (CL_FP16 or CL_BF16), 16-byte
 *             aligned.  bf16 activations are read as fp16: exact for
 *             2^-17 <= |x| <= 65504, rounded to a multiple of 2^-24 below
 *             that range and saturated above it.
 *  T          1..64 tokens
 *  y          device [T][d_out] of out_dtype (CL_FP16, CL_BF16 or CL_FP32)
 *  ws         device workspace of at least cl_linear_workspace(w, c, T) bytes,
 *             256-byte aligned.  It receives A x and the prepared
 *             activations; calls that may overlap must use separate
 *             workspaces.
 * Errors: CL_EINVAL / CL_EUNSUPPORTED for bad descriptors, dtypes or T,
 * CL_EWORKSPACE for a missing or short workspace, CL_EHIP on launch failure.
 */
cl_status cl_linear_decode(const cl_qweight* w, const cl_lowrank* c, const void* x, int32_t T,
                           int32_t act_dtype, void* y, int32_t out_dtype, void* ws,
                           size_t ws_bytes, void* stream);

/*
 * cl_linear_decode_noalloc -- cl_linear_decode for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation): the same kernels and the same result,
 * bit for bit, with the workspace taken from a scratch array the library
 * holds on each device instead of a caller's buffer.  The call allocates
 * nothing; on its first call on a device it looks up that device's array.
 *
 *  w, c, x, T, act_dtype, y, out_dtype, stream  as cl_linear_decode
 * The scratch holds CL_NOALLOC_SCRATCH_BYTES per device (enough for T <= 64,
 * d_in <= 16384 and rank <= 256); a call needing more (cl_linear_workspace
 * of its arguments) returns CL_EWORKSPACE.  Every call on a device uses the
 * same array and overwrites what the last call left there (nothing in it
 * needs to start at zero), so calls that may overlap on one device -- on
 * different streams, or from different threads -- race; serialize them.
 * Errors: as cl_linear_decode.
 */
#define CL_NOALLOC_SCRATCH_BYTES (4u << 20)
cl_status cl_linear_decode_noalloc(const cl_qweight* w, const cl_lowrank* c, const void* x, int32_t T,
                                   int32_t act_dtype, void* y, int32_t out_dtype, void* stream);

/*
 * cl_linear_decode_window -- one compensation window: n linears that read the
 * same activations x, each with its own backbone, factors and output.  The
 * paper groups the Q, K and V projections, and the gate and up projections,
 * into such windows so they share one hand-off of the activations and one
 * compensation pass (Section 4.2.2, Communication Fusion; Appendix A.1).
 * Here a window costs one A x / activation-preparation launch and one
 * backbone launch over all n matrices; each output equals what
 * cl_linear_decode would give for that linear alone (bitwise).
 *
 *  n          1..8 linears, all with the same d_in, bits and group_size
 *  w          host array of n weight descriptors
 *  c          host array of n factor descriptors (rank 0 allowed), or NULL
 *             for no compensation at all
 *  x          device [T][d_in] of act_dtype, 16-byte aligned (as above)
 *  y          host array of n device pointers, y[i] is [T][w[i].d_out]
 *  ws         device workspace of cl_linear_window_workspace(n, w, c, T)
 *             bytes, 256-byte aligned
 * Errors: as cl_linear_decode, and CL_EINVAL for n outside 1..8 or linears
 * that differ in d_in, bits or group_size.
 */
cl_status cl_linear_decode_window(int32_t n, const cl_qweight* w, const cl_lowrank* c, const void* x,
                                  int32_t T, int32_t act_dtype, void* const* y, int32_t out_dtype,
                                  void* ws, size_t ws_bytes, void* stream);

/* Workspace bytes for cl_linear_decode_window (0 for arguments it would reject). */
size_t cl_linear_window_workspace(int32_t n, const cl_qweight* w, const cl_lowrank* c, int32_t tokens);

/*
 * cl_linear_decode_glu -- the gate/up window of a gated MLP with its
 * elementwise epilogue fused into the backbone launch:
 *     h = SiLU(g) * u,  g = gate(x), u = up(x),  SiLU(v) = v / (1 + e^-v),
 * each of g and u the compensated linear of cl_linear_decode (Section 4.1)
 * taken as one window (Section 4.2.2, Communication Fusion).  g and u stay in
 * fp32 registers: the epilogue is applied to them unrounded and h is rounded
 * once to out_dtype; neither g nor u is written to memory.
 *
 *  w          host array {gate, up}: same d_in, d_out, bits and group_size
 *  c          host array {gate factors, up factors} (rank 0 allowed), or NULL
 *  x          device [T][d_in] of act_dtype, 16-byte aligned
 *  h          device [T][d_out] of out_dtype
 *  ws         device workspace of cl_linear_window_workspace(2, w, c, T)
 *             bytes, 256-byte aligned
 * Errors: as cl_linear_decode_window with n = 2, and CL_EINVAL when gate and
 * up differ in d_out.
 */
cl_status cl_linear_decode_glu(const cl_qweight* w, const cl_lowrank* c, const void* x, int32_t T,
                               int32_t act_dtype, void* h, int32_t out_dtype, void* ws, size_t ws_bytes,
                               void* stream);

/*
 * cl_linear_prefill -- compensated linear for many tokens (Section 4.1):
 *     Y = X deq(Q)^T + (X A[:rank]^T) B[:, :rank]^T.
 * A dense contraction on MFMA: a first kernel writes X' (X as fp16 in the
 * k order the code unpack produces, into the workspace) and, with a rank
 * term, T = X A^T (fp16, in the workspace); then one GEMM streams X' tiles
 * into LDS, dequantizes the weight codes in registers (fp16 s * (q - z), one
 * rounding per weight), multiplies on v_mfma_f32_16x16x32_f16 with float32
 * accumulation, folds the rank-r term in as extra K steps over [T | B] into
 * the same output tile and rounds once to out_dtype.  bf16 activations are
 * converted to fp16 (exact for 2^-17 <= |x| <= 65504, as in
 * cl_linear_decode).  T is rounded once to fp16, so |X A^T| must stay below
 * 65504 (below 2^-14 its resolution is fp16's, 2^-25 absolute).
 *
 *  X          device [M][d_in] of act_dtype, 16-byte aligned
 *  M          >= 1 tokens, M * d_in < 2^31
 *  Y          device [M][d_out] of out_dtype
 *  ws         device workspace of cl_prefill_workspace(w, c, M) bytes
 *             (2 M128 d_in for X', M128 the tokens rounded up to 128;
 *             2 M r32 for T, r32 the rank rounded up to 32; with a rank
 *             term, 4 M r32 ceil(d_in / 256) for its partial products;
 *             each part rounded up to 256 bytes), 256-byte aligned
 * Errors: as cl_linear_decode; CL_EUNSUPPORTED if d_in is not a multiple of
 * 64 or M * d_in >= 2^31.
 */
cl_status cl_linear_prefill(const cl_qweight* w, const cl_lowrank* c, const void* X, int32_t M,
                            int32_t act_dtype, void* Y, int32_t out_dtype, void* ws, size_t ws_bytes,
                            void* stream);

/* Workspace bytes for cl_linear_prefill (0 for rejected arguments). */
size_t cl_prefill_workspace(const cl_qweight* w, const cl_lowrank* c, int32_t M);

/*
 * cl_moe_linear_decode -- compensated linear of a MoE layer for a few decode
 * tokens: for every token t and routing slot j with expert e = ids[t][j],
 *     y[t][j] = deq(Q_e) x + B_e[:, :r_e] (A_e[:r_e] x),
 * x = x[t] (x_per_slot = 0, e.g. gate/up) or x[t][j] (x_per_slot = 1, e.g.
 * down).  All routed experts' same projection is processed in one step, the
 * paper's cross-expert reorganisation (Section 4.2.2; Appendix A.1, MoE
 * Layer); only routed experts' codes, scales, zeros and factors are read.
 * Two kernels are enqueued (routing + A x + activation preparation, then the
 * backbone over every routed expert).
 *
 *  w_expert0  descriptor of expert 0; experts are stacked contiguously: expert
 *             e's q, scales and zeros start e times one expert's size after
 *             expert 0's
 *  A          device fp16 [E][r_max][d_in];  B  device fp16 [E][d_out][r_max]
 *             (both may be NULL when r_max = 0)
 *  ranks      device int32 [E], expert e's rank (clamped to 0..r_max)
 *  x          device [T][d_in] or [T][k][d_in] of act_dtype, 16-byte aligned
 *  topk_ids   device int32 [T][k].  The ids are read on the device only, so
 *             an id outside 0..E-1 cannot fail the call: that slot's output
 *             row is written as zeros and the device records the slot and id;
 *             cl_moe_status() reports the record as CL_EINVAL.
 *  y          device [T][k][d_out] of out_dtype
 *  ws         device workspace of cl_moe_workspace(...) bytes, 256-byte aligned
 * Limits: E <= 1024, T in 1..64, T*k <= 1024, r_max <= 256, d_in <= 8192 * bits
 *         (16384 for 4-bit); beyond them CL_EUNSUPPORTED.
 * Errors: as cl_linear_decode.
 */
cl_status cl_moe_linear_decode(const cl_qweight* w_expert0, const uint16_t* A, const uint16_t* B,
                               int32_t r_max, const int32_t* ranks, int32_t num_experts, const void* x,
                               int32_t x_per_slot, const int32_t* topk_ids, int32_t T, int32_t k,
                               int32_t act_dtype, void* y, int32_t out_dtype, void* ws, size_t ws_bytes,
                               void* stream);

/*
 * Workspace bytes for cl_moe_linear_decode (0 for rejected arguments).  The
 * workspace holds the routing tables, A_e x per slot ([T k][r_max] float) and
 * the activations prepared for the backbone ([rows][d_in] fp16 plus
 * per-chunk sums, rows = T or T k), so the size depends on d_in, the code
 * width and x_per_slot as well as on E, T, k and r_max: the query takes the
 * expert-0 descriptor (for d_in, bits and group size) and x_per_slot.
 */
size_t cl_moe_workspace(const cl_qweight* w_expert0, int32_t r_max, int32_t num_experts, int32_t T,
                        int32_t k, int32_t x_per_slot);

/*
 * cl_moe_status -- the out-of-range routing ids that MoE calls met on the
 * current device (Section 4.2.2's cross-expert grouping reads the routing
 * table on the device; see topk_ids above).  Waits for `stream` (work
 * enqueued on other streams is not waited for), then reads and clears the
 * device's record: CL_OK if no MoE call met an id outside 0..E-1 since the
 * record was last read, else CL_EINVAL with the slot and id of one such
 * entry in cl_last_error().  CL_EHIP if the runtime fails.  All MoE calls on
 * a device share one record.
 */
cl_status cl_moe_status(void* stream);

/*
 * cl_moe_linear_decode_window -- n MoE linears (1 <= n <= 4) over the same
 * routing and the same activations, e.g. a layer's gate and up projections:
 * the paper groups a MoE layer's Gate/Up work into one window (Section
 * 4.2.2; Appendix A.1, MoE Layer).  One preparation kernel derives the
 * routing once per workgroup and computes A_e x for every linear, and one
 * backbone kernel covers every linear's routed experts; linear i's result
 * equals cl_moe_linear_decode on it alone, bit for bit.
 *
 *  n          number of linears
 *  w_expert0  host array [n] of expert-0 descriptors; all share d_in, bits
 *             and group size (d_out may differ)
 *  A, B       host arrays [n] of device factor pointers, as in
 *             cl_moe_linear_decode (entries may be NULL where r_max[i] = 0)
 *  r_max      host int32 [n];  ranks  host array [n] of device int32 [E]
 *  slot_ranks NULL, or host array [n] of device int32 [T][k] (entries may be
 *             NULL): per-slot ranks, clamped to 0..r_max[i], in place of
 *             ranks[i][e].  The paper's expert-activation term scales each
 *             routed expert's compensation priority by k times its routing
 *             weight (Section 4.3.3, Expert Activation for MoE Models), so a
 *             slot's rank can differ from its expert's static rank; slot
 *             (t, j) then uses the prefix A_e[:r_tj], B_e[:, :r_tj]
 *  y          host array [n] of device outputs [T][k][d_out_i] of out_dtype
 *  ws         device workspace of cl_moe_window_workspace(...) bytes
 * The host arrays are read during the call only.  Other arguments, limits and
 * errors as cl_moe_linear_decode; linears that differ in d_in, bits or group
 * size give CL_EINVAL.
 */
cl_status cl_moe_linear_decode_window(int32_t n, const cl_qweight* w_expert0, const uint16_t* const* A,
                                      const uint16_t* const* B, const int32_t* r_max,
                                      const int32_t* const* ranks, const int32_t* const* slot_ranks,
                                      int32_t num_experts, const void* x, int32_t x_per_slot,
                                      const int32_t* topk_ids, int32_t T, int32_t k, int32_t act_dtype,
                                      void* const* y, int32_t out_dtype, void* ws, size_t ws_bytes,
                                      void* stream);

/* Workspace bytes for cl_moe_linear_decode_window (0 for rejected arguments). */
size_t cl_moe_window_workspace(int32_t n, const cl_qweight* w_expert0, const int32_t* r_max,
                               int32_t num_experts, int32_t T, int32_t k, int32_t x_per_slot);

/*
 * cl_moe_linear_decode_gated -- the down projection of a MoE layer applied to
 * the experts' gated activations: for every slot (t, j) with e = ids[t][j],
 *     h = SiLU(g[t][j]) * u[t][j]  (elementwise, SiLU(v) = v / (1 + e^-v)),
 *     y[t][j] = deq(Q_e) h + B_e[:, :r] (A_e[:r] h),
 * with g and u the slot's gate and up outputs (cl_moe_linear_decode_window
 * over the gate and up linears with fp16 or bf16 outputs).  The expert
 * nonlinearity between the gate/up and down windows of the cross-expert
 * reorganisation (Section 4.2.2; Appendix A.1, MoE Layer) is formed by the
 * down call: with few slots (the one-launch path of cl_moe_linear_decode) as
 * each workgroup reads its activations, otherwise by one small kernel that
 * writes h for every slot into the workspace ahead of the preparation and
 * backbone kernels.  Each h is computed in fp32, saturated at +-65504 and
 * rounded to fp16, the activation precision of every decode path.
 *
 *  g, u       device [T][k][d_in] of act_dtype (fp16 or bf16), 16-byte
 *             aligned; d_in is the down projection's input (the FFN width)
 *  slot_ranks device int32 [T][k] per-slot ranks (clamped to 0..r_max) used in
 *             place of ranks[e], or NULL
 *  ws         device workspace of cl_moe_gated_workspace(w_expert0, r_max, E,
 *             T, k) bytes, 256-byte aligned
 * Everything else, the limits and the routing-error record are as for
 * cl_moe_linear_decode with x_per_slot = 1.
 * Errors: as cl_moe_linear_decode; CL_EINVAL for a null g or u.
 */
cl_status cl_moe_linear_decode_gated(const cl_qweight* w_expert0, const uint16_t* A, const uint16_t* B,
                                     int32_t r_max, const int32_t* ranks, const int32_t* slot_ranks,
                                     int32_t num_experts, const void* g, const void* u, const int32_t* topk_ids,
                                     int32_t T, int32_t k, int32_t act_dtype, void* y, int32_t out_dtype, void* ws,
                                     size_t ws_bytes, void* stream);

/* Workspace bytes for cl_moe_linear_decode_gated: those of the down call with
 * per-slot activations plus T * k * d_in fp16 values (0 for rejected
 * arguments). */
size_t cl_moe_gated_workspace(const cl_qweight* w_expert0, int32_t r_max, int32_t num_experts, int32_t T,
                              int32_t k);

/*
 * cl_allocate_ranks -- compensation ranks of the n linears of one
 * compensation window from their residual spectra (host code; no GPU).
 * Section 4.3.1 (intrinsic recoverability), Section 4.3.4 (priority and
 * rank allocation) and Appendix B.1 (second-difference knee, window
 * normalisation, two-stage allocation, discrete alignment):
 *   1. per linear, sigma / sigma_1 and its second differences at the
 *      interior indices; if the first largest exceeds tau, the salient set
 *      is the leading components up to and including that index and
 *      phi = mean(salient sigma) / mean(residual sigma), else the salient
 *      set is empty and phi = 1 (a residual set of zeros gives phi = inf,
 *      which takes the window's whole recoverability share);
 *   2. V = phi / sum(phi), S = sens / sum(sens) over the window (all-zero
 *      sensitivities count as equal), P = (V S) / sum(V S) * layer_score,
 *      continuous rank P * r_std;
 *   3. the window's total continuous rank is shared in proportion to the
 *      continuous ranks, first over the salient sets (each capped at its
 *      size), what is left over the residual sets (capped likewise), by
 *      water-filling;
 *   4. each result goes to the nearest of levels[] not above
 *      min(r_max, len[i]) (ties to the lower).
 * All arithmetic is fp64 with sums in index order.  MoE expert activation
 * (Section 4.3.3) scales a slot's rank afterwards (see slot_ranks above).
 *
 *  n            1..64 linears
 *  sigma        host array of n host pointers; sigma[i] holds len[i] >= 1
 *               singular values, finite, >= 0, descending (the sigma that
 *               cl_build_compensation writes, copied to the host)
 *  sens         host [n] matrix-level sensitivities D_i >= 0 (the paper's
 *               KL divergences; any non-negative proxy)
 *  layer_score  S_l >= 0 (see cl_layer_sensitivity)
 *  r_std        reference rank >= 0 (the largest rank whose compensation
 *               stays hidden behind the backbone, Section 4.3.4)
 *  levels       host [nlevels] admissible ranks, strictly increasing,
 *               levels[0] == 0, 1 <= nlevels <= 64
 *  r_max        cap on every rank (the stored factor count)
 *  tau          knee threshold >= 0 (0.01 in the paper)
 *  ranks        host [n] output
 * Errors: CL_EINVAL for any argument outside the above (nothing written).
 */
cl_status cl_allocate_ranks(int32_t n, const float* const* sigma, const int32_t* len, const double* sens,
                            double layer_score, double r_std, const int32_t* levels, int32_t nlevels,
                            int32_t r_max, double tau, int32_t* ranks);

/*
 * cl_layer_sensitivity -- layer-level scores S_l from layer-level
 * sensitivities D_l (Section 4.3.2; Appendix B.1; host code): the K layers
 * with the largest D (ties to the lower index) score 1, every other layer
 * D_l / min over those K of D (1 when that minimum is 0).
 *
 *  L      1..4096 layers;  D  host [L], finite, >= 0
 *  K      1..L;            S  host [L] output
 * Errors: CL_EINVAL for any argument outside the above (nothing written).
 */
cl_status cl_layer_sensitivity(int32_t L, const double* D, int32_t K, double* S);

/* Message describing the last non-CL_OK status returned on this thread. */
const char* cl_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* CL_H_ */
