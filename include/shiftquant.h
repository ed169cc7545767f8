/*
 * shiftquant.h -- C ABI of libshiftquant, the ShiftQuant backward path for
 * AMD Instinct MI355X (gfx950).
 *
 * ShiftQuant ("Towards Accurate and Efficient Sub-8-Bit Integer Training",
 * arXiv 2411.10948) quantizes the output gradient G_B = dY [M, C_out] of a
 * linear (or im2col'd conv) layer to b-bit integers whose channels fall into
 * N_G groups with power-of-two scales (Sec. 3.1), so that both backward GEMMs
 *     dX = dY . W      (loss propagation, inner dimension C_out)
 *     dW = dY^T . X    (weight gradient,  inner dimension M)
 * run as plain integer GEMMs with the group scales applied as bit shifts
 * (Sec. 3.2, "ShiftMM"; App. D).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Every array argument is a DEVICE pointer owned by the caller.  The
 *    library never allocates device memory, never frees caller memory and
 *    never synchronizes the host: all work is enqueued on `stream` (a
 *    hipStream_t passed as void*, NULL = the default stream) and completes
 *    in stream order.  Scratch memory is passed in as `workspace`; its size
 *    comes from the matching *_workspace_size query.
 *  - Matrices are row-major with a leading dimension `ld` in elements;
 *    a buffer [rows, ld] must hold rows * ld elements.
 *  - int8 code matrices (q_fold, q_t, wq_t, xq_t) and the workspace must be
 *    16-byte aligned with ld a multiple of 16.  fp32/int32 arrays must be
 *    4-byte aligned.
 *  - Arguments are validated synchronously before anything is launched; on
 *    failure nothing is enqueued and a status other than SQ_OK is returned.
 *    sq_last_error() then describes the failure (thread-local).
 *  - Data-dependent anomalies cannot be seen on the host: they are reported
 *    in the `flags` word of the device-resident sq_scale and the codes are
 *    then all 0 (see SQ_FLAG_*).
 *  - Calls that share a workspace, layout or output buffer must not overlap
 *    in time (enqueue them on one stream, or synchronize between them).
 */
#ifndef SHIFTQUANT_H
#define SHIFTQUANT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    SQ_OK = 0,
    SQ_ERR_INVALID_ARGUMENT = 1,   /* null pointer, bad size, stride or alignment  */
    SQ_ERR_OVERFLOW_RISK = 2,      /* the worst-case int32 accumulator would overflow */
    SQ_ERR_UNSUPPORTED = 3,        /* valid request outside what the library supports */
    SQ_ERR_WORKSPACE_TOO_SMALL = 4,
    SQ_ERR_HIP = 5                 /* a HIP runtime call or kernel launch failed     */
} sq_status;

/* Rounding of the gradient codes. */
enum {
    SQ_ROUND_NEAREST_EVEN = 0,     /* round(.) of App. D, ties to even                 */
    SQ_ROUND_STOCHASTIC = 1        /* SR of App. B, Eq. "sq", Philox4x32-10 uniforms   */
};

/* Bits of sq_scale.flags.  When either is set every code is 0, every channel
 * is in the last group and inv = step = 0. */
enum {
    SQ_FLAG_NONFINITE = 1u,        /* the tensor holds NaN or +-Inf                     */
    SQ_FLAG_ZERO = 2u              /* max |x| < 2^-96 (all-zero, tiny or empty tensor)  */
};

/* Layout of the int8 code matrices a call writes or reads (sq_quant_params.layout).
 *   SQ_LAYOUT_ROWS  row-major: element (r, k) at r * ld + k.
 *   SQ_LAYOUT_TILED tile-major: element (r, k) at
 *                     ((r / 16) * (ld / 64) + k / 64) * 1024 + (r % 16) * 64 + k % 64,
 *                   i.e. 16 x 64 tiles of 1 KB, the tiles of a 16-row group in
 *                   order of k.  ld must be a multiple of 64 and the buffer
 *                   must hold roundup(rows, 16) * ld bytes.  The GEMMs read
 *                   one K tile of 16 rows as one contiguous 1 KB block, which
 *                   keeps their operand streams sequential in HBM.  Writers fill
 *                   the K padding up to the next multiple of 64 with zeros
 *                   (q_fold columns [C_out, roundup(C_out, 64)), q_t and
 *                   transposed tensor columns [rows, roundup(rows, 64))).
 *                   Taken by sq_quantize_grad(_noalloc, _from_ranges),
 *                   sq_gemm_dgrad(_ranged), sq_gemm_wgrad and sq_quantize_tensor
 *                   (transpose = 2); the other calls that take sq_quant_params
 *                   return SQ_ERR_UNSUPPORTED for it. */
enum {
    SQ_LAYOUT_ROWS = 0,
    SQ_LAYOUT_TILED = 1
};

/* Quantizer parameters (host memory, read during the call only). */
typedef struct {
    int32_t bits;         /* b in [2, 8]: codes lie in [-Q, Q], Q = 2^(b-1) - 1            */
    int32_t num_groups;   /* N_G in [1, 8] (the paper's default is 4, Sec. 5.1)            */
    int32_t round_mode;   /* SQ_ROUND_*                                                    */
    int32_t layout;       /* SQ_LAYOUT_*: layout of the int8 code matrices of the call     */
    uint64_t seed;        /* stochastic rounding: Philox key                               */
    uint64_t offset;      /* stochastic rounding: stream offset (e.g. the training step)   */
} sq_quant_params;

/* Device-resident scale of a quantized tensor (written by the quantizers,
 * read by the GEMMs and sq_dequant).
 *   r_max : tau_0, the tensor's absolute maximum (Sec. 3.1)
 *   inv   : s = fl(Q / r_max), the scale of group 0 (App. B writes SR(X S) S^-1)
 *   step  : s^-1 = fl(r_max / Q), the quantization step of group 0
 *   flags : SQ_FLAG_* */
typedef struct {
    float r_max;
    float inv;
    float step;
    uint32_t flags;
} sq_scale;

/* ---------------------------------------------------------------------------
 * Size queries (host only, no device work).
 * ------------------------------------------------------------------------- */

/* Layout descriptor of the shift-folded dgrad operand produced by
 * sq_quantize_grad and consumed by sq_gemm_dgrad.
 *   *layout_bytes : size of the device buffer `layout`
 *   *min_ld_fold  : smallest admissible ld_fold for q_fold (a multiple of 16);
 *                   q_fold rows hold C_out main columns followed, from column
 *                   roundup(C_out, 64), by the appended columns of the fold:
 *                   none when N_G - 1 <= T (see sq_quantize_grad), else at
 *                   most roundup(C_out, 64) + 64 (N_G - 1). */
sq_status sq_grad_layout_size(int64_t C_out, const sq_quant_params* p,
                              size_t* layout_bytes, int64_t* min_ld_fold);

sq_status sq_quantize_grad_workspace_size(int64_t M, int64_t C_out, const sq_quant_params* p,
                                          size_t* bytes);
sq_status sq_quantize_tensor_workspace_size(int64_t rows, int64_t cols, size_t* bytes);
sq_status sq_gemm_dgrad_workspace_size(int64_t M, int64_t C_out, int64_t C_in,
                                       const sq_quant_params* p, size_t* bytes);
sq_status sq_gemm_wgrad_workspace_size(int64_t M, int64_t C_out, int64_t C_in,
                                       const sq_quant_params* p, size_t* bytes);

/* ---------------------------------------------------------------------------
 * sq_quantize_grad -- ShiftQuant of the output gradient.
 *
 * Follows Sec. 3.1 (channel ranges r_c, power-of-two thresholds
 * tau_g = r_max 2^-g), App. D (group g quantized with step
 * (r_max / Q) 2^-g) and App. B Eq. "sq" (stochastic rounding):
 *   r_c   = max_m |dY[m, c]|,  r_max = max_c r_c
 *   g_c   = the group whose interval (r_max 2^-(g+1), r_max 2^-g] holds r_c,
 *           the last group N_G - 1 also holding everything below
 *   v     = fl(dY[m, c] * fl(inv * 2^g_c)),  inv = fl(Q / r_max)
 *   code  = clamp(round(v), -Q, Q), round = ties-to-even or stochastic:
 *           floor(v) + [u16 < fl(v - floor(v)) * 2^16] with u16 the 16-bit
 *           half (i mod 2, low half first) of word (i / 2) mod 4 of
 *           Philox4x32-10(counter = (i / 8 as two 32-bit words, offset as two
 *           words), key = seed as two words), i = m * C_out + c.  One
 *           Philox block serves 8 elements; the rounding bias is below 2^-16
 *           of a step.
 *
 * Inputs : dY [M, ld_dY] fp32 (M >= 0, C_out >= 0, ld_dY >= C_out).
 * Outputs (any of q_fold / q_t may be NULL to skip it):
 *   q_fold [M, ld_fold] int8, the dgrad operand with the shifts of
 *          ShiftMM folded in.  The shifts sh_c = N_G - 1 - g_c are cut into
 *          windows [B, B + T] of T + 1 values, T the largest shift with
 *          Q 2^T <= 127, and each channel is stored once, as
 *          code << (sh_c - B) for its window's base B (this fits int8).  The
 *          window holding the most channels (lowest B on ties) uses the
 *          channel's own column c.  Every other non-empty window is a region
 *          of appended columns from column roundup(C_out, 64): its channels
 *          in ascending order, padded to a multiple of 64 columns; column c
 *          of such a channel holds 0.  When N_G - 1 <= T (b <= 5 at N_G = 4)
 *          there is one window and nothing is appended.  `layout` records
 *          the windows, and sq_gemm_dgrad applies their bases as left shifts
 *          of its accumulator.  Columns in [C_out, roundup(C_out, 64)) and
 *          the padding of appended regions are left unwritten (with
 *          SQ_LAYOUT_TILED the former are written as zeros).
 *   q_t    [C_out, ld_t] int8 (ld_t >= M), the codes themselves, transposed:
 *          q_t[c, m] = code(m, c); this is the wgrad operand.
 *   group  [C_out] uint8, g_c.
 *   scale  one sq_scale (r_max, inv, step, flags).
 *   layout [layout_bytes], the fold descriptor for sq_gemm_dgrad.
 * Workspace: sq_quantize_grad_workspace_size bytes.
 * Errors: SQ_ERR_INVALID_ARGUMENT, SQ_ERR_WORKSPACE_TOO_SMALL, SQ_ERR_HIP.
 * ------------------------------------------------------------------------- */
sq_status sq_quantize_grad(const float* dY, int64_t M, int64_t C_out, int64_t ld_dY,
                           const sq_quant_params* p,
                           int8_t* q_fold, int64_t ld_fold,
                           int8_t* q_t, int64_t ld_t,
                           uint8_t* group, sq_scale* scale, int32_t* layout,
                           void* workspace, size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * sq_quantize_grad_noalloc -- sq_quantize_grad without a workspace argument,
 * for callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc).
 *
 * Same arguments, results and errors as sq_quantize_grad, minus workspace /
 * workspace_bytes.  Its scratch is a fixed 16 MiB device array inside the
 * library (one copy per GPU, held until the process ends); the call itself
 * allocates nothing.  A gradient whose quantizer scratch
 * (sq_quantize_grad_workspace_size) exceeds 1 MiB (about 65,000 channels) is rejected with
 * SQ_ERR_WORKSPACE_TOO_SMALL before any launch.  All calls on one GPU share
 * that array: calls that overlap in time on one GPU (other streams, other
 * host threads) race and must be serialized by the caller.  The first call
 * on a device looks up its scratch address (hipGetSymbolAddress) with that
 * device current.
 * ------------------------------------------------------------------------- */
sq_status sq_quantize_grad_noalloc(const float* dY, int64_t M, int64_t C_out, int64_t ld_dY,
                                   const sq_quant_params* p,
                                   int8_t* q_fold, int64_t ld_fold,
                                   int8_t* q_t, int64_t ld_t,
                                   uint8_t* group, sq_scale* scale, int32_t* layout, void* stream);

/* ---------------------------------------------------------------------------
 * sq_quantize_tensor -- per-tensor symmetric quantization of W or X.
 *
 * The paper's INT8 baseline quantizes weights, activations and gradients per
 * tensor (Sec. 5.1); it is ShiftQuant with a single group:
 *   a = max |T|,  inv = fl(Q / a),  step = fl(a / Q),
 *   code = clamp(round_half_even(fl(T * inv)), -Q, Q),  Q = 2^(bits-1) - 1.
 * Input : T [rows, ld] fp32 (ld >= cols).
 * Output: transpose == 0: q [rows, ld_q] int8 (ld_q >= cols)
 *         transpose == 1: q [cols, ld_q] int8 (ld_q >= rows), q[j, i] = code(i, j)
 *         transpose == 2: the same matrix tile-major (SQ_LAYOUT_TILED; ld_q a
 *         multiple of 64, >= roundup(rows, 64); columns [rows, roundup(rows,
 *         64)) written as zeros), the operand of the tile-major GEMMs
 *         (sq_gemm_dgrad takes W^T codes and sq_gemm_wgrad X^T codes, i.e.
 *         W [C_out, C_in] and X [M, C_in] quantized with transpose = 1).
 *         scale: one sq_scale.
 * Errors: SQ_ERR_INVALID_ARGUMENT, SQ_ERR_WORKSPACE_TOO_SMALL, SQ_ERR_HIP.
 * ------------------------------------------------------------------------- */
sq_status sq_quantize_tensor(const float* T, int64_t rows, int64_t cols, int64_t ld, int32_t bits,
                             int32_t transpose, int8_t* q, int64_t ld_q, sq_scale* scale,
                             void* workspace, size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * sq_quantize_channels -- per-channel symmetric quantization of a weight
 * matrix.
 *
 * Sec. 5.1 quantizes weights per output channel in the forward pass and per
 * input channel in loss propagation.  Each channel is quantized like a
 * tensor of its own (see sq_quantize_tensor): amax over the channel,
 * inv = fl(Q / amax), step = fl(amax / Q),
 * code = clamp(round_half_even(fl(T * inv)), -Q, Q); a channel whose amax is
 * NaN/Inf or below 2^-96 gets SQ_FLAG_NONFINITE / SQ_FLAG_ZERO in its scale
 * and all-zero codes.
 * Input : T [rows, ld] fp32; axis 0: one scale per row (W [C_out, C_in] per
 *         output channel), axis 1: one per column (per input channel).
 * Output: q as in sq_quantize_tensor (transpose 0: [rows, ld_q], 1:
 *         [cols, ld_q]); scales [rows] (axis 0) or [cols] (axis 1) sq_scale.
 * Workspace: sq_quantize_channels_workspace_size bytes (0 for axis 0).
 * Errors: SQ_ERR_INVALID_ARGUMENT, SQ_ERR_WORKSPACE_TOO_SMALL, SQ_ERR_HIP.
 * ------------------------------------------------------------------------- */
sq_status sq_quantize_channels_workspace_size(int64_t rows, int64_t cols, int32_t axis, size_t* bytes);
sq_status sq_quantize_channels(const float* T, int64_t rows, int64_t cols, int64_t ld, int32_t bits,
                               int32_t axis, int32_t transpose, int8_t* q, int64_t ld_q, sq_scale* scales,
                               void* workspace, size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * sq_gemm_forward -- forward pass Y = X . W^T with ShiftQuant activations
 * and per-output-channel weights (Sec. 5.1; the first GEMM of Fig. "MMs").
 *
 * X is quantized by sq_quantize_grad (ShiftQuant groups over its channels,
 * which are this product's inner dimension), so the product is ShiftMM as in
 * sq_gemm_dgrad, with the weight scale taken per output column:
 *   acc[m, n] = sum_c (code_X(m, c) * wq[n, c]) << (N_G - 1 - g_c)     (int32)
 *   Y[m, n]   = fl(float(acc[m, n]) * gamma_n),
 *   gamma_n   = fl(fl(xscale.step * wscales[n].step) * 2^-(N_G - 1)).
 * The same call is loss propagation with per-input-channel weights: pass the
 * gradient's codes as X, W^T codes as wq and their per-column scales.
 * Inputs : xq_fold, ld_fold, layout, group, xscale from sq_quantize_grad of
 *          X [M, C_in] with the same p; wq [C_out, ld_w] int8 W codes
 *          (ld_w >= C_in) with wscales [C_out] from sq_quantize_channels
 *          (axis 0, transpose 0).
 * Outputs (either may be NULL, not both): acc [M, ld_acc] int32,
 *          Y [M, ld_Y] fp32.
 * Workspace: sq_gemm_dgrad_workspace_size(M, C_in, C_out, p) bytes.
 * Errors: SQ_ERR_INVALID_ARGUMENT; SQ_ERR_OVERFLOW_RISK when
 *         C_in * Q * 2^(N_G-1) * 128 >= 2^31; SQ_ERR_WORKSPACE_TOO_SMALL;
 *         SQ_ERR_HIP.
 * ------------------------------------------------------------------------- */
sq_status sq_gemm_forward(const int8_t* xq_fold, int64_t ld_fold, const int32_t* layout,
                          const uint8_t* group, const sq_scale* xscale,
                          const int8_t* wq, int64_t ld_w, const sq_scale* wscales,
                          int64_t M, int64_t C_in, int64_t C_out, const sq_quant_params* p,
                          int32_t* acc, int64_t ld_acc, float* Y, int64_t ld_Y,
                          void* workspace, size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * sq_gemm_dgrad -- loss propagation dX = dY . W as ShiftMM.
 *
 * Eq. "dq_mm_f" and App. D (left-shift form): with 0-indexed groups,
 *   acc[n, k] = sum_c (code(n, c) * wq[c, k]) << (N_G - 1 - g_c)      (int32)
 *   dX[n, k]  = fl(float(acc[n, k]) * alpha),
 *   alpha     = fl(fl(gscale.step * wscale.step) * 2^-(N_G - 1)).
 * Sec. 3.2 shifts every product before it is accumulated; here the shift of
 * each inner index c is folded into the int8 operand (q_fold) up to its
 * window's base B, and the bases are applied once per window to the int32
 * accumulator, which visits the windows in descending B (Horner's rule).
 * Inputs : q_fold, ld_fold, layout, group, gscale from sq_quantize_grad with
 *          the same M, C_out and p; wq_t [C_in, ld_w] int8 = W^T codes
 *          (ld_w >= C_out); wscale its sq_scale.
 * Outputs (either may be NULL, not both): acc [M, ld_acc] int32,
 *          dX [M, ld_dX] fp32.
 * Errors: SQ_ERR_INVALID_ARGUMENT; SQ_ERR_OVERFLOW_RISK when
 *         C_out * Q * 2^(N_G-1) * 128 >= 2^31; SQ_ERR_WORKSPACE_TOO_SMALL;
 *         SQ_ERR_HIP.
 * ------------------------------------------------------------------------- */
sq_status sq_gemm_dgrad(const int8_t* q_fold, int64_t ld_fold, const int32_t* layout,
                        const uint8_t* group, const sq_scale* gscale,
                        const int8_t* wq_t, int64_t ld_w, const sq_scale* wscale,
                        int64_t M, int64_t C_out, int64_t C_in, const sq_quant_params* p,
                        int32_t* acc, int64_t ld_acc, float* dX, int64_t ld_dX,
                        void* workspace, size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * sq_gemm_wgrad -- weight gradient dW = dY^T . X.
 *
 * The third training GEMM (Fig. "MMs"); its inner dimension is the token
 * index, so every output row c lies in one gradient group and the group
 * scale is a per-row factor (Eq. "dq_mm_f" applied to this product):
 *   acc[c, k] = sum_m code(m, c) * xq[m, k]                             (int32)
 *   dW[c, k]  = fl(float(acc[c, k]) * beta_c),
 *   beta_c    = fl(fl(gscale.step * xscale.step) * 2^-g_c).
 * Inputs : q_t [C_out, ld_t] int8 and group, gscale from sq_quantize_grad;
 *          xq_t [C_in, ld_x] int8 = X^T codes (ld_x >= M); xscale its scale.
 * Outputs (either may be NULL, not both): acc [C_out, ld_acc] int32,
 *          dW [C_out, ld_dW] fp32.
 * Errors: SQ_ERR_INVALID_ARGUMENT; SQ_ERR_OVERFLOW_RISK when
 *         M * Q * 128 >= 2^31; SQ_ERR_WORKSPACE_TOO_SMALL; SQ_ERR_HIP.
 * ------------------------------------------------------------------------- */
sq_status sq_gemm_wgrad(const int8_t* q_t, int64_t ld_t, const uint8_t* group, const sq_scale* gscale,
                        const int8_t* xq_t, int64_t ld_x, const sq_scale* xscale,
                        int64_t M, int64_t C_out, int64_t C_in, const sq_quant_params* p,
                        int32_t* acc, int64_t ld_acc, float* dW, int64_t ld_dW,
                        void* workspace, size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * sq_gemm_dgrad_grouped -- the GEMM-based implementation of the same loss
 * propagation, kept as a comparison for ShiftMM.
 *
 * Sec. 3.2 describes it in three steps: extract one pair of smaller matrices
 * per group (memory rearrangement: the group's code columns and weight rows
 * side by side), multiply each pair with a plain GEMM, then shift each
 * product by N_G - 1 - g and sum.  The result is the accumulator and dX of
 * sq_gemm_dgrad, bit for bit; only the cost differs.
 * Inputs, outputs and errors as sq_gemm_dgrad; the workspace
 * (sq_gemm_dgrad_grouped_workspace_size bytes, 256-byte aligned) holds the
 * rearranged operands [M + C_in, C_out + 63 N_G] and N_G int32 products
 * [M, C_in].  SQ_ERR_UNSUPPORTED when a rearranged operand spans 2^31 bytes.
 * ------------------------------------------------------------------------- */
sq_status sq_gemm_dgrad_grouped_workspace_size(int64_t M, int64_t C_out, int64_t C_in,
                                               const sq_quant_params* p, size_t* bytes);
sq_status sq_gemm_dgrad_grouped(const int8_t* q_fold, int64_t ld_fold, const int32_t* layout,
                                const uint8_t* group, const sq_scale* gscale,
                                const int8_t* wq_t, int64_t ld_w, const sq_scale* wscale,
                                int64_t M, int64_t C_out, int64_t C_in, const sq_quant_params* p,
                                int32_t* acc, int64_t ld_acc, float* dX, int64_t ld_dX,
                                void* workspace, size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * sq_conv_dgrad -- input gradient of a stride-1 convolution, im2col and
 * col2im both implicit.
 *
 * The ResNet layers of Sec. 5 are convolutions that the GEMM of Eq. "dq_mm_f"
 * serves through im2col: X_col [N Ho Wo, KH KW C_in] with columns in
 * (r, s, ci) order, dX_col = dY . W, and dX = col2im(dX_col), col2im being
 * the adjoint of im2col.  This call computes dX directly, without writing
 * dX_col: with sh_c = N_G - 1 - g_c (0-indexed groups),
 *   acc[(n, ih, iw), ci] = sum_{r < KH, s < KW} sum_c
 *                          (code((n, ih + PH - r, iw + PW - s), c) * wq[c, (r, s, ci)]) << sh_c
 * over the window taps whose output pixel lies inside the Ho x Wo grid,
 * Ho = H + 2 PH - KH + 1, Wo = W + 2 PW - KW + 1, and
 *   dX = fl(float(acc) * alpha), alpha as in sq_gemm_dgrad.
 * The forward convolution this differentiates reads input pixel
 * (n, oh + r - PH, ow + s - PW) at tap (r, s) of output pixel (n, oh, ow).
 * Inputs : q_fold, ld_fold, layout, group, gscale from sq_quantize_grad of
 *          dY [N Ho Wo, C_out] (NHWC pixel order); wq_t [KH KW C_in, ld_w]
 *          int8 = W^T codes of W [C_out, KH KW C_in] (ld_w >= C_out);
 *          wscale its sq_scale.  1 <= KH, KW <= 15, 0 <= PH < KH,
 *          0 <= PW < KW, N H W < 2^31, N Ho Wo ld_fold < 2^31 bytes.
 * Outputs (either may be NULL, not both): acc [N H W, ld_acc] int32,
 *          dX [N H W, ld_dX] fp32 (NHWC).
 * Workspace: sq_conv_dgrad_workspace_size bytes (the weights regathered in
 *          the order of the implicit K sequence).
 * Errors: SQ_ERR_INVALID_ARGUMENT; SQ_ERR_OVERFLOW_RISK when
 *         KH KW C_out Q 2^(N_G-1) 128 >= 2^31; SQ_ERR_UNSUPPORTED beyond the
 *         size limits above; SQ_ERR_WORKSPACE_TOO_SMALL; SQ_ERR_HIP.
 * ------------------------------------------------------------------------- */
sq_status sq_conv_dgrad_workspace_size(int64_t C_out, int64_t C_in, int32_t KH, int32_t KW,
                                       const sq_quant_params* p, size_t* bytes);
sq_status sq_conv_dgrad(const int8_t* q_fold, int64_t ld_fold, const int32_t* layout,
                        const uint8_t* group, const sq_scale* gscale,
                        const int8_t* wq_t, int64_t ld_w, const sq_scale* wscale,
                        int64_t N, int64_t H, int64_t W, int64_t C_out, int64_t C_in,
                        int32_t KH, int32_t KW, int32_t PH, int32_t PW, const sq_quant_params* p,
                        int32_t* acc, int64_t ld_acc, float* dX, int64_t ld_dX,
                        void* workspace, size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * sq_dequant -- int32 accumulator to fp32 (Eq. "dq_mm_f": the inverse
 * scales multiply the integer sum once, outside the accumulation).
 *   kind 0 (dgrad): out = fl(float(acc) * alpha), alpha as in sq_gemm_dgrad
 *   kind 1 (wgrad): out[r, :] = fl(float(acc[r, :]) * beta_r), beta_r as in
 *                   sq_gemm_wgrad with g_r = group[r]
 *   kind 2 (per-column weight scales): out[:, c] = fl(float(acc[:, c]) * gamma_c),
 *                   gamma_c as in sq_gemm_forward, oscale an array [cols]
 * Inputs : acc [rows, ld_acc] int32; group [rows] (kind 1 only); gscale and
 *          oscale (the W scale for kind 0, the X scale for kind 1).
 * Output : out [rows, ld_out] fp32.
 * Errors: SQ_ERR_INVALID_ARGUMENT, SQ_ERR_HIP.
 * ------------------------------------------------------------------------- */
sq_status sq_dequant(const int32_t* acc, int64_t rows, int64_t cols, int64_t ld_acc, int32_t kind,
                     const uint8_t* group, const sq_scale* gscale, const sq_scale* oscale,
                     int32_t num_groups, float* out, int64_t ld_out, void* stream);

/* ---------------------------------------------------------------------------
 * sq_conv_dgrad_ranged -- sq_conv_dgrad that also writes the channel ranges
 * of dX for the quantizer of the layer below.
 *
 * Sec. 3.1's r_c = max_m |dY[m, c]| of the next layer's gradient, taken as
 * the conv input gradient dX [N H W, C_in] is stored:
 *   dX_ranges[s, c] = bits of max |dX[m, c]| over rows m in [s R, (s+1) R),
 * sign bit cleared, s < *range_slabs = ceil(N H W / R), R = *range_rows.
 * The streaming kernel (C_out <= 64 with one fold window, C_in <= 64 and a
 * multiple of 4, same-size window of at most 9 taps) takes them per block of
 * its own rows (R a multiple of 128, at most 512 slabs); the other conv
 * kernels store dX and one pass takes 32-row slab maxima (R = 32).
 * dX_ranges must hold sq_gemm_dgrad_range_slabs(N H W) x C_in words (the
 * most either path writes).  *range_slabs and *range_rows (host memory) are
 * set before the call returns, so the caller passes the slab count on to
 * sq_quantize_grad_from_ranges / sq_quantize_grad_conv_from_ranges without a
 * synchronization.  Arguments, outputs and errors as sq_conv_dgrad, with dX
 * required; SQ_ERR_UNSUPPORTED beyond 2^21 input pixels.
 * ------------------------------------------------------------------------- */
sq_status sq_conv_dgrad_ranged(const int8_t* q_fold, int64_t ld_fold, const int32_t* layout,
                               const uint8_t* group, const sq_scale* gscale,
                               const int8_t* wq_t, int64_t ld_w, const sq_scale* wscale,
                               int64_t N, int64_t H, int64_t W, int64_t C_out, int64_t C_in,
                               int32_t KH, int32_t KW, int32_t PH, int32_t PW, const sq_quant_params* p,
                               int32_t* acc, int64_t ld_acc, float* dX, int64_t ld_dX,
                               uint32_t* dX_ranges, int64_t* range_slabs, int64_t* range_rows,
                               void* workspace, size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * sq_gemm_dgrad_ranged -- sq_gemm_dgrad that also writes the channel ranges
 * of dX for the quantizer of the layer below.
 *
 * In a chain of layers dX is the next dY to be quantized, and the quantizer's
 * first step is r_c = max_m |dY[m, c]| (Sec. 3.1).  Here the GEMM's epilogue
 * takes those maxima from the values it stores:
 *   dX_ranges[s, c] = bits of max |dX[m, c]| over rows m in [32 s, 32 s + 32),
 * sign bit cleared, s < sq_gemm_dgrad_range_slabs(M) = ceil(M / 32); they are
 * the `ranges` input of sq_quantize_grad_from_ranges.  The maxima come from
 * the GEMM's epilogue when C_out is a multiple of 64 (and every operand's byte
 * offsets fit in 31 bits); otherwise one extra pass over the stored dX takes
 * them.  Arguments, outputs and errors as sq_gemm_dgrad, with dX required;
 * SQ_ERR_UNSUPPORTED beyond 2^21 rows on the second path.
 * ------------------------------------------------------------------------- */
sq_status sq_gemm_dgrad_range_slabs(int64_t M, int64_t* slabs);
sq_status sq_gemm_dgrad_ranged(const int8_t* q_fold, int64_t ld_fold, const int32_t* layout,
                               const uint8_t* group, const sq_scale* gscale,
                               const int8_t* wq_t, int64_t ld_w, const sq_scale* wscale,
                               int64_t M, int64_t C_out, int64_t C_in, const sq_quant_params* p,
                               int32_t* acc, int64_t ld_acc, float* dX, int64_t ld_dX, uint32_t* dX_ranges,
                               void* workspace, size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * Implicit-im2col weight gradient of a stride-1 convolution.
 *
 * The wgrad of the im2col'd conv layer (Fig. "MMs", third GEMM, on the conv
 * layers of Sec. 5), computed without the im2col:
 *   acc[co, (r KW + s) C_in + ci] = sum_{n, oh, ow} code(n, oh, ow, co)
 *                                   xq(n, oh + r - PH, ow + s - PW, ci)
 * (zero outside the input), with the epilogue of sq_gemm_wgrad
 * (dW[co, :] = fl(float(acc[co, :]) * beta_co)).  Columns follow the (r, s, ci)
 * order of W [C_out, KH KW C_in].  Stride 1, 0 <= PH < KH, 0 <= PW < KW,
 * KH, KW <= 16; Ho = H + 2 PH - KH + 1, Wo = W + 2 PW - KW + 1.
 *
 * Both operands live on a padded pixel grid of Hp = H + 2 PH rows and
 * Wp = roundup(W + 2 PW, 16) columns per image, on which tap (r, s) is the
 * constant shift r Wp + s of the pixel index:
 *   q_tp [C_out, ld_tp >= q_ld]: gradient code (n, oh, ow, c) at column
 *        n Hp Wp + oh Wp + ow of row c, every other column 0.
 *   xs   [C_in, ld_xs >= x_ld]: input pixel (n, ih, iw) of channel ci at
 *        column n Hp Wp + (ih + PH) Wp + iw + PW of row ci, 0 in the padding
 *        and in the x_ld - q_ld = (KH - 1) Wp + 64 columns past the grid, so
 *        that tap (r, s) of grid position P reads column P + r Wp + s.
 * sq_conv_wgrad_layout gives x_rows = C_in, x_ld and q_ld.
 * sq_conv_pack_input builds xs from the input codes xq_t [C_in, ld_xq >= N H W]
 *   (sq_quantize_tensor, transpose 1) and writes every byte of xs (x_ld
 *   columns); in training the input codes come from the forward pass, and
 *   the pack runs once per step.
 * sq_conv_pack_grad builds q_tp from transposed codes q_t [C_out, ld_t >= N Ho Wo]
 *   and writes every byte of q_tp.
 * sq_quantize_input_conv is the forward pass's quantizer of the layer input
 *   X [N H W, ld_X] (NHWC rows, fp32): the per-tensor b-bit codes of
 *   sq_quantize_tensor (Sec. 5.1: activations quantized per tensor) written
 *   straight onto the padded input grid xs, optionally also
 *   row-major into xq [N H W, ld_xq >= C_in] (the forward's layout; NULL to
 *   skip).  xs's padding is never written, so the caller zero-fills that
 *   buffer once; then no pack is needed.  Workspace:
 *   sq_quantize_tensor_workspace_size(N H W, C_in).  Errors as
 *   sq_quantize_tensor, plus SQ_ERR_UNSUPPORTED beyond 2^32 grid pixels.
 * sq_quantize_grad_conv is sq_quantize_grad for the conv's gradient
 *   dY [N Ho Wo, ld_dY] (same codes, groups, scale, layout, q_fold, workspace)
 *   that writes the transposed codes straight onto the padded grid: q_tp's
 *   padding is never written, so the caller zero-fills that buffer once.
 * sq_quantize_grad_conv_from_ranges is the same with the channel ranges
 *   given as partial maxima (see sq_quantize_grad_from_ranges), e.g. the
 *   dX_ranges of sq_conv_dgrad_ranged of the layer above.
 * sq_conv_wgrad runs the int8 product over the padded grid (K = N Hp Wp
 *   rounded up to 64) with every tap read from the one copy of the input at
 *   its shift r Wp + s (1 x 1 windows: a plain int8 GEMM of the two grids),
 *   then, when K is split, the sum of the int32 partials.
 * Outputs: acc [C_out, ld_acc] int32 and/or dW [C_out, ld_dW] fp32, each row
 *          KH KW C_in wide.
 * Workspace: sq_conv_wgrad_workspace_size bytes (split-K partials, may be 0).
 * Errors: SQ_ERR_INVALID_ARGUMENT; SQ_ERR_OVERFLOW_RISK when
 *         N Ho Wo Q 128 >= 2^31; SQ_ERR_UNSUPPORTED when a padded grid
 *         exceeds 2^31 bytes; SQ_ERR_WORKSPACE_TOO_SMALL; SQ_ERR_HIP.
 * ------------------------------------------------------------------------- */
sq_status sq_conv_wgrad_layout(int64_t N, int64_t H, int64_t W, int64_t C_in, int32_t KH, int32_t KW,
                               int32_t PH, int32_t PW, int64_t* x_rows, int64_t* x_ld, int64_t* q_ld);
sq_status sq_conv_pack_input(const int8_t* xq_t, int64_t ld_xq, int64_t N, int64_t H, int64_t W, int64_t C_in,
                             int32_t KH, int32_t KW, int32_t PH, int32_t PW, int8_t* xs, int64_t ld_xs,
                             void* stream);
sq_status sq_conv_pack_grad(const int8_t* q_t, int64_t ld_t, int64_t N, int64_t H, int64_t W, int64_t C_out,
                            int32_t KH, int32_t KW, int32_t PH, int32_t PW, int8_t* q_tp, int64_t ld_tp,
                            void* stream);
sq_status sq_quantize_input_conv(const float* X, int64_t N, int64_t H, int64_t W, int64_t C_in, int64_t ld_X,
                                 int32_t KH, int32_t KW, int32_t PH, int32_t PW, int32_t bits,
                                 int8_t* xq, int64_t ld_xq, int8_t* xs, int64_t ld_xs, sq_scale* scale,
                                 void* workspace, size_t workspace_bytes, void* stream);
sq_status sq_quantize_grad_conv(const float* dY, int64_t N, int64_t H, int64_t W, int64_t C_out, int64_t ld_dY,
                                int32_t KH, int32_t KW, int32_t PH, int32_t PW, const sq_quant_params* p,
                                int8_t* q_fold, int64_t ld_fold, int8_t* q_tp, int64_t ld_tp,
                                uint8_t* group, sq_scale* scale, int32_t* layout,
                                void* workspace, size_t workspace_bytes, void* stream);
sq_status sq_quantize_grad_conv_from_ranges(const float* dY, int64_t N, int64_t H, int64_t W, int64_t C_out,
                                            int64_t ld_dY, int32_t KH, int32_t KW, int32_t PH, int32_t PW,
                                            const sq_quant_params* p, const uint32_t* ranges, int64_t range_slabs,
                                            int8_t* q_fold, int64_t ld_fold, int8_t* q_tp, int64_t ld_tp,
                                            uint8_t* group, sq_scale* scale, int32_t* layout,
                                            void* workspace, size_t workspace_bytes, void* stream);
sq_status sq_conv_wgrad_workspace_size(int64_t N, int64_t H, int64_t W, int64_t C_out, int64_t C_in,
                                       int32_t KH, int32_t KW, int32_t PH, int32_t PW,
                                       const sq_quant_params* p, size_t* bytes);
sq_status sq_conv_wgrad(const int8_t* q_tp, int64_t ld_tp, const uint8_t* group, const sq_scale* gscale,
                        const int8_t* xs, int64_t ld_xs, const sq_scale* xscale,
                        int64_t N, int64_t H, int64_t W, int64_t C_out, int64_t C_in,
                        int32_t KH, int32_t KW, int32_t PH, int32_t PW, const sq_quant_params* p,
                        int32_t* acc, int64_t ld_acc, float* dW, int64_t ld_dW,
                        void* workspace, size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * sq_quantize_grad_from_ranges -- sq_quantize_grad with the channel ranges
 * supplied by the producer of dY.
 *
 * The quantizer's first step (r_c = max_m |dY[m, c]|, Sec. 3.1) reads all of
 * dY once before the codes can be formed; a kernel that writes dY can take
 * those maxima on the fly instead.  `ranges` holds them as partial maxima:
 * ranges[s, c], s < range_slabs, is the bit pattern of max |dY[m, c]| over
 * some subset of the rows (sign bit cleared, so NaN and Inf compare above
 * every finite value), the subsets covering all M rows; r_c is the maximum
 * over s.  Everything else -- outputs, layout, workspace
 * (sq_quantize_grad_workspace_size), errors -- is as in sq_quantize_grad, and
 * the results are identical when the ranges are exact.
 * sq_l1bn_backward writes such ranges for its dx.
 * ------------------------------------------------------------------------- */
sq_status sq_quantize_grad_from_ranges(const float* dY, int64_t M, int64_t C_out, int64_t ld_dY,
                                       const sq_quant_params* p, const uint32_t* ranges, int64_t range_slabs,
                                       int8_t* q_fold, int64_t ld_fold,
                                       int8_t* q_t, int64_t ld_t,
                                       uint8_t* group, sq_scale* scale, int32_t* layout,
                                       void* workspace, size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * Fully-quantized L1 batch normalization (L1BNQ), Sec. 4 (Fig. l1bnq) and
 * App. C.1 / C.2: input features, statistics and parameters are quantized,
 * and the normalization divides by the L1 deviation instead of the standard
 * deviation.
 *
 * Per-channel state written by sq_l1bn_forward and read by sq_l1bn_backward
 * (device memory, one entry per channel):
 *   mu       m_c = round_half_even(S_c / M), S_c = sum_m q[m, c]: the batch mean
 *            quantized onto the input's own 8-bit grid (mu^q = s_x m_c)
 *   sigma    k_c = max(1, round_half_even(127 A_c / A_max)): the L1 deviation
 *            sigma_c = s_x A_c / M quantized per tensor to 8 bits under the
 *            step max_c sigma_c / 127 (0 when the layer is flagged ZERO)
 *   sign_sum P_c = sum_m sgn(q[m, c] - m_c)
 *   gamma, beta  gamma^q_c, beta^q_c: the parameters quantized per tensor to
 *            8 bits (as sq_quantize_tensor), dequantized
 *   kappa    fl32(gamma^q_c 127 M / (A_max k_c)), evaluated in binary64
 *   dev_sum  A_c = sum_m |q[m, c] - m_c|
 * Layer state: rows M, dev_max A_max = max_c A_c, x_step s_x (the input's
 * step), flags (SQ_FLAG_ZERO when A_max = 0: every channel constant), and the
 * scales of gamma and beta.
 * ------------------------------------------------------------------------- */
typedef struct {
    int32_t mu;
    int32_t sigma;
    int32_t sign_sum;
    float gamma;
    float beta;
    float kappa;
    int64_t dev_sum;
} sq_l1bn_channel;      /* 32 bytes */

typedef struct {
    int64_t rows;
    int64_t dev_max;
    float x_step;
    uint32_t flags;
    sq_scale gamma_scale;
    sq_scale beta_scale;
} sq_l1bn_layer;        /* 56 bytes */

/* Partial-maximum slabs that sq_l1bn_backward writes to dx_ranges
 * ([slabs, C] uint32) for M rows and C channels. */
sq_status sq_l1bn_range_slabs(int64_t M, int64_t C, int64_t* slabs);
sq_status sq_l1bn_forward_workspace_size(int64_t M, int64_t C, size_t* bytes);
sq_status sq_l1bn_backward_workspace_size(int64_t M, int64_t C, const sq_quant_params* p, size_t* bytes);

/* ---------------------------------------------------------------------------
 * sq_l1bn_forward -- L1BNQ forward over a batch (training statistics).
 *   y[m, c] = fl(fl(kappa_c (q[m, c] - m_c)) + beta^q_c),
 * i.e. gamma^q (x^q - mu^q) / sigma^q + beta^q with x^q = s_x q (App. C.2's
 * normalization with quantized statistics); with A_max = 0, y = beta^q.
 * Inputs : xq [M, ld_x] int8, the 8-bit per-tensor codes of the layer input
 *          (sq_quantize_tensor, bits 8), 16-byte aligned, ld_x % 16 == 0;
 *          xscale its sq_scale (device); gamma, beta [C] fp32 (device).
 *          1 <= M <= 2^24.
 * Outputs: y [M, ld_y] fp32; chan [C] and layer (device) for the backward.
 * Workspace: sq_l1bn_forward_workspace_size bytes.
 * Errors: SQ_ERR_INVALID_ARGUMENT, SQ_ERR_UNSUPPORTED (M > 2^24),
 *         SQ_ERR_WORKSPACE_TOO_SMALL, SQ_ERR_HIP.
 * ------------------------------------------------------------------------- */
sq_status sq_l1bn_forward(const int8_t* xq, int64_t M, int64_t C, int64_t ld_x, const sq_scale* xscale,
                          const float* gamma, const float* beta, float* y, int64_t ld_y,
                          sq_l1bn_channel* chan, sq_l1bn_layer* layer,
                          void* workspace, size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * sq_l1bn_backward -- L1BNQ backward.
 * The incoming gradient dy is quantized with ShiftQuant (as sq_quantize_grad
 * with params p; codes qg, groups g_c, channel steps delta_c = step 2^-g_c);
 * the L1 normalization is differentiated exactly (App. C.1 with
 * sigma = mean |x - mu|, which brings in s = sgn(x - mu)), the quantizers of
 * mu and sigma passed straight through:
 *   dx = (gamma^q / sigma^q)(g - mean g - mean(g xhat)(s - mean s)).
 * With integer sums G1 = sum qg, G2 = sum qg (q - m), P = sign_sum,
 * rho = 127 M / (A_max k), lambda = gamma^q rho / s_x, in binary64:
 *   dbeta = delta G1,  dgamma = (delta G2) rho,  D = dgamma / M,
 *   a = lambda delta,  b = -(lambda D),  e = lambda (D P / M - delta G1 / M),
 * each rounded once to fp32, and dx = fl(fl(fl(a qg) + fl(b sgn(q - m))) + e).
 * With A_max = 0: dgamma = 0 and dx = 0.
 * Inputs : dy [M, ld_dy] fp32; p (b, N_G, rounding of the gradient codes);
 *          xq, ld_x, chan, layer: the forward's input codes and state.
 * Outputs: dx [M, ld_dx] fp32; dgamma, dbeta [C] fp32; group [C] and gscale:
 *          the gradient quantizer's groups and scale; dx_ranges (may be NULL):
 *          [sq_l1bn_range_slabs, C] partial maxima of |dx| per channel, the
 *          input of sq_quantize_grad_from_ranges for the layer below.
 * Workspace: sq_l1bn_backward_workspace_size bytes.
 * Errors: as sq_l1bn_forward.
 * ------------------------------------------------------------------------- */
sq_status sq_l1bn_backward(const float* dy, int64_t M, int64_t C, int64_t ld_dy, const sq_quant_params* p,
                           const int8_t* xq, int64_t ld_x, const sq_l1bn_channel* chan,
                           const sq_l1bn_layer* layer, float* dx, int64_t ld_dx,
                           float* dgamma, float* dbeta, uint8_t* group, sq_scale* gscale,
                           uint32_t* dx_ranges, void* workspace, size_t workspace_bytes, void* stream);

/* Static description of a status code. */
const char* sq_status_string(sq_status s);

/* Message of the last failed call on this thread ("" if none);
 * sq_last_error_string is the same function under a second name. */
const char* sq_last_error(void);
const char* sq_last_error_string(void);

#ifdef __cplusplus
}
#endif

#endif /* SHIFTQUANT_H */
