// Internal declarations of libshiftquant (kernels and their launchers).
// Not part of the public ABI; see include/shiftquant.h for that.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "shiftquant.h"

namespace sq {

// ---------------------------------------------------------------------------
// Fold layout descriptor (int32 words in a caller-provided device buffer).
//
// ShiftMM needs sum_c code_c * w_c * 2^sh_c with sh_c = N_G - 1 - g_c.  The
// shifts are cut into windows of T + 1 consecutive values (T: the largest
// shift with Q * 2^T <= 127); a channel of window [B, B + T] is stored once,
// as code << (sh_c - B), which fits int8.  The window holding the most
// channels stays in the channel's own column of q_fold (the main columns);
// every other window is a compacted region of appended columns.  The dgrad
// visits the regions in descending B as one flat K sequence -- appended
// columns [0, H), the main columns [0, base), appended columns [H, D) -- and
// shifts the accumulator left by B_prev - B at each region start and by the
// last B at the end (Horner's rule), which gives the sum exactly.
//   [0] NR     regions (1..kMaxRegions; the main columns are one of them)
//   [1] D      appended columns in use (a multiple of kFoldPad)
//   [2] base   q_fold column of appended column 0 (= roundup(C, kFoldPad))
//   [3] F      final left shift of the accumulator
//   [4] H      appended columns visited before the main columns
//   [8 + r]    flat K column where region r starts (r < NR; INT32_MAX after)
//   [16 + r]   left shift of the accumulator before region r (0 for r = 0)
//   [kLayoutHeader + j], j < ext_max: channel of appended column j, -1 = pad
//   [kLayoutHeader + ext_max + c], c < C: channel descriptor
//              ((pos + 1) << 4) | t: code << t sits in main column c when
//              pos = -1, else in appended column pos (main column c is 0)
// ---------------------------------------------------------------------------
constexpr int kLayoutHeader = 32;
constexpr int kMaxRegions = 8;
constexpr int kFoldPad = 64;        // regions are padded to the GEMM K tile
constexpr int kLayNR = 0, kLayD = 1, kLayBase = 2, kLayF = 3, kLayH = 4, kLayStart = 8, kLayShift = 16;

__host__ __device__ inline int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

// Tile-major code matrix (SQ_LAYOUT_TILED): element (r, k) of a matrix with
// leading dimension ld (a multiple of 64) sits in the 1 KB tile of rows
// 16 (r / 16) .. + 15 and columns 64 (k / 64) .. + 63, the tiles of a row
// group ordered by k, each tile row-major.  The GEMM's operand loads of one
// K tile then read whole 1 KB blocks of memory instead of 64-byte pieces of
// rows far apart.
__host__ __device__ inline int64_t tiled_off(int64_t r, int64_t k, int64_t ld) {
    return (((r >> 4) * (ld >> 6) + (k >> 6)) << 10) + ((r & 15) << 6) + (k & 63);
}

// Host-side constants of one quantizer configuration.
struct QuantCfg {
    int bits;
    int Q;             // 2^(bits-1) - 1
    int num_groups;    // N_G
    int T;             // largest shift with Q * 2^T <= 127
    int round_mode;
    uint64_t seed;
    uint64_t offset;
};

QuantCfg make_cfg(const sq_quant_params& p);

// Worst-case appended columns for C channels: 0 when every shift fits one
// window, else the non-main channels (< C) plus the padding of at most N_G - 1
// appended regions.
int64_t fold_ext_max(int64_t C, const QuantCfg& c);
__host__ __device__ inline int64_t fold_ext_base(int64_t C) { return round_up(C, kFoldPad); }
// Layout words for C channels: header, appended-column list, channel descriptors.
inline int64_t fold_layout_words(int64_t C, const QuantCfg& c) { return kLayoutHeader + fold_ext_max(C, c) + C; }

// ---- quantizer (sq_quant.hip) ----
// First-level abs-max: rows cut into `slabs`, chunks of 4 * tpr channels.
struct ColmaxPlan {
    int vec;
    int tpr;
    int64_t chunks;
    int64_t slabs;
    int64_t rows_per_slab;
};
ColmaxPlan colmax_plan(int64_t M, int64_t C, bool vec);
// uint32 words of scratch: slab maxima, then the channel ranges and the
// per-block maxima of the second reduction level (rbits = partial + slabs * C),
// the second level's shift counts and the abs-max blocks' maxima
int64_t colmax_workspace_words(int64_t M, int64_t C);
// block_max (optional): the maximum of each abs-max block, *n_block_max of them
hipError_t launch_colmax(const float* x, int64_t M, int64_t C, int64_t ld, uint32_t* partial, int64_t* slabs,
                         hipStream_t s, uint32_t* block_max = nullptr, int64_t* n_block_max = nullptr);
hipError_t launch_finalize_grad(const uint32_t* partial, int64_t slabs, int64_t C, const QuantCfg& cfg,
                                uint32_t* rbits, uint8_t* group, sq_scale* scale, int32_t* layout,
                                int64_t ext_max, hipStream_t s);
// abs-max pass + finalize of the gradient quantizer over the scratch ws
// (colmax_workspace_words(M, C) words)
hipError_t launch_colmax_finalize_grad(const float* x, int64_t M, int64_t C, int64_t ld, const QuantCfg& cfg,
                                       uint32_t* ws, uint8_t* group, sq_scale* scale, int32_t* layout,
                                       int64_t ext_max, hipStream_t s);
hipError_t launch_finalize_tensor(const uint32_t* partial, int64_t slabs, int64_t C, int Q, uint32_t* rbits,
                                  sq_scale* scale, hipStream_t s);
// Padded pixel grid of the transposed codes (conv wgrad): row m = (n, oh, ow)
// of an Ho x Wo output grid goes to column n HpWp + oh Wp + ow; Wo = 0: plain
// (column m).  Every value below 2^32.
// Padded pixel grid of a transposed code matrix: pixel m = (n, oh, ow) of an
// Ho x Wo image goes to column n HpWp + oh Wp + ow + off (Wo == 0: no grid).
struct PadGrid {
    uint32_t Wo = 0, HoWo = 0, Wp = 0, HpWp = 0, off = 0;
};
// group == nullptr: every channel in group 0 with shift 0 (per-tensor mode);
// desc: the channel descriptors of the fold layout (nullptr: all main, t = 0).
// tiled: q_fold and q_t tile-major (tiled_off), their K padding (q_fold
// columns [C, roundup(C, 64)), q_t columns [M, roundup(M, 64))) written as
// zeros; not with a padded pixel grid.
hipError_t launch_quantize(const float* x, int64_t M, int64_t C, int64_t ld, const uint8_t* group,
                           const sq_scale* scale, const QuantCfg& cfg,
                           int8_t* q_fold, int64_t ld_fold, int8_t* q_t, int64_t ld_t,
                           const int32_t* desc, hipStream_t s, PadGrid pg = PadGrid(), bool tiled = false);

// Per-channel weight quantization: axis 0 one scale per row, axis 1 one per
// column (partial: colmax scratch, axis 1 only).
hipError_t launch_quantize_channels(const float* x, int64_t rows, int64_t cols, int64_t ld, int bits, int axis,
                                   int transpose, int8_t* q, int64_t ld_q, sq_scale* scales, uint32_t* partial,
                                   hipStream_t s);

// ---- GEMMs (sq_gemm.hip) ----
struct GemmArgs {
    int64_t Mg, Ng;                 // output rows / columns
    const int8_t* A; int64_t lda;   // [Mg, lda], K contiguous
    const int8_t* B; int64_t ldb;   // [Ng, ldb], K contiguous
    int64_t K;
    const int8_t* extA; int64_t ld_extA;   // appended K columns (dgrad fold), may be null
    const int8_t* extB; int64_t ld_extB;
    const int32_t* layout;          // fold layout (dgrad), may be null
    int splits;                     // split-K factor over the main segment
    int32_t* acc; int64_t ld_acc;   // int32 output
    float* out; int64_t ld_out;     // fp32 output
    int32_t* part;                  // split-K: partial tiles [splits, Mg, Ng] instead of acc/out
    int epi_mode;                   // 0: dgrad scale, 1: wgrad per-row scale, 2: per-column scales os[n]
    const sq_scale* gs;
    const sq_scale* os;
    const uint8_t* group;
    int num_groups;
    // Implicit-im2col convolution (conv dgrad), used when taps > 0: output
    // row (n, ih, iw) of [Mg = N * H * W], and A = q_fold rows of the
    // N * Ho * Wo output pixels (a_rows of them).  K visits every 64-column
    // tile of the fold's flat sequence once per tap (r, s) of the KH x KW
    // window, reading A row (n, ih + PH - r, iw + PW - s), or zeros where that
    // pixel lies outside the Ho x Wo grid; B holds the matching weight columns.
    int taps;
    int cv_KW, cv_PH, cv_PW;
    int64_t cv_H, cv_W, cv_Ho, cv_Wo, a_rows;
    int64_t K_used;                 // code columns in use (C_out)
    // device {first K column, K columns} replacing [0, K) (the per-group
    // GEMMs of the GEMM-based comparison), may be null
    const int32_t* kseg;
    // with out: max |out| per 32-row slab and column, as bit patterns,
    // [ceil(Mg / 32), Ng] (producer-side channel ranges of the next quantizer)
    uint32_t* ranges;
    // A, B, extA and extB tile-major (tiled_off; leading dimensions multiples
    // of 64, K a multiple of 64); extA is then the whole fold matrix and its
    // appended columns start at column ext_koff
    int tiled;
    int64_t ext_koff;
};

hipError_t launch_gemm(const GemmArgs& a, hipStream_t s);
// whether the direct-load pipelined kernel takes the product
bool gemm_pipe_ok(const GemmArgs& a);
// max |x| per 32-row slab and column (bit patterns): ranges [ceil(M / 32), N]
hipError_t launch_slab_colmax(const float* x, int64_t M, int64_t N, int64_t ld, uint32_t* ranges, hipStream_t s);
hipError_t launch_gather_ext(const int8_t* wq_t, int64_t ld_w, int64_t C_in, const int32_t* layout,
                             int8_t* wext, int64_t ld_ext, int64_t ext_max, hipStream_t s, bool tiled = false);
// Conv dgrad: B operand [C_in, ld_bc] in the order of the conv K sequence;
// conv_bc_ld(C_out, taps, ext_max) is its leading dimension, enough for any fold.
inline int64_t conv_bc_ld(int64_t C_out, int64_t taps, int64_t ext_max) {
    return round_up(taps * (round_up(C_out, kFoldPad) + ext_max), 64);
}
// Conv dgrad: a describes the product with a.B = wq_t (W^T codes [taps * C_in,
// ld_w]); kernels that need the weights in the K order of the implicit GEMM
// gather them into bc first.
// With a.ranges (and a.out): per-slab channel maxima of |dX|, slab s covering
// rows [s R, (s + 1) R), R returned in *range_rows.
hipError_t launch_conv_dgrad(const GemmArgs& a, int8_t* bc, int64_t ld_bc, hipStream_t s,
                             int64_t* range_rows = nullptr);
// GEMM-based loss propagation (comparison for ShiftMM): group plan,
// rearranged operands, per-group products, shift-and-sum.
int64_t grouped_width(int64_t C_out, int num_groups);
hipError_t launch_group_plan(const uint8_t* group, int64_t C, int num_groups, const int32_t* desc, int64_t base_col,
                             int32_t* plan, int64_t wmax, hipStream_t s);
hipError_t launch_gather_cols(const int8_t* src, int64_t ld_src, int64_t rows, const int32_t* col, int64_t wmax,
                              int8_t* dst, int64_t ld_dst, hipStream_t s);
hipError_t launch_group_combine(const int32_t* part, int num_groups, int64_t M, int64_t N, int32_t* acc,
                                int64_t ld_acc, float* out, int64_t ld_out, const sq_scale* gs, const sq_scale* os,
                                hipStream_t s);
hipError_t launch_splitk_reduce(const int32_t* ws, int splits, const GemmArgs& a, hipStream_t s);
hipError_t launch_dequant(const int32_t* acc, int64_t rows, int64_t cols, int64_t ld_acc, int kind,
                          const uint8_t* group, const sq_scale* gs, const sq_scale* os,
                          int num_groups, float* out, int64_t ld_out, hipStream_t s);
int wgrad_splits(int64_t M, int64_t C_out, int64_t C_in);

// Padded pixel grids of the implicit-im2col conv wgrad (see sq_conv_wgrad):
// out[c, G] for G < ld_out (a multiple of 16), G = n Hp Wp + hp Wp + wp, is
// pixel (n, hp - top, wp - left) of the content grid Hc x Wc of image n, i.e.
// in[c, (n Hc + h) Wc + w], or 0 outside the content.  Wp and ld_in are
// multiples of 16, in 16-byte aligned.
hipError_t launch_grid_pack(const int8_t* in, int64_t ld_in, int64_t C, int64_t N, int64_t Hc, int64_t Wc,
                            int64_t top, int64_t left, int64_t Hp, int64_t Wp, int8_t* out, int64_t ld_out,
                            hipStream_t s);

// Implicit-im2col conv wgrad from one copy of the input grid (k_conv_wgrad):
// acc[co, (r KW + s) C_in + ci] = sum_P A[co, P] X[ci, P + r Wp + s] over
// P < K (K a multiple of 64); X rows readable (zeros) through column
// K + (KH - 1) Wp + 64.  The plan fixes the kernel variant, the tiles and the
// K splits; splits > 1 write int32 partials [splits, C_out, KH KW C_in] to
// `part`, which launch_splitk_reduce then sums with the epilogue.
struct ConvWgradPlan {
    int fm = 1, kwc = 0, rbc = 0;   // output-channel fragments per block, compile-time KW / tap rows (0: runtime)
    int rb = 1, tap_groups = 1;     // tap rows per block and blocks along the window height
    int64_t tiles_ci = 1, tiles = 1;
    int64_t chunks = 0;             // 16-tile K chunks
    int splits = 1, per = 1;        // K splits, chunks per split
};
ConvWgradPlan conv_wgrad_plan(int64_t K, int64_t C_out, int64_t C_in, int KH, int KW, int64_t Wp);
struct ConvWgradArgs {
    const int8_t* A; int64_t lda;   // gradient codes on the grid [C_out, lda]
    const int8_t* X; int64_t ldx;   // input codes on the grid [C_in, ldx]
    int64_t C_out, C_in, Wp, ktiles;
    int KH, KW;
    int32_t* part;                  // split K: partials [splits, C_out, KH KW C_in]
    int32_t* acc; int64_t ld_acc;   // no split: int32 and / or fp32 outputs
    float* out; int64_t ld_out;
    const uint8_t* group;
    const sq_scale* gs;
    const sq_scale* os;
};
hipError_t launch_conv_wgrad(const ConvWgradArgs& a, const ConvWgradPlan& plan, hipStream_t s);

// ---- L1BNQ (sq_l1bn.hip) ----
// Partial-maximum slabs of the backward's dx ranges; int32 partial words of
// the column sums.
int64_t l1bn_range_slabs(int64_t M, int64_t C);
int64_t l1bn_part_words(int64_t M, int64_t C);
hipError_t launch_l1bn_forward(const int8_t* xq, int64_t M, int64_t C, int64_t ld_x, const sq_scale* xs,
                               const float* gamma, const float* beta, float* y, int64_t ld_y, sq_l1bn_channel* ch,
                               sq_l1bn_layer* layer, int32_t* part, hipStream_t s);
// After the gradient codes qg [M, ldg] are formed: sums, constants
// (coef [C, 4] scratch), dx and its ranges.
hipError_t launch_l1bn_backward(const int8_t* qg, int64_t ldg, const int8_t* xq, int64_t ld_x, int64_t M, int64_t C,
                                const sq_l1bn_channel* ch, const sq_l1bn_layer* layer, const uint8_t* group,
                                const sq_scale* gscale, float* dx, int64_t ld_dx, float* dgamma, float* dbeta,
                                uint32_t* ranges, int32_t* part, float* coef, hipStream_t s);

// ---- device helpers ----
// 2^k as a float, exact for -126 <= k <= 127 (from its bit pattern).
__device__ __forceinline__ float pow2f(int k) { return __uint_as_float((uint32_t)(k + 127) << 23); }

}  // namespace sq
