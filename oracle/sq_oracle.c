/*
 * ShiftQuant backward path: CPU ORACLE.  TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow C implementation of what the GPU path computes, written
 * from "Towards Accurate and Efficient Sub-8-Bit Integer Training" (arXiv
 * 2411.10948).  The outer loops over independent outputs (channels, rows,
 * output elements) carry OpenMP pragmas; every output is still computed by
 * one thread in the plain loop order, so the results do not depend on the
 * thread count (sqo_set_threads; one thread unless set).  Only the tests, the smoke check and the
 * benchmark's CPU-baseline leg may load it; the product library never does.
 * It shares no code, header or table with the HIP sources.
 *
 * Floating point: IEEE binary32, round-to-nearest-even, no contraction
 * (built with -ffp-contract=off -fno-fast-math), denormals kept.
 * Integer GEMMs accumulate in int64 and are range-checked against int32.
 *
 * Readings of the paper that these functions follow (the paper is silent,
 * ambiguous or self-inconsistent on each):
 *  R1 thresholds decrease from tau_0 = r_max: tau_g = r_max * 2^-g and the
 *     0-indexed group g holds channel ranges in (tau_{g+1}, tau_g]; the last
 *     group also takes everything down to 0 (Sec. 3.1 grouping objective
 *     constraints and the power-of-two threshold equation).
 *  R2 the range of a channel is its absolute maximum and the zero point is 0
 *     (symmetric quantization; Eq. dq_mm_f has no zero-point term).
 *  R3 b-bit codes take values in [-Q, Q] with Q = 2^(b-1) - 1.
 *  R4 group 0 (the one that holds r_max) uses the step r_max / Q and group g
 *     the step (r_max / Q) * 2^-g (App. D per-group formula, 0-indexed).
 *  R5 scaling multiplies by the scale s = fl(Q / r_max) * 2^g, as App. B
 *     writes SR(X S) S^-1; the dequantization factor is fl(r_max / Q).
 *  R6 deterministic rounding is round-half-to-even; stochastic rounding draws
 *     a 16-bit uniform from Philox4x32-10 (see sqo_quantize_grad).
 *  R7 codes are clamped to [-Q, Q] after rounding.
 *  R8 the dgrad accumulator is the left-shift form of App. D (each group's
 *     product shifted left by N_G-1-g); the wgrad accumulator is unshifted and
 *     its group scale is applied per output row.
 *  R9 a tensor whose absolute maximum is NaN/Inf is flagged NONFINITE, one
 *     whose maximum is below 2^-96 (including 0) is flagged ZERO; both give
 *     all-zero codes, every channel in the last group and zero scales.
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define SQO_OK 0
#define SQO_ERR_ARG 1
#define SQO_ERR_RANGE 2

#define SQO_FLAG_NONFINITE 1u
#define SQO_FLAG_ZERO 2u

typedef struct {
    float r_max;   /* tau_0: absolute maximum of the tensor               */
    float inv0;    /* s_{G_B} = fl(Q / r_max): scale of group 0            */
    float d0;      /* s_{G_B}^-1 = fl(r_max / Q): step of group 0          */
    uint32_t flags;
} sqo_scale;

static uint32_t f2u(float f) { uint32_t u; memcpy(&u, &f, 4); return u; }
static float u2f(uint32_t u) { float f; memcpy(&f, &u, 4); return f; }

/* 2^k as a float, exact for -126 <= k <= 127 (built from its bit pattern). */
static float pow2f(int k) { return u2f((uint32_t)(k + 127) << 23); }

static int32_t qmax_of(int bits) { return (1 << (bits - 1)) - 1; }

/* Thread count of the OpenMP loops (1 = the plain serial program). */
static int g_threads = 1;
int sqo_set_threads(int n) { g_threads = n > 0 ? n : 1; return g_threads; }
int sqo_max_threads(void) { return omp_get_num_procs(); }

/* ---------------------------------------------------------------------------
 * Philox4x32-10, Salmon, Moraes, Dror and Shaw, "Parallel random numbers: as
 * easy as 1, 2, 3", SC'11.  One round maps the counter (x0,x1,x2,x3) with key
 * (k0,k1) through two 32x32->64-bit products with the multipliers
 * 0xD2511F53 and 0xCD9E8D57; the key is bumped by the Weyl constants
 * 0x9E3779B9 and 0xBB67AE85 between rounds.
 * ------------------------------------------------------------------------- */
void sqo_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4])
{
    uint32_t x0 = ctr[0], x1 = ctr[1], x2 = ctr[2], x3 = ctr[3];
    uint32_t k0 = key[0], k1 = key[1];
    for (int round = 0; round < 10; ++round) {
        uint64_t p0 = (uint64_t)0xD2511F53u * x0;
        uint64_t p1 = (uint64_t)0xCD9E8D57u * x2;
        uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
        uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
        uint32_t y0 = hi1 ^ x1 ^ k0;
        uint32_t y1 = lo1;
        uint32_t y2 = hi0 ^ x3 ^ k1;
        uint32_t y3 = lo0;
        x0 = y0; x1 = y1; x2 = y2; x3 = y3;
        k0 += 0x9E3779B9u;
        k1 += 0xBB67AE85u;
    }
    out[0] = x0; out[1] = x1; out[2] = x2; out[3] = x3;
}

/* The 16-bit uniform integer that stochastic rounding compares against for
 * the element with logical index idx = m * C + c: one Philox block serves 8
 * consecutive indices.  counter = (idx / 8 split into two words, offset
 * split into two words), key = seed split into two words; the element takes
 * 16-bit half (idx % 2) (low half first) of output word (idx / 2) % 4. */
uint32_t sqo_sr_uniform16(uint64_t idx, uint64_t seed, uint64_t offset)
{
    uint64_t blk = idx >> 3;
    uint32_t ctr[4] = {(uint32_t)blk, (uint32_t)(blk >> 32), (uint32_t)offset, (uint32_t)(offset >> 32)};
    uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    uint32_t w[4];
    sqo_philox4x32_10(ctr, key, w);
    return (w[(idx >> 1) & 3u] >> (16u * (uint32_t)(idx & 1u))) & 0xFFFFu;
}

/* ---------------------------------------------------------------------------
 * Sec. 3.1: r_i is the range of channel i (R2: its absolute maximum).
 * The absolute value is taken on the bit pattern (sign bit cleared) and the
 * maximum on the unsigned pattern, which orders every non-NaN float by value
 * and places NaN above +Inf.  nonfinite is set when any element is NaN/Inf.
 * ------------------------------------------------------------------------- */
int sqo_channel_range(const float* x, int64_t M, int64_t C, int64_t ld, float* r, int* nonfinite)
{
    if (!x || !r || M < 0 || C < 0 || ld < C) return SQO_ERR_ARG;
    int nf = 0;
#pragma omp parallel for num_threads(g_threads) reduction(|:nf) schedule(static)
    for (int64_t c = 0; c < C; ++c) {
        uint32_t best = 0;
        for (int64_t m = 0; m < M; ++m) {
            uint32_t a = f2u(x[m * ld + c]) & 0x7FFFFFFFu;
            if (a >= 0x7F800000u) nf = 1;
            if (a > best) best = a;
        }
        r[c] = u2f(best);
    }
    if (nonfinite) *nonfinite = nf;
    return SQO_OK;
}

/* Sec. 3.1, power-of-two grouping (R1): group g of channel c is the first g
 * whose lower threshold tau_{g+1} = r_max * 2^-(g+1) lies strictly below r_c;
 * the last group N_G-1 takes the rest (tau_{N_G} = 0). */
int sqo_group_of(float r_c, float r_max, int num_groups)
{
    for (int g = 0; g < num_groups - 1; ++g) {
        float tau_next = r_max * pow2f(-(g + 1));
        if (r_c > tau_next) return g;
    }
    return num_groups - 1;
}

static int check_qparams(int bits, int num_groups)
{
    return (bits >= 2 && bits <= 8 && num_groups >= 1 && num_groups <= 8) ? SQO_OK : SQO_ERR_ARG;
}

/* ---------------------------------------------------------------------------
 * ShiftQuant of the output gradient G_B = dY [M, C] (App. D, App. B Eq. sq).
 *   Q = 2^(bits-1) - 1, s = fl(Q / r_max), d = fl(r_max / Q)     (R3, R5)
 *   channel c in group g_c uses the scale s * 2^{g_c}              (R4)
 *   v = fl(x * (s * 2^{g_c}))
 *   round_mode 0: q = clamp(round_half_even(v), -Q, Q)             (R6, R7)
 *   round_mode 1: l = floor(v), f = fl(v - l);  q = l + 1 with probability
 *     f (App. B Eq. sq), realised as [u16 < f * 2^16] with u16 from
 *     sqo_sr_uniform16(m * C + c, seed, offset), so P(l + 1) = ceil(f 2^16) /
 *     2^16 (a bias below 2^-16 steps); then clamp.
 * Outputs q [M, C] (row stride C), g [C], *scale.
 * ------------------------------------------------------------------------- */
int sqo_quantize_grad(const float* dY, int64_t M, int64_t C, int64_t ld, int bits, int num_groups,
                      int round_mode, uint64_t seed, uint64_t offset,
                      int8_t* q, uint8_t* g, float* r_out, sqo_scale* scale)
{
    if (!dY || !q || !g || !scale || M < 0 || C < 0 || ld < C) return SQO_ERR_ARG;
    if (check_qparams(bits, num_groups) || (round_mode != 0 && round_mode != 1)) return SQO_ERR_ARG;
    const int32_t Q = qmax_of(bits);

    /* channel ranges r_c and the tensor range tau_0 = r_max */
    float* r = r_out ? r_out : (float*)malloc(sizeof(float) * (size_t)(C > 0 ? C : 1));
    if (!r) return SQO_ERR_ARG;
    int nonfinite = 0;
    sqo_channel_range(dY, M, C, ld, r, &nonfinite);
    uint32_t rmax_bits = 0;
    for (int64_t c = 0; c < C; ++c)
        if (f2u(r[c]) > rmax_bits) rmax_bits = f2u(r[c]);
    float r_max = u2f(rmax_bits);
    scale->r_max = r_max;
    scale->flags = 0;
    if (nonfinite) scale->flags = SQO_FLAG_NONFINITE;
    else if (r_max < pow2f(-96)) scale->flags = SQO_FLAG_ZERO;
    if (scale->flags) {
        scale->inv0 = 0.0f;
        scale->d0 = 0.0f;
        for (int64_t c = 0; c < C; ++c) g[c] = (uint8_t)(num_groups - 1);
        memset(q, 0, (size_t)(M * C));
        if (!r_out) free(r);
        return SQO_OK;
    }
    scale->inv0 = (float)Q / r_max;
    scale->d0 = r_max / (float)Q;

    /* group of each channel */
    for (int64_t c = 0; c < C; ++c) g[c] = (uint8_t)sqo_group_of(r[c], r_max, num_groups);
    if (!r_out) free(r);

    const float two16 = pow2f(16);
#pragma omp parallel for num_threads(g_threads) schedule(static)
    for (int64_t m = 0; m < M; ++m) {
        for (int64_t c = 0; c < C; ++c) {
            float s_c = scale->inv0 * pow2f(g[c]);
            float v = dY[m * ld + c] * s_c;
            float qf;
            if (round_mode == 0) {
                qf = rintf(v);
            } else {
                float l = floorf(v);
                float f = v - l;
                uint32_t u = sqo_sr_uniform16((uint64_t)(m * C + c), seed, offset);
                qf = ((float)u < f * two16) ? l + 1.0f : l;
            }
            if (qf > (float)Q) qf = (float)Q;
            if (qf < (float)-Q) qf = (float)-Q;
            q[m * C + c] = (int8_t)(int32_t)qf;
        }
    }
    return SQO_OK;
}

/* Per-tensor symmetric quantization of W or X: the paper's INT8 baseline
 * quantizes weights, activations and gradients per tensor (Sec. 5.1).
 *   a = max |T|, s = fl(Q / a), d = fl(a / Q), t = clamp(rint(fl(T * s)), -Q, Q)
 * Same flag rules as the gradient quantizer (R9).  Output q [rows, cols]. */
int sqo_quantize_tensor(const float* T, int64_t rows, int64_t cols, int64_t ld, int bits,
                        int8_t* q, sqo_scale* scale)
{
    if (!T || !q || !scale || rows < 0 || cols < 0 || ld < cols || bits < 2 || bits > 8) return SQO_ERR_ARG;
    const int32_t Q = qmax_of(bits);
    uint32_t amax = 0;
    int nonfinite = 0;
    for (int64_t i = 0; i < rows; ++i)
        for (int64_t j = 0; j < cols; ++j) {
            uint32_t a = f2u(T[i * ld + j]) & 0x7FFFFFFFu;
            if (a >= 0x7F800000u) nonfinite = 1;
            if (a > amax) amax = a;
        }
    float a = u2f(amax);
    scale->r_max = a;
    scale->flags = nonfinite ? SQO_FLAG_NONFINITE : (a < pow2f(-96) ? SQO_FLAG_ZERO : 0u);
    if (scale->flags) {
        scale->inv0 = 0.0f;
        scale->d0 = 0.0f;
        memset(q, 0, (size_t)(rows * cols));
        return SQO_OK;
    }
    scale->inv0 = (float)Q / a;
    scale->d0 = a / (float)Q;
    for (int64_t i = 0; i < rows; ++i)
        for (int64_t j = 0; j < cols; ++j) {
            float v = rintf(T[i * ld + j] * scale->inv0);
            if (v > (float)Q) v = (float)Q;
            if (v < (float)-Q) v = (float)-Q;
            q[i * cols + j] = (int8_t)(int32_t)v;
        }
    return SQO_OK;
}

/* ---------------------------------------------------------------------------
 * Per-channel symmetric quantization of a weight matrix (Sec. 5.1: weights
 * are quantized per output channel in the forward pass and per input channel
 * in loss propagation).  axis 0: one scale per row of T, axis 1: one per
 * column.  Each channel is quantized like a tensor of its own: amax over the
 * channel, inv = fl(Q / amax), step = fl(amax / Q), code = clamp(rint(fl(x *
 * inv)), -Q, Q); a channel whose amax is NaN/Inf or below 2^-96 gets its flag
 * and all-zero codes.  q is [rows, cols]; scales has rows (axis 0) or cols
 * (axis 1) entries.
 * ------------------------------------------------------------------------- */
int sqo_quantize_channels(const float* T, int64_t rows, int64_t cols, int64_t ld, int bits, int axis,
                          int8_t* q, sqo_scale* scales)
{
    if (!T || !q || !scales || rows < 0 || cols < 0 || ld < cols || bits < 2 || bits > 8 || (axis != 0 && axis != 1))
        return SQO_ERR_ARG;
    const int32_t Q = qmax_of(bits);
    int64_t nch = axis == 0 ? rows : cols, len = axis == 0 ? cols : rows;
    for (int64_t ch = 0; ch < nch; ++ch) {
        uint32_t amax = 0;
        int nonfinite = 0;
        for (int64_t e = 0; e < len; ++e) {
            float x = axis == 0 ? T[ch * ld + e] : T[e * ld + ch];
            uint32_t a = f2u(x) & 0x7FFFFFFFu;
            if (a >= 0x7F800000u) nonfinite = 1;
            if (a > amax) amax = a;
        }
        sqo_scale* sc = &scales[ch];
        float a = u2f(amax);
        sc->r_max = a;
        sc->flags = nonfinite ? SQO_FLAG_NONFINITE : (a < pow2f(-96) ? SQO_FLAG_ZERO : 0u);
        sc->inv0 = sc->flags ? 0.0f : (float)Q / a;
        sc->d0 = sc->flags ? 0.0f : a / (float)Q;
        for (int64_t e = 0; e < len; ++e) {
            int64_t i = axis == 0 ? ch : e, j = axis == 0 ? e : ch;
            float v = sc->flags ? 0.0f : rintf(T[i * ld + j] * sc->inv0);
            if (v > (float)Q) v = (float)Q;
            if (v < (float)-Q) v = (float)-Q;
            q[i * cols + j] = (int8_t)(int32_t)v;
        }
    }
    return SQO_OK;
}

/* Dequantization with one weight scale per output column (the forward pass
 * with per-output-channel weights, or loss propagation with per-input-channel
 * weights; Eq. dq_mm_f with S_W per channel):
 *   gamma_k = fl(fl(d_a * d_w[k]) * 2^-(N_G-1)),   out[i, k] = fl(float(A[i, k]) * gamma_k). */
void sqo_dequant_cols(const int32_t* A, int64_t n_rows, int64_t n_cols, float d_a, const float* d_w, int num_groups,
                      float* out)
{
    for (int64_t k = 0; k < n_cols; ++k) {
        float gamma = (d_a * d_w[k]) * pow2f(-(num_groups - 1));
        for (int64_t i = 0; i < n_rows; ++i) out[i * n_cols + k] = (float)A[i * n_cols + k] * gamma;
    }
}

/* ---------------------------------------------------------------------------
 * Loss propagation (Eq. dq_mm_f and App. D, left-shift form, R8):
 *   A[n, k] = sum_c  (q[n, c] * wq[c, k]) << (N_G - 1 - g_c)
 * ShiftMM (Sec. 3.2) shifts each product before it is accumulated; that is
 * what this loop does, in int64.  q [M, C_out], wq [C_out, C_in] (W in the
 * PyTorch layout, so dX = dY . W).  Only the rows listed in `rows` (or all
 * rows when rows == NULL) are computed, into A [n_rows, C_in].
 * ------------------------------------------------------------------------- */
int sqo_dgrad(const int8_t* q, int64_t M, int64_t C_out, const uint8_t* g, int num_groups,
              const int8_t* wq, int64_t C_in, const int64_t* rows, int64_t n_rows, int32_t* A)
{
    if (!q || !g || !wq || !A || num_groups < 1 || num_groups > 8) return SQO_ERR_ARG;
    int64_t nr = rows ? n_rows : M;
    for (int64_t i = 0; i < nr; ++i)
        if (rows && (rows[i] < 0 || rows[i] >= M)) return SQO_ERR_ARG;
    int err = SQO_OK;
#pragma omp parallel for num_threads(g_threads) schedule(dynamic, 1)
    for (int64_t i = 0; i < nr; ++i) {
        int64_t n = rows ? rows[i] : i;
        for (int64_t k = 0; k < C_in; ++k) {
            int64_t acc = 0;
            for (int64_t c = 0; c < C_out; ++c) {
                int shift = num_groups - 1 - (int)g[c];
                int64_t prod = (int64_t)q[n * C_out + c] * (int64_t)wq[c * C_in + k];
                acc += prod * ((int64_t)1 << shift);
            }
            if (acc > INT32_MAX || acc < INT32_MIN) {
#pragma omp atomic write
                err = SQO_ERR_RANGE;
            }
            A[i * C_in + k] = (int32_t)acc;
        }
    }
    return err;
}

/* ---------------------------------------------------------------------------
 * Loss propagation of a stride-1 convolution lowered to the GEMM of
 * Eq. dq_mm_f by im2col (the ResNet layers of Sec. 5 are convolutions).  The
 * forward conv reads, for output pixel (n, oh, ow), the input pixels
 * (n, oh + r - PH, ow + s - PW) of the KH x KW window, and im2col orders a
 * column row as (r, s, ci); W is [C_out, KH * KW * C_in] in that order.  The
 * input gradient is the col2im (the adjoint of im2col) of the im2col'd dgrad:
 *   A[(n, ih, iw), ci] = sum_{r, s} sum_co (q[(n, oh, ow), co] * wq[co, (r, s, ci)]) << sh_co
 * with oh = ih + PH - r and ow = iw + PW - s, terms outside the Ho x Wo output
 * grid being absent; sh_co = N_G - 1 - g_co as in sqo_dgrad.  q is the code
 * matrix of dY [N * Ho * Wo, C_out] (NHWC), Ho = H + 2 PH - KH + 1 and
 * Wo = W + 2 PW - KW + 1.  `pix` lists input pixels (n * H + ih) * W + iw
 * (NULL = all N * H * W of them); A is [n_pix, C_in], accumulated in int64.
 * ------------------------------------------------------------------------- */
int sqo_conv_dgrad(const int8_t* q, int64_t N, int64_t H, int64_t W, int64_t C_out, const uint8_t* g,
                   int num_groups, const int8_t* wq, int64_t C_in, int KH, int KW, int PH, int PW,
                   const int64_t* pix, int64_t n_pix, int32_t* A)
{
    if (!q || !g || !wq || !A || num_groups < 1 || num_groups > 8) return SQO_ERR_ARG;
    if (N < 0 || H < 1 || W < 1 || C_out < 0 || C_in < 0 || KH < 1 || KW < 1 || PH < 0 || PW < 0)
        return SQO_ERR_ARG;
    int64_t Ho = H + 2 * (int64_t)PH - KH + 1, Wo = W + 2 * (int64_t)PW - KW + 1;
    if (Ho < 1 || Wo < 1) return SQO_ERR_ARG;
    int64_t taps_ci = (int64_t)KH * KW * C_in;   /* columns of W */
    int64_t np = pix ? n_pix : N * H * W;
    for (int64_t i = 0; i < np; ++i)
        if (pix && (pix[i] < 0 || pix[i] >= N * H * W)) return SQO_ERR_ARG;
    int err = SQO_OK;
#pragma omp parallel for num_threads(g_threads) schedule(dynamic, 16)
    for (int64_t i = 0; i < np; ++i) {
        int64_t p = pix ? pix[i] : i;
        int64_t n = p / (H * W), ih = (p / W) % H, iw = p % W;
        for (int64_t ci = 0; ci < C_in; ++ci) {
            int64_t acc = 0;
            for (int r = 0; r < KH; ++r) {
                int64_t oh = ih + PH - r;
                if (oh < 0 || oh >= Ho) continue;
                for (int s = 0; s < KW; ++s) {
                    int64_t ow = iw + PW - s;
                    if (ow < 0 || ow >= Wo) continue;
                    const int8_t* qrow = q + ((n * Ho + oh) * Wo + ow) * C_out;
                    int64_t col = ((int64_t)r * KW + s) * C_in + ci;
                    for (int64_t co = 0; co < C_out; ++co) {
                        int shift = num_groups - 1 - (int)g[co];
                        int64_t prod = (int64_t)qrow[co] * (int64_t)wq[co * taps_ci + col];
                        acc += ((int64_t)1 << shift) * prod;
                    }
                }
            }
            if (acc > INT32_MAX || acc < INT32_MIN) {
#pragma omp atomic write
                err = SQO_ERR_RANGE;
            }
            A[i * C_in + ci] = (int32_t)acc;
        }
    }
    return err;
}

/* Weight gradient (the third training GEMM, Fig. "MMs"): inner dimension is
 * the token index, so each output row c lies in one gradient group:
 *   B[c, k] = sum_m q[m, c] * xq[m, k]            (unshifted, R8)
 * q [M, C_out], xq [M, C_in]; rows lists output channels c (NULL = all). */
int sqo_wgrad(const int8_t* q, int64_t M, int64_t C_out, const int8_t* xq, int64_t C_in,
              const int64_t* rows, int64_t n_rows, int32_t* B)
{
    if (!q || !xq || !B) return SQO_ERR_ARG;
    int64_t nr = rows ? n_rows : C_out;
    for (int64_t i = 0; i < nr; ++i)
        if (rows && (rows[i] < 0 || rows[i] >= C_out)) return SQO_ERR_ARG;
    int err = SQO_OK;
#pragma omp parallel for num_threads(g_threads) collapse(2) schedule(dynamic, 16)
    for (int64_t i = 0; i < nr; ++i) {
        for (int64_t k = 0; k < C_in; ++k) {
            int64_t c = rows ? rows[i] : i;
            int64_t acc = 0;
            for (int64_t m = 0; m < M; ++m)
                acc += (int64_t)q[m * C_out + c] * (int64_t)xq[m * C_in + k];
            if (acc > INT32_MAX || acc < INT32_MIN) {
#pragma omp atomic write
                err = SQO_ERR_RANGE;
            }
            B[i * C_in + k] = (int32_t)acc;
        }
    }
    return err;
}

/* Dequantization of the dgrad accumulator (Eq. dq_mm_f: the product of the two
 * inverse scales stays outside the integer sum; App. D left-shift form adds
 * 2^-(N_G-1) for the 0-indexed groups):
 *   alpha = fl(fl(d_G * d_W) * 2^-(N_G-1)),   dX = fl(float(A) * alpha). */
void sqo_dequant_dgrad(const int32_t* A, int64_t n, float d_grad, float d_w, int num_groups, float* out)
{
    float alpha = (d_grad * d_w) * pow2f(-(num_groups - 1));
#pragma omp parallel for num_threads(g_threads) schedule(static)
    for (int64_t i = 0; i < n; ++i) out[i] = (float)A[i] * alpha;
}

/* Dequantization of the wgrad accumulator: output row c carries its group's
 * step d_G * 2^-g_c times the activation step d_X:
 *   beta_c = fl(fl(d_G * d_X) * 2^-g_c),      dW[c, k] = fl(float(B[c, k]) * beta_c). */
void sqo_dequant_wgrad(const int32_t* B, int64_t n_rows, int64_t C_in, const uint8_t* g_rows,
                       float d_grad, float d_x, float* out)
{
#pragma omp parallel for num_threads(g_threads) schedule(static)
    for (int64_t i = 0; i < n_rows; ++i) {
        float beta = (d_grad * d_x) * pow2f(-(int)g_rows[i]);
        for (int64_t k = 0; k < C_in; ++k) out[i * C_in + k] = (float)B[i * C_in + k] * beta;
    }
}

/* ---------------------------------------------------------------------------
 * Fully-quantized L1 batch normalization (L1BNQ), Sec. 4 (Fig. l1bnq) and
 * App. C.  The paper draws the layer as a figure and states only the
 * normalization equations, so this follows two readings:
 *
 *  R16 forward.  The layer's input is the 8-bit per-tensor code q of x (step
 *      s_x); statistics are per channel c over the M rows (N*H*W) of the batch.
 *      The mean is quantized onto the input's own grid,
 *        m_c = round_half_even(S_c / M),  S_c = sum_m q[m, c],
 *      so x - mu^q = s_x (q - m_c) exactly.  sigma is the L1 deviation
 *      (App. C.1) taken as a mean, sigma_c = s_x A_c / M with
 *      A_c = sum_m |q - m_c|, and is quantized per tensor to 8 bits under the
 *      step max_c sigma_c / 127:
 *        k_c = max(1, round_half_even(127 A_c / A_max)),  A_max = max_c A_c,
 *      (s_x and M cancel in the ratio; the smallest code is kept at 1 so the
 *      denominator of the quantized normalization of App. C.2 is never 0).
 *      gamma and beta are quantized per tensor to 8 bits like W and X.  Then
 *        kappa_c = fl32(gamma^q_c * 127 M / (A_max k_c))   (binary64),
 *        y = fl(fl(kappa_c * (q - m_c)) + beta^q_c).
 *      A_max = 0 (every channel constant): kappa = 0, k = 0, y = beta^q.
 *  R17 backward.  The derivative of the L1 normalization (App. C.1's
 *      derivation with sigma = mean |x - mu|, which brings in the signs
 *      s = sgn(x - mu)), the quantizers of mu and sigma passed straight
 *      through:  dx = (gamma / sigma)(g - mean g - mean(g xhat)(s - mean s)).
 *      The incoming gradient is quantized with ShiftQuant (codes qg, channel
 *      steps delta_c = d0 2^-g_c), so the channel sums are integers:
 *        G1 = sum qg,  G2 = sum qg (q - m),  P = sum sgn(q - m).
 *      With rho = 127 M / (A_max k) (xhat per code step) and
 *      lambda = gamma^q rho / s_x (gamma^q / sigma^q), in binary64:
 *        dbeta = delta G1,  dgamma = (delta G2) rho,  D = dgamma / M,
 *        a = lambda delta,  b = -(lambda D),  e = lambda (D P / M - delta G1 / M),
 *      each rounded once to binary32, and
 *        dx = fl(fl(fl(a qg) + fl(b sgn(q - m))) + e).
 *      A_max = 0: dgamma = 0 and dx = 0.
 * ------------------------------------------------------------------------- */

/* round_half_even(num / den) of integers, den > 0 */
static int64_t div_round_even(int64_t num, int64_t den)
{
    int64_t q = num / den, r = num % den;
    if (r < 0) { q -= 1; r += den; }          /* floor division, 0 <= r < den */
    if (2 * r > den || (2 * r == den && (q & 1))) q += 1;
    return q;
}

int sqo_l1bn_forward(const int8_t* q, int64_t M, int64_t C, float x_step, const float* gamma,
                     const float* beta, float* y, int32_t* mu, int32_t* sigma, int32_t* sign_sum,
                     int64_t* dev_sum, float* gamma_q, float* beta_q, float* kappa, int64_t* dev_max)
{
    if (!q || !gamma || !beta || !y || !mu || !sigma || !sign_sum || !dev_sum || !gamma_q || !beta_q ||
        !kappa || !dev_max || M < 1 || C < 0)
        return SQO_ERR_ARG;
    (void)x_step;   /* cancels out of the normalized value */
    int64_t amax = 0;
    for (int64_t c = 0; c < C; ++c) {
        int64_t S = 0;
        for (int64_t m = 0; m < M; ++m) S += q[m * C + c];
        int64_t mc = div_round_even(S, M);
        int64_t A = 0, P = 0;
        for (int64_t m = 0; m < M; ++m) {
            int64_t d = (int64_t)q[m * C + c] - mc;
            A += d < 0 ? -d : d;
            P += (d > 0) - (d < 0);
        }
        mu[c] = (int32_t)mc;
        dev_sum[c] = A;
        sign_sum[c] = (int32_t)P;
        if (A > amax) amax = A;
    }
    *dev_max = amax;
    /* parameters: 8-bit per-tensor codes */
    int8_t* gc = (int8_t*)malloc((size_t)(C > 0 ? C : 1));
    int8_t* bc = (int8_t*)malloc((size_t)(C > 0 ? C : 1));
    sqo_scale gs, bs;
    if (!gc || !bc) { free(gc); free(bc); return SQO_ERR_ARG; }
    sqo_quantize_tensor(gamma, 1, C, C, 8, gc, &gs);
    sqo_quantize_tensor(beta, 1, C, C, 8, bc, &bs);
    for (int64_t c = 0; c < C; ++c) {
        gamma_q[c] = gs.d0 * (float)gc[c];
        beta_q[c] = bs.d0 * (float)bc[c];
        if (amax == 0) {
            sigma[c] = 0;
            kappa[c] = 0.0f;
        } else {
            int64_t k = div_round_even(127 * dev_sum[c], amax);
            if (k < 1) k = 1;
            sigma[c] = (int32_t)k;
            double num = (double)gamma_q[c] * (127.0 * (double)M);
            kappa[c] = (float)(num / ((double)amax * (double)k));
        }
    }
    free(gc);
    free(bc);
    for (int64_t m = 0; m < M; ++m)
        for (int64_t c = 0; c < C; ++c) {
            float d = (float)((int32_t)q[m * C + c] - mu[c]);
            y[m * C + c] = kappa[c] * d + beta_q[c];
        }
    return SQO_OK;
}

int sqo_l1bn_backward(const int8_t* qg, const uint8_t* grp, float d0, int64_t M, int64_t C, const int8_t* q,
                      float x_step, const int32_t* mu, const int32_t* sigma, const int32_t* sign_sum,
                      const float* gamma_q, int64_t dev_max, float* dx, float* dgamma, float* dbeta)
{
    if (!qg || !grp || !q || !mu || !sigma || !sign_sum || !gamma_q || !dx || !dgamma || !dbeta || M < 1 || C < 0)
        return SQO_ERR_ARG;
    for (int64_t c = 0; c < C; ++c) {
        int64_t G1 = 0, G2 = 0;
        for (int64_t m = 0; m < M; ++m) {
            G1 += qg[m * C + c];
            G2 += (int64_t)qg[m * C + c] * ((int64_t)q[m * C + c] - mu[c]);
        }
        const double delta = (double)(d0 * pow2f(-(int)grp[c]));
        const double db = delta * (double)G1;
        dbeta[c] = (float)db;
        float a = 0.0f, b = 0.0f, e = 0.0f;
        if (dev_max == 0) {
            dgamma[c] = 0.0f;
        } else {
            const double rho = (127.0 * (double)M) / ((double)dev_max * (double)sigma[c]);
            const double lambda = ((double)gamma_q[c] * rho) / (double)x_step;
            const double dg = (delta * (double)G2) * rho;
            const double D = dg / (double)M;
            const double gbar = db / (double)M;
            const double sbar = (double)sign_sum[c] / (double)M;
            dgamma[c] = (float)dg;
            a = (float)(lambda * delta);
            b = (float)(-(lambda * D));
            e = (float)(lambda * (D * sbar - gbar));
        }
        for (int64_t m = 0; m < M; ++m) {
            int32_t d = (int32_t)q[m * C + c] - mu[c];
            float s = (float)((d > 0) - (d < 0));
            dx[m * C + c] = (a * (float)qg[m * C + c] + b * s) + e;
        }
    }
    return SQO_OK;
}

/* ---------------------------------------------------------------------------
 * Weight gradient of a stride-1 convolution (R14), written from the
 * definition: with the forward conv Y[n, oh, ow, co] =
 * sum_{r, s, ci} X[n, oh + r - PH, ow + s - PW, ci] W[co, r, s, ci] (zero
 * outside the input), the gradient of <dY, Y> with respect to W is
 *   B[co, (r KW + s) C_in + ci] = sum_{n, oh, ow} q[n, oh, ow, co] x[n, oh + r - PH, ow + s - PW, ci],
 * i.e. the wgrad of the im2col'd layer (Fig. "MMs", third GEMM) without the
 * im2col.  q [N Ho Wo, C_out] gradient codes, x [N H W, C_in] input codes,
 * int64 accumulation, int32 result [C_out, KH KW C_in].
 * ------------------------------------------------------------------------- */
int sqo_conv_wgrad(const int8_t* q, int64_t N, int64_t H, int64_t W, int64_t C_out, const int8_t* x,
                   int64_t C_in, int KH, int KW, int PH, int PW, int32_t* B)
{
    if (!q || !x || !B || N < 0 || H < 1 || W < 1 || C_out < 0 || C_in < 0 || KH < 1 || KW < 1 || PH < 0 ||
        PW < 0)
        return SQO_ERR_ARG;
    int64_t Ho = H + 2 * (int64_t)PH - KH + 1, Wo = W + 2 * (int64_t)PW - KW + 1;
    if (Ho < 1 || Wo < 1) return SQO_ERR_ARG;
    int64_t cols = (int64_t)KH * KW * C_in;
    int err = SQO_OK;
#pragma omp parallel for num_threads(g_threads) collapse(4) schedule(dynamic, 1)
    for (int64_t co = 0; co < C_out; ++co)
        for (int r = 0; r < KH; ++r)
            for (int s = 0; s < KW; ++s)
                for (int64_t ci = 0; ci < C_in; ++ci) {
                    int64_t acc = 0;
                    for (int64_t n = 0; n < N; ++n)
                        for (int64_t oh = 0; oh < Ho; ++oh) {
                            int64_t ih = oh + r - PH;
                            if (ih < 0 || ih >= H) continue;
                            for (int64_t ow = 0; ow < Wo; ++ow) {
                                int64_t iw = ow + s - PW;
                                if (iw < 0 || iw >= W) continue;
                                acc += (int64_t)q[((n * Ho + oh) * Wo + ow) * C_out + co] *
                                       (int64_t)x[((n * H + ih) * W + iw) * C_in + ci];
                            }
                        }
                    if (acc > INT32_MAX || acc < INT32_MIN) {
#pragma omp atomic write
                        err = SQO_ERR_RANGE;
                    }
                    B[co * cols + ((int64_t)r * KW + s) * C_in + ci] = (int32_t)acc;
                }
    return err;
}
