// Fully-quantized L1 batch normalization (L1BNQ), Sec. 4 (Fig. l1bnq) and
// App. C: forward and backward over 8-bit input codes [M, C] (M = N*H*W rows,
// channels contiguous).
//
// Every statistic is an integer sum over a channel's column, so the kernels
// are column reductions plus one elementwise pass:
//   forward   S_c = sum q                 -> m_c (mean code)
//             A_c = sum |q - m_c|, P_c = sum sgn(q - m_c)
//                                         -> k_c (8-bit sigma code), gamma^q,
//                                            beta^q, kappa_c
//             y = fl(fl(kappa_c (q - m_c)) + beta^q_c)
//   backward  (ShiftQuant codes qg of dy, by the quantizer kernels)
//             G1_c = sum qg, G2_c = sum qg (q - m_c)
//                                         -> dgamma, dbeta, a_c, b_c, e_c
//             dx = fl(fl(fl(a_c qg) + fl(b_c sgn(q - m_c))) + e_c)
// Per-channel constants are evaluated in binary64 and rounded once to
// binary32; the library is built without FMA contraction, so the operation
// order written here is the order executed.
//
// Work split: a thread owns 16 channels of a row (one 16-byte code load);
// 256 / (C / 16) rows are in flight per block and each block takes a
// contiguous range of rows, so every load is a coalesced row segment.  A
// block reduces its rows in LDS and writes one partial per channel; a second
// kernel (one wave per channel) adds the partials.  Block partials are int32:
// with M <= 2^24 and at most 512 row blocks a block holds at most 32768 rows,
// and |qg (q - m)| <= 127 * 254.

#include <algorithm>

#include "sq_internal.h"

namespace sq {

namespace {

constexpr int kBnThreads = 256;
constexpr int kBnChunk = 16;                 // channels per thread (one 16-byte load)
constexpr int kBnWaves = 16;                 // waves of a channel-reduction block

struct BnGeom {
    int64_t chunks;   // ceil(C / 16)
    int cis;          // chunks per block column (<= 256)
    int lanes;        // rows in flight per block
    int64_t slabs;    // block columns (gridDim.y)
    int64_t nb;       // row blocks (gridDim.x)
    int64_t rpb;      // rows per block
};

BnGeom bn_geom(int64_t M, int64_t C, int64_t max_blocks, int64_t min_rows) {
    BnGeom g{};
    g.chunks = (C + kBnChunk - 1) / kBnChunk;
    g.cis = (int)std::min<int64_t>(g.chunks, kBnThreads);
    g.lanes = kBnThreads / g.cis;
    g.slabs = (g.chunks + g.cis - 1) / g.cis;
    g.nb = std::max<int64_t>(1, std::min<int64_t>(max_blocks, (M + min_rows - 1) / min_rows));
    g.rpb = (M + g.nb - 1) / g.nb;
    g.nb = (M + g.rpb - 1) / g.rpb;   // no empty block
    return g;
}

constexpr int64_t kSumBlocks = 512, kSumMinRows = 64;
constexpr int64_t kApplyBlocks = 1024, kApplyMinRows = 64;

BnGeom sum_geom(int64_t M, int64_t C) { return bn_geom(M, C, kSumBlocks, kSumMinRows); }

__device__ __forceinline__ void unpack16(const int4 v, int (&out)[16]) {
    const uint32_t w[4] = {(uint32_t)v.x, (uint32_t)v.y, (uint32_t)v.z, (uint32_t)v.w};
#pragma unroll
    for (int i = 0; i < 16; ++i) out[i] = (int)(int8_t)(w[i >> 2] >> (8 * (i & 3)));
}

__device__ __forceinline__ int sgn(int d) { return (d > 0) - (d < 0); }

// round_half_even(num / den), den > 0
__device__ __forceinline__ int64_t div_round_even(int64_t num, int64_t den) {
    int64_t q = num / den, r = num % den;
    if (r < 0) {
        q -= 1;
        r += den;
    }
    if (2 * r > den || (2 * r == den && (q & 1))) q += 1;
    return q;
}

// Block-level sum of one per-thread accumulator array over the lanes that
// share a chunk; writes part[c] for the block's channels.
__device__ __forceinline__ void block_colsum(int32_t* red, const int32_t (&acc)[16], bool active, int lane, int cl,
                                             const BnGeom& g, int64_t C, int32_t* __restrict__ part) {
    const int width = g.cis * kBnChunk;
    __syncthreads();
    if (active) {
#pragma unroll
        for (int i = 0; i < 16; ++i) red[lane * width + cl * kBnChunk + i] = acc[i];
    }
    __syncthreads();
    // every thread adds a strided subset of the lanes of one channel; the
    // subsets' sums go through LDS once more (width <= 256 channels here:
    // wider block columns have one lane, nothing to add)
    const int64_t cbase = (int64_t)blockIdx.y * width;
    if (g.lanes == 1) {
        for (int k = threadIdx.x; k < width; k += kBnThreads)
            if (cbase + k < C) part[(int64_t)blockIdx.x * C + cbase + k] = red[k];
        return;
    }
    const int J = kBnThreads / width, k = threadIdx.x % width, j = threadIdx.x / width;
    int32_t sub = 0;
    if (j < J)
        for (int l = j; l < g.lanes; l += J) sub += red[l * width + k];
    __syncthreads();
    if (j < J) red[j * width + k] = sub;
    __syncthreads();
    if (threadIdx.x < width && cbase + threadIdx.x < C) {
        int32_t s = 0;
        for (int i = 0; i < J; ++i) s += red[i * width + threadIdx.x];
        part[(int64_t)blockIdx.x * C + cbase + threadIdx.x] = s;
    }
}

// OP 0: S = sum q.  OP 1: A = sum |q - m|, P = sum sgn(q - m).
// OP 2: G1 = sum qg, G2 = sum qg (q - m)  (a = qg codes, x = input codes).
// part: [2][nb][C] int32.
template <int OP>
__global__ __launch_bounds__(kBnThreads) void k_bn_colsum(const int8_t* __restrict__ a, int64_t lda,
                                                          const int8_t* __restrict__ x, int64_t ldx,
                                                          const sq_l1bn_channel* __restrict__ ch, int64_t M,
                                                          int64_t C, BnGeom g, int32_t* __restrict__ part) {
    __shared__ int32_t red[kBnThreads * kBnChunk];
    const int tid = threadIdx.x, cl = tid % g.cis, lane = tid / g.cis;
    const int64_t chunk = (int64_t)blockIdx.y * g.cis + cl, c0 = chunk * kBnChunk;
    const bool active = lane < g.lanes && chunk < g.chunks;
    const int64_t r0 = (int64_t)blockIdx.x * g.rpb, r1 = std::min<int64_t>(M, r0 + g.rpb);
    int32_t s0[16], s1[16];
    int mu[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
        s0[i] = 0;
        s1[i] = 0;
        // clamped index, select after the load (no branch per channel)
        mu[i] = OP >= 1 ? ch[std::min<int64_t>(c0 + i, C - 1)].mu : 0;
    }
    if (active) {
        constexpr int U = 4;   // rows in flight per thread
        int64_t m = r0 + lane;
        for (; m + (U - 1) * (int64_t)g.lanes < r1; m += U * (int64_t)g.lanes) {
            int4 va[U], vx[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int64_t mm = m + u * (int64_t)g.lanes;
                va[u] = *reinterpret_cast<const int4*>(a + mm * lda + c0);
                if (OP == 2) vx[u] = *reinterpret_cast<const int4*>(x + mm * ldx + c0);
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                int qa[16], qx[16];
                unpack16(va[u], qa);
                if (OP == 2) unpack16(vx[u], qx);
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    if (OP == 0) {
                        s0[i] += qa[i];
                    } else if (OP == 1) {
                        const int d = qa[i] - mu[i];
                        s0[i] += d < 0 ? -d : d;
                        s1[i] += sgn(d);
                    } else {
                        s0[i] += qa[i];
                        s1[i] += qa[i] * (qx[i] - mu[i]);
                    }
                }
            }
        }
        for (; m < r1; m += g.lanes) {
            int qa[16], qx[16];
            unpack16(*reinterpret_cast<const int4*>(a + m * lda + c0), qa);
            if (OP == 2) unpack16(*reinterpret_cast<const int4*>(x + m * ldx + c0), qx);
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                if (OP == 0) {
                    s0[i] += qa[i];
                } else if (OP == 1) {
                    const int d = qa[i] - mu[i];
                    s0[i] += d < 0 ? -d : d;
                    s1[i] += sgn(d);
                } else {
                    s0[i] += qa[i];
                    s1[i] += qa[i] * (qx[i] - mu[i]);
                }
            }
        }
    }
    block_colsum(red, s0, active, lane, cl, g, C, part);
    if (OP >= 1) block_colsum(red, s1, active, lane, cl, g, C, part + g.nb * C);
}

// Per-channel totals of the block partials: a block of 16 waves takes 64
// consecutive channels (one per lane, so every load is a coalesced 256-byte
// row segment of the partials), the waves split the partial rows, and LDS
// adds the 16 wave sums.
//   OP 0: mean code.  OP 1: deviation and sign sums.
//   OP 2: backward constants (a, b, e), dgamma, dbeta.
template <int OP>
__global__ __launch_bounds__(64 * kBnWaves) void k_bn_chan(const int32_t* __restrict__ part, int64_t nb, int64_t M,
                                                           int64_t C, sq_l1bn_channel* __restrict__ ch,
                                                           const sq_l1bn_layer* __restrict__ layer,
                                                           const uint8_t* __restrict__ group,
                                                           const sq_scale* __restrict__ gscale,
                                                           float* __restrict__ coef, float* __restrict__ dgamma,
                                                           float* __restrict__ dbeta) {
    __shared__ int64_t sh0[kBnWaves][64], sh1[kBnWaves][64];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int64_t c = (int64_t)blockIdx.x * 64 + lane;
    const int64_t cc = std::min<int64_t>(c, C - 1);
    constexpr int U = 8;
    int64_t t0 = 0, t1 = 0;
    for (int64_t b0 = w; b0 < nb; b0 += (int64_t)kBnWaves * U) {
        int32_t v0[U], v1[U];
        // clamped row, select after the load: the loads issue back to back
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t b = std::min<int64_t>(b0 + (int64_t)kBnWaves * u, nb - 1);
            v0[u] = part[b * C + cc];
            v1[u] = OP >= 1 ? part[(nb + b) * C + cc] : 0;
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const bool in = b0 + (int64_t)kBnWaves * u < nb;
            t0 += in ? v0[u] : 0;
            t1 += in ? v1[u] : 0;
        }
    }
    sh0[w][lane] = t0;
    sh1[w][lane] = t1;
    __syncthreads();
    if (w != 0 || c >= C) return;
    t0 = t1 = 0;
#pragma unroll
    for (int i = 0; i < kBnWaves; ++i) {
        t0 += sh0[i][lane];
        t1 += sh1[i][lane];
    }
    if (OP == 0) {
        sq_l1bn_channel v{};
        v.mu = (int32_t)div_round_even(t0, M);
        ch[c] = v;
    } else if (OP == 1) {
        ch[c].dev_sum = t0;
        ch[c].sign_sum = (int32_t)t1;
    } else {
        const sq_l1bn_channel cv = ch[c];
        const sq_l1bn_layer L = *layer;
        const double delta = (double)__fmul_rn(gscale->step, pow2f(-(int)group[c]));
        const double db = delta * (double)t0;
        dbeta[c] = (float)db;
        float ca = 0.0f, cb = 0.0f, ce = 0.0f;
        if (L.dev_max == 0) {
            dgamma[c] = 0.0f;
        } else {
            const double rho = (127.0 * (double)M) / ((double)L.dev_max * (double)cv.sigma);
            const double lambda = ((double)cv.gamma * rho) / (double)L.x_step;
            const double dg = (delta * (double)t1) * rho;
            const double D = dg / (double)M;
            const double gbar = db / (double)M;
            const double sbar = (double)cv.sign_sum / (double)M;
            dgamma[c] = (float)dg;
            ca = (float)(lambda * delta);
            cb = (float)(-(lambda * D));
            ce = (float)(lambda * (D * sbar - gbar));
        }
        reinterpret_cast<float4*>(coef)[c] = make_float4(ca, cb, ce, 0.0f);
    }
}

constexpr int kParThreads = 1024;

__device__ __forceinline__ uint32_t abs_bits(float v) { return __float_as_uint(v) & 0x7FFFFFFFu; }

// 8-bit per-tensor scale of a parameter vector (the quantizer of W and X).
__device__ __forceinline__ sq_scale param_scale(uint32_t amax) {
    sq_scale s{};
    const float a = __uint_as_float(amax);
    s.r_max = a;
    s.flags = amax >= 0x7F800000u ? SQ_FLAG_NONFINITE : (a < pow2f(-96) ? SQ_FLAG_ZERO : 0u);
    if (!s.flags) {
        s.inv = 127.0f / a;
        s.step = a / 127.0f;
    }
    return s;
}

__device__ __forceinline__ float param_value(float v, const sq_scale& s) {
    if (s.flags) return 0.0f;
    // the code is an integer: a negative value that rounds to 0 gives +0
    const int code = (int)fminf(fmaxf(rintf(__fmul_rn(v, s.inv)), -127.0f), 127.0f);
    return __fmul_rn(s.step, (float)code);
}

// One block: A_max, the parameter scales, then every channel's sigma code,
// gamma^q, beta^q and kappa.
__global__ __launch_bounds__(kParThreads) void k_bn_params(sq_l1bn_channel* __restrict__ ch, int64_t M, int64_t C,
                                                           const float* __restrict__ gamma,
                                                           const float* __restrict__ beta,
                                                           const sq_scale* __restrict__ xs,
                                                           sq_l1bn_layer* __restrict__ layer) {
    __shared__ int64_t sh_a[kParThreads / 64];
    __shared__ uint32_t sh_g[kParThreads / 64], sh_b[kParThreads / 64];
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    int64_t amax = 0;
    uint32_t gmax = 0u, bmax = 0u;
    for (int64_t c = tid; c < C; c += kParThreads) {
        amax = std::max<int64_t>(amax, ch[c].dev_sum);
        gmax = std::max(gmax, abs_bits(gamma[c]));
        bmax = std::max(bmax, abs_bits(beta[c]));
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        amax = std::max<int64_t>(amax, __shfl_xor(amax, o, 64));
        gmax = std::max(gmax, (uint32_t)__shfl_xor((int)gmax, o, 64));
        bmax = std::max(bmax, (uint32_t)__shfl_xor((int)bmax, o, 64));
    }
    if (lane == 0) {
        sh_a[w] = amax;
        sh_g[w] = gmax;
        sh_b[w] = bmax;
    }
    __syncthreads();
    amax = 0;
    gmax = bmax = 0u;
    for (int i = 0; i < kParThreads / 64; ++i) {
        amax = std::max<int64_t>(amax, sh_a[i]);
        gmax = std::max(gmax, sh_g[i]);
        bmax = std::max(bmax, sh_b[i]);
    }
    const sq_scale gs = param_scale(gmax), bs = param_scale(bmax);
    for (int64_t c = tid; c < C; c += kParThreads) {
        sq_l1bn_channel v = ch[c];
        v.gamma = param_value(gamma[c], gs);
        v.beta = param_value(beta[c], bs);
        if (amax == 0) {
            v.sigma = 0;
            v.kappa = 0.0f;
        } else {
            const int64_t k = std::max<int64_t>(1, div_round_even(127 * v.dev_sum, amax));
            v.sigma = (int32_t)k;
            const double num = (double)v.gamma * (127.0 * (double)M);
            v.kappa = (float)(num / ((double)amax * (double)k));
        }
        ch[c] = v;
    }
    if (tid == 0) {
        sq_l1bn_layer L{};
        L.rows = M;
        L.dev_max = amax;
        L.x_step = xs->step;
        L.flags = amax == 0 ? SQ_FLAG_ZERO : 0u;
        L.gamma_scale = gs;
        L.beta_scale = bs;
        *layer = L;
    }
}

// Elementwise pass.  Forward (BWD = false): y = fl(fl(kappa (q - m)) + beta),
// a = input codes.  Backward: dx = fl(fl(fl(a qg) + fl(b sgn(q - m))) + e),
// a = gradient codes, x = input codes; with `ranges`, each block also writes
// the channel maxima of |dx| over its rows (bit patterns) to ranges[block, c].
// A thread owns one channel quad of a row (a 4-byte code load, one float4
// store), so a wave's loads and stores cover contiguous row segments.
struct QuadGeom {
    int64_t quads;    // ceil(C / 4)
    int qis;          // quads per block column (<= 256)
    int lanes;        // rows in flight per block
    int64_t slabs, nb, rpb;
};

QuadGeom quad_geom(int64_t M, int64_t C) {
    QuadGeom g{};
    g.quads = (C + 3) / 4;
    g.qis = (int)std::min<int64_t>(g.quads, kBnThreads);
    g.lanes = kBnThreads / g.qis;
    g.slabs = (g.quads + g.qis - 1) / g.qis;
    g.nb = std::max<int64_t>(1, std::min<int64_t>(kApplyBlocks, (M + kApplyMinRows - 1) / kApplyMinRows));
    g.rpb = (M + g.nb - 1) / g.nb;
    g.nb = (M + g.rpb - 1) / g.rpb;
    return g;
}

__device__ __forceinline__ void unpack4(uint32_t w, int (&out)[4]) {
#pragma unroll
    for (int i = 0; i < 4; ++i) out[i] = (int)(int8_t)(w >> (8 * i));
}

template <bool BWD>
__global__ __launch_bounds__(kBnThreads) void k_bn_apply(const int8_t* __restrict__ a, int64_t lda,
                                                         const int8_t* __restrict__ x, int64_t ldx,
                                                         const sq_l1bn_channel* __restrict__ ch,
                                                         const float* __restrict__ coef, int64_t M, int64_t C,
                                                         QuadGeom g, float* __restrict__ out, int64_t ld_out,
                                                         bool vec_out, uint32_t* __restrict__ ranges) {
    __shared__ uint32_t red[BWD ? kBnThreads * 4 : 1];
    const int tid = threadIdx.x, cl = tid % g.qis, lane = tid / g.qis;
    const int64_t quad = (int64_t)blockIdx.y * g.qis + cl, c0 = quad * 4;
    const bool active = lane < g.lanes && quad < g.quads;
    const int64_t r0 = (int64_t)blockIdx.x * g.rpb, r1 = std::min<int64_t>(M, r0 + g.rpb);
    const bool full = c0 + 4 <= C && vec_out;
    int mu[4];
    float k0[4], k1[4], k2[4];
    uint32_t rmax[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        // clamped index, select after the load (no branch per channel)
        const int64_t cc = std::min<int64_t>(c0 + i, C - 1);
        const bool ok = c0 + i < C;
        const sq_l1bn_channel v = ch[cc];
        mu[i] = v.mu;
        if (BWD) {
            const float4 k = reinterpret_cast<const float4*>(coef)[cc];
            k0[i] = ok ? k.x : 0.0f;
            k1[i] = ok ? k.y : 0.0f;
            k2[i] = ok ? k.z : 0.0f;
        } else {
            k0[i] = ok ? v.kappa : 0.0f;
            k1[i] = ok ? v.beta : 0.0f;
            k2[i] = 0.0f;
        }
        rmax[i] = 0u;
    }
    auto row_out = [&](int64_t m, uint32_t wa, uint32_t wx) {
        int qa[4], qx[4];
        unpack4(wa, qa);
        if (BWD) unpack4(wx, qx);
        float v[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            if (BWD) {
                const float s = (float)sgn(qx[i] - mu[i]);
                v[i] = __fadd_rn(__fadd_rn(__fmul_rn(k0[i], (float)qa[i]), __fmul_rn(k1[i], s)), k2[i]);
                if (c0 + i < C) rmax[i] = std::max(rmax[i], abs_bits(v[i]));
            } else {
                v[i] = __fadd_rn(__fmul_rn(k0[i], (float)(qa[i] - mu[i])), k1[i]);
            }
        }
        float* row = out + m * ld_out + c0;
        if (full) {
            *reinterpret_cast<float4*>(row) = make_float4(v[0], v[1], v[2], v[3]);
        } else {
#pragma unroll
            for (int i = 0; i < 4; ++i)
                if (c0 + i < C) row[i] = v[i];
        }
    };
    if (active) {
        constexpr int U = 8;   // rows in flight per thread
        int64_t m = r0 + lane;
        for (; m + (U - 1) * (int64_t)g.lanes < r1; m += U * (int64_t)g.lanes) {
            uint32_t wa[U], wx[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int64_t mm = m + u * (int64_t)g.lanes;
                wa[u] = *reinterpret_cast<const uint32_t*>(a + mm * lda + c0);
                wx[u] = BWD ? *reinterpret_cast<const uint32_t*>(x + mm * ldx + c0) : 0u;
            }
#pragma unroll
            for (int u = 0; u < U; ++u) row_out(m + u * (int64_t)g.lanes, wa[u], wx[u]);
        }
        for (; m < r1; m += g.lanes)
            row_out(m, *reinterpret_cast<const uint32_t*>(a + m * lda + c0),
                    BWD ? *reinterpret_cast<const uint32_t*>(x + m * ldx + c0) : 0u);
    }
    if (BWD && ranges) {
        const int width = g.qis * 4;
        __syncthreads();
        if (active) {
#pragma unroll
            for (int i = 0; i < 4; ++i) red[lane * width + cl * 4 + i] = rmax[i];
        }
        __syncthreads();
        const int64_t cbase = (int64_t)blockIdx.y * width;
        for (int k = tid; k < width; k += kBnThreads) {
            const int64_t c = cbase + k;
            if (c >= C) continue;
            uint32_t mx = 0u;
            for (int l = 0; l < g.lanes; ++l) mx = std::max(mx, red[l * width + k]);
            ranges[(int64_t)blockIdx.x * C + c] = mx;
        }
    }
}

}  // namespace

int64_t l1bn_range_slabs(int64_t M, int64_t C) { return M > 0 && C > 0 ? quad_geom(M, C).nb : 0; }

int64_t l1bn_part_words(int64_t M, int64_t C) { return 2 * sum_geom(M, C).nb * C; }

hipError_t launch_l1bn_forward(const int8_t* xq, int64_t M, int64_t C, int64_t ld_x, const sq_scale* xs,
                               const float* gamma, const float* beta, float* y, int64_t ld_y, sq_l1bn_channel* ch,
                               sq_l1bn_layer* layer, int32_t* part, hipStream_t s) {
    if (C <= 0) return hipSuccess;
    const BnGeom gs = sum_geom(M, C);
    const QuadGeom ga = quad_geom(M, C);
    const dim3 sum_grid((unsigned)gs.nb, (unsigned)gs.slabs), chan_grid((unsigned)((C + 63) / 64));
    hipLaunchKernelGGL(k_bn_colsum<0>, sum_grid, dim3(kBnThreads), 0, s, xq, ld_x, nullptr, 0, ch, M, C, gs, part);
    hipLaunchKernelGGL(k_bn_chan<0>, chan_grid, dim3(64 * kBnWaves), 0, s, part, gs.nb, M, C, ch, nullptr, nullptr,
                       nullptr, nullptr, nullptr, nullptr);
    hipLaunchKernelGGL(k_bn_colsum<1>, sum_grid, dim3(kBnThreads), 0, s, xq, ld_x, nullptr, 0, ch, M, C, gs, part);
    hipLaunchKernelGGL(k_bn_chan<1>, chan_grid, dim3(64 * kBnWaves), 0, s, part, gs.nb, M, C, ch, nullptr, nullptr,
                       nullptr, nullptr, nullptr, nullptr);
    hipLaunchKernelGGL(k_bn_params, dim3(1), dim3(kParThreads), 0, s, ch, M, C, gamma, beta, xs, layer);
    const bool vec = (ld_y % 4 == 0) && (reinterpret_cast<uintptr_t>(y) % 16 == 0);
    hipLaunchKernelGGL(k_bn_apply<false>, dim3((unsigned)ga.nb, (unsigned)ga.slabs), dim3(kBnThreads), 0, s, xq, ld_x,
                       nullptr, 0, ch, nullptr, M, C, ga, y, ld_y, vec, nullptr);
    return hipGetLastError();
}

hipError_t launch_l1bn_backward(const int8_t* qg, int64_t ldg, const int8_t* xq, int64_t ld_x, int64_t M, int64_t C,
                                const sq_l1bn_channel* ch, const sq_l1bn_layer* layer, const uint8_t* group,
                                const sq_scale* gscale, float* dx, int64_t ld_dx, float* dgamma, float* dbeta,
                                uint32_t* ranges, int32_t* part, float* coef, hipStream_t s) {
    if (C <= 0) return hipSuccess;
    const BnGeom gs = sum_geom(M, C);
    const QuadGeom ga = quad_geom(M, C);
    hipLaunchKernelGGL(k_bn_colsum<2>, dim3((unsigned)gs.nb, (unsigned)gs.slabs), dim3(kBnThreads), 0, s, qg, ldg, xq,
                       ld_x, ch, M, C, gs, part);
    hipLaunchKernelGGL(k_bn_chan<2>, dim3((unsigned)((C + 63) / 64)), dim3(64 * kBnWaves), 0, s, part,
                       gs.nb, M, C, const_cast<sq_l1bn_channel*>(ch), layer, group, gscale, coef, dgamma, dbeta);
    const bool vec = (ld_dx % 4 == 0) && (reinterpret_cast<uintptr_t>(dx) % 16 == 0);
    hipLaunchKernelGGL(k_bn_apply<true>, dim3((unsigned)ga.nb, (unsigned)ga.slabs), dim3(kBnThreads), 0, s, qg, ldg,
                       xq, ld_x, ch, coef, M, C, ga, dx, ld_dx, vec, ranges);
    return hipGetLastError();
}

}  // namespace sq
