// ShiftQuant quantizer kernels for gfx950.
//
// Stream-ordered passes (the tensor range r_max is global, so the gradient is
// read twice):
//   k_colmax         per-channel abs-max r_c (Sec. 3.1) as unsigned bit
//                    patterns: coalesced float4 row loads, one maximum per
//                    channel per row slab (plain stores, no atomics)
//   k_colmax_reduce  (many channels only) combines the slabs per channel and
//                    leaves one maximum per block
//   k_finalize       one block: r_max, group ids (power-of-two thresholds,
//                    Sec. 3.1), scales, flags, and the fold layout for dgrad
//   k_quantize       scale, round (ties-to-even or Philox stochastic rounding,
//                    App. B Eq. "sq"), clamp; writes the shift-folded dgrad
//                    operand row-major and the codes transposed
//
// All fp32 arithmetic is IEEE with round-to-nearest-even and no contraction
// (the library is built with -ffp-contract=off and the products below use the
// _rn intrinsics), so the codes are a bit-exact function of the inputs.
#include <algorithm>

#include "sq_internal.h"

namespace sq {

namespace {

// ---------------------------------------------------------------------------
// Philox4x32-10 (Salmon et al., SC'11): counter-based uniform bits for
// stochastic rounding.  Written independently of any other implementation.
// ---------------------------------------------------------------------------
struct U4 { uint32_t x, y, z, w; };

__device__ __forceinline__ U4 philox4x32_10(U4 c, uint32_t k0, uint32_t k1) {
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        const uint64_t p0 = (uint64_t)0xD2511F53u * c.x;   // one 32x32->64 product each
        const uint64_t p1 = (uint64_t)0xCD9E8D57u * c.z;
        c = U4{(uint32_t)(p1 >> 32) ^ c.y ^ k0, (uint32_t)p1, (uint32_t)(p0 >> 32) ^ c.w ^ k1, (uint32_t)p0};
        k0 += 0x9E3779B9u;
        k1 += 0xBB67AE85u;
    }
    return c;
}

__device__ __forceinline__ U4 philox_block(uint64_t blk, const QuantCfg& cfg) {
    return philox4x32_10(U4{(uint32_t)blk, (uint32_t)(blk >> 32), (uint32_t)cfg.offset,
                            (uint32_t)(cfg.offset >> 32)},
                         (uint32_t)cfg.seed, (uint32_t)(cfg.seed >> 32));
}

__device__ __forceinline__ uint32_t pick(const U4& w, int i) {
    return i == 0 ? w.x : (i == 1 ? w.y : (i == 2 ? w.z : w.w));
}

// The 24-bit uniform of the element with logical index idx = m * C + c.
__device__ __forceinline__ uint32_t sr_uniform24(uint64_t idx, const QuantCfg& cfg) {
    return pick(philox_block(idx >> 2, cfg), (int)(idx & 3u)) >> 8;
}

// One code: v = fl(x * s); round; clamp to [-Q, Q].  u24 is the 24-bit
// uniform used only by stochastic rounding.
template <bool SR>
__device__ __forceinline__ int quant_one(float x, float s, float Qf, uint32_t u24) {
    const float v = __fmul_rn(x, s);
    float qf;
    if (SR) {
        const float l = floorf(v);
        const float f = __fsub_rn(v, l);
        qf = ((float)u24 < __fmul_rn(f, 16777216.0f)) ? __fadd_rn(l, 1.0f) : l;
    } else {
        qf = rintf(v);
    }
    qf = fminf(fmaxf(qf, -Qf), Qf);
    return (int)qf;
}

__device__ __forceinline__ uint32_t absbits(float x) { return __float_as_uint(x) & 0x7FFFFFFFu; }

// ---------------------------------------------------------------------------
// Per-channel abs-max, first level.  The rows are cut into slabs; block
// (chunk, slab) reduces its slab for the chunk's channels and stores the
// slab maxima to partial[slab * C + c] (plain stores: same-address atomics
// from many blocks serialise, so the slabs are combined in a second step).
// Thread (rl, tc) covers VEC channels starting at (chunk * tpr + tc) * VEC and
// rows rl, rl + kColThreads / tpr, ... of the slab, 8 loads in flight.
// ---------------------------------------------------------------------------
constexpr int kColThreads = 512;

template <int VEC>
__global__ __launch_bounds__(kColThreads) void k_colmax(const float* __restrict__ x, int64_t M, int64_t C,
                                                        int64_t ld, int tpr, int64_t rows_per_slab,
                                                        uint32_t* __restrict__ partial) {
    __shared__ uint32_t red[kColThreads * VEC];
    const int tid = threadIdx.x;
    const int nrl = kColThreads / tpr;
    const int rl = tid / tpr, tc = tid % tpr;
    const int64_t c0 = ((int64_t)blockIdx.x * tpr + tc) * VEC;
    const int64_t m_begin = (int64_t)blockIdx.y * rows_per_slab;
    const int64_t m_end = min(M, m_begin + rows_per_slab);
    uint32_t best[VEC];
#pragma unroll
    for (int j = 0; j < VEC; ++j) best[j] = 0u;

    if (c0 < C) {
        int64_t m = m_begin + rl;
        if constexpr (VEC == 4) {
            if (c0 + 4 <= C) {
                for (; m + 7 * (int64_t)nrl < m_end; m += 8 * (int64_t)nrl) {
                    float4 v[8];
#pragma unroll
                    for (int u = 0; u < 8; ++u)
                        v[u] = *reinterpret_cast<const float4*>(x + (m + u * (int64_t)nrl) * ld + c0);
#pragma unroll
                    for (int u = 0; u < 8; ++u) {
                        best[0] = max(best[0], absbits(v[u].x));
                        best[1] = max(best[1], absbits(v[u].y));
                        best[2] = max(best[2], absbits(v[u].z));
                        best[3] = max(best[3], absbits(v[u].w));
                    }
                }
                for (; m < m_end; m += nrl) {
                    const float4 v = *reinterpret_cast<const float4*>(x + m * ld + c0);
                    best[0] = max(best[0], absbits(v.x));
                    best[1] = max(best[1], absbits(v.y));
                    best[2] = max(best[2], absbits(v.z));
                    best[3] = max(best[3], absbits(v.w));
                }
            }
        }
        for (; m < m_end; m += nrl) {   // scalar path (and the ragged last vector)
#pragma unroll
            for (int j = 0; j < VEC; ++j)
                if (c0 + j < C) best[j] = max(best[j], absbits(x[m * ld + c0 + j]));
        }
    }
#pragma unroll
    for (int j = 0; j < VEC; ++j) red[tid * VEC + j] = best[j];
    __syncthreads();
    if (rl == 0 && c0 < C) {
        for (int r = 1; r < nrl; ++r)
#pragma unroll
            for (int j = 0; j < VEC; ++j) best[j] = max(best[j], red[(r * tpr + tc) * VEC + j]);
        uint32_t* dst = partial + (int64_t)blockIdx.y * C + c0;
#pragma unroll
        for (int j = 0; j < VEC; ++j)
            if (c0 + j < C) dst[j] = best[j];
    }
}

// max over the S slab maxima of channel c (8 loads in flight per thread)
__device__ __forceinline__ uint32_t reduce_slabs(const uint32_t* __restrict__ partial, int64_t S, int64_t C,
                                                 int64_t c) {
    uint32_t a[8] = {0u, 0u, 0u, 0u, 0u, 0u, 0u, 0u};
    int64_t s = 0;
    for (; s + 8 <= S; s += 8) {
#pragma unroll
        for (int u = 0; u < 8; ++u) a[u] = max(a[u], partial[(s + u) * C + c]);
    }
    for (; s < S; ++s) a[0] = max(a[0], partial[s * C + c]);
#pragma unroll
    for (int u = 1; u < 8; ++u) a[0] = max(a[0], a[u]);
    return a[0];
}

// ---------------------------------------------------------------------------
// Block-wide helpers (any multiple of 64 threads up to 1024).
// ---------------------------------------------------------------------------
__device__ uint32_t block_max_u32(uint32_t v, uint32_t* sh) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = max(v, (uint32_t)__shfl_xor((int)v, o, 64));
    const int w = threadIdx.x >> 6, nw = blockDim.x >> 6;
    __syncthreads();
    if ((threadIdx.x & 63) == 0) sh[w] = v;
    __syncthreads();
    v = 0u;
    for (int i = 0; i < nw; ++i) v = max(v, sh[i]);
    __syncthreads();
    return v;
}

// Exclusive prefix sum of v over the block (thread order), plus the total.
__device__ int block_excl_scan(int v, int* sh, int* total) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
    int x = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(x, o, 64);
        if (lane >= o) x += y;
    }
    __syncthreads();
    if (lane == 63) sh[w] = x;
    __syncthreads();
    int base = 0, tot = 0;
    for (int i = 0; i < nw; ++i) {
        if (i < w) base += sh[i];
        tot += sh[i];
    }
    __syncthreads();
    *total = tot;
    return base + x - v;
}

// Second level for many channels: rbits[c] = max over slabs, and the block's
// maximum in bmax[blockIdx.x].
constexpr int kRedThreads = 256;

__global__ __launch_bounds__(kRedThreads) void k_colmax_reduce(const uint32_t* __restrict__ partial, int64_t S,
                                                               int64_t C, uint32_t* __restrict__ rbits,
                                                               uint32_t* __restrict__ bmax) {
    __shared__ uint32_t shu[kRedThreads / 64];
    const int64_t c = (int64_t)blockIdx.x * kRedThreads + threadIdx.x;
    uint32_t r = 0u;
    if (c < C) {
        r = reduce_slabs(partial, S, C, c);
        rbits[c] = r;
    }
    r = block_max_u32(r, shu);
    if (threadIdx.x == 0) bmax[blockIdx.x] = r;
}

// Channel ranges for fewer channels than threads: W channels x L slab lanes,
// combined through LDS.  Thread tid < C returns r_{tid}; the others 0.
constexpr int kFinThreads = 1024;

__device__ uint32_t small_channel_ranges(const uint32_t* __restrict__ partial, int64_t S, int64_t C,
                                         uint32_t* lanes) {
    const int tid = threadIdx.x;
    int W = 1;
    while (W < C) W <<= 1;
    const int L = kFinThreads / W;
    const int cl = tid % W, lane = tid / W;
    uint32_t a[8] = {0u, 0u, 0u, 0u, 0u, 0u, 0u, 0u};
    if (cl < C) {
        int64_t sl = lane;
        for (; sl + 7 * (int64_t)L < S; sl += 8 * (int64_t)L) {
#pragma unroll
            for (int u = 0; u < 8; ++u) a[u] = max(a[u], partial[(sl + u * (int64_t)L) * C + cl]);
        }
        for (; sl < S; sl += L) a[0] = max(a[0], partial[sl * C + cl]);
    }
#pragma unroll
    for (int u = 1; u < 8; ++u) a[0] = max(a[0], a[u]);
    lanes[tid] = a[0];
    __syncthreads();
    uint32_t r = 0u;
    if (tid < C)
        for (int l = 0; l < L; ++l) r = max(r, lanes[l * W + tid]);
    __syncthreads();
    return r;
}

// Group of a channel: the smallest j < N_G - 1 with r_c * 2^(j+1) > r_max,
// else N_G - 1.  Products with powers of two are exact (an overflow to +Inf
// still compares correctly), so this equals the threshold test
// r_c > r_max * 2^-(j+1) of Sec. 3.1.
__device__ __forceinline__ int group_of(float r_c, float r_max, int num_groups) {
    for (int j = 0; j < num_groups - 1; ++j)
        if (__fmul_rn(r_c, pow2f(j + 1)) > r_max) return j;
    return num_groups - 1;
}

__device__ __forceinline__ int excess_of(int g, const QuantCfg& cfg) {
    const int sh = cfg.num_groups - 1 - g;
    return sh > cfg.T ? sh - cfg.T : 0;
}

__device__ __forceinline__ sq_scale make_scale(uint32_t mb, float Qf) {
    const float r_max = __uint_as_float(mb);
    uint32_t flags = 0u;
    if (mb >= 0x7F800000u) flags = SQ_FLAG_NONFINITE;
    else if (r_max < pow2f(-96)) flags = SQ_FLAG_ZERO;
    sq_scale s;
    s.r_max = r_max;
    s.inv = flags ? 0.0f : __fdiv_rn(Qf, r_max);
    s.step = flags ? 0.0f : __fdiv_rn(r_max, Qf);
    s.flags = flags;
    return s;
}

// ---------------------------------------------------------------------------
// Finalize for the gradient quantizer (one block).  With C < kFinThreads the
// slab maxima are combined here; otherwise k_colmax_reduce has written rbits
// and one maximum per block.  Thread tid owns the contiguous channels
// [tid * R, tid * R + R), R = ceil(C / kFinThreads), so each fold region's
// channel list comes out of a single block-wide scan.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kFinThreads) void k_finalize_grad(const uint32_t* __restrict__ partial, int64_t S,
                                                               int64_t C, QuantCfg cfg,
                                                               uint32_t* __restrict__ rbits,
                                                               const uint32_t* __restrict__ bmax, int64_t nb,
                                                               uint8_t* __restrict__ group,
                                                               sq_scale* __restrict__ scale,
                                                               int32_t* __restrict__ layout) {
    __shared__ uint32_t shu[16];
    __shared__ int shi[16];
    __shared__ uint32_t lanes[kFinThreads];
    const int tid = threadIdx.x;

    uint32_t mb = 0u;
    if (C < kFinThreads) {
        const uint32_t r = small_channel_ranges(partial, S, C, lanes);
        if (tid < C) rbits[tid] = r;   // read back below by the same thread
        mb = r;
    } else {
        for (int64_t i = tid; i < nb; i += kFinThreads) mb = max(mb, bmax[i]);
    }
    mb = block_max_u32(mb, shu);
    const sq_scale sc = make_scale(mb, (float)cfg.Q);
    if (tid == 0) *scale = sc;
    const float r_max = sc.r_max;
    const bool flagged = sc.flags != 0u;

    const int64_t R = (C + kFinThreads - 1) / kFinThreads;
    const int64_t c_lo = min(C, (int64_t)tid * R), c_hi = min(C, c_lo + R);
    auto group_at = [&](int64_t c) {
        return flagged ? cfg.num_groups - 1 : group_of(__uint_as_float(rbits[c]), r_max, cfg.num_groups);
    };

    int emax = 0;
    for (int64_t c = c_lo; c < c_hi; ++c) {
        const int g = group_at(c);
        group[c] = (uint8_t)g;
        emax = max(emax, excess_of(g, cfg));
    }
    const int E = (int)block_max_u32((uint32_t)emax, shu);

    // Appended regions, in the order the dgrad visits them: region r holds,
    // in ascending order, the channels whose excess exceeds j = E - 1 - r,
    // padded with -1 to a multiple of kFoldPad columns.
    int32_t* ext = layout + kLayoutHeader;
    int start = 0;
    for (int r = 0; r < E; ++r) {
        const int j = E - 1 - r;
        int cnt = 0;
        for (int64_t c = c_lo; c < c_hi; ++c) cnt += excess_of(group_at(c), cfg) > j;
        int total = 0;
        int pos = start + block_excl_scan(cnt, shi, &total);
        for (int64_t c = c_lo; c < c_hi; ++c)
            if (excess_of(group_at(c), cfg) > j) ext[pos++] = (int32_t)c;
        const int padded = (int)round_up(total, kFoldPad);
        for (int i = total + tid; i < padded; i += kFinThreads) ext[start + i] = -1;
        if (tid == 0) layout[4 + r] = start;
        start += padded;
    }
    if (tid == 0) {
        layout[0] = E;
        layout[1] = start;
        layout[2] = (int32_t)fold_ext_base(C);
        layout[3] = 0;
        for (int r = E; r < kMaxRegions; ++r) layout[4 + r] = start;
    }
}

// Finalize for per-tensor quantization (one block): the tensor's absolute
// maximum is the maximum over all slab maxima.
__global__ __launch_bounds__(kFinThreads) void k_finalize_tensor(const uint32_t* __restrict__ partial, int64_t S,
                                                                 int64_t C, int Q, const uint32_t* __restrict__ bmax,
                                                                 int64_t nb, sq_scale* __restrict__ scale) {
    __shared__ uint32_t shu[16];
    __shared__ uint32_t lanes[kFinThreads];
    uint32_t mb = 0u;
    if (C < kFinThreads) mb = small_channel_ranges(partial, S, C, lanes);
    else
        for (int64_t i = threadIdx.x; i < nb; i += kFinThreads) mb = max(mb, bmax[i]);
    mb = block_max_u32(mb, shu);
    if (threadIdx.x == 0) *scale = make_scale(mb, (float)Q);
}

// ---------------------------------------------------------------------------
// Quantize.  Thread (tr, tc4) of a block handles 16 consecutive rows x 4
// consecutive channels of a row tile: channels c0 = tile_c + 4 * tc4 and rows
// m_base = tile_m + 16 * tr.  It writes the shift-folded codes of each row as
// one 4-byte store into q_fold (a wave covers whole 128-byte lines) and the 16
// codes of each of its channels as one 16-byte store into q_t, so the
// transpose needs no LDS.  tc4n (a power of two <= 32) threads span the
// channel tile; a row tile has 16 * kBlock / tc4n rows.
// ---------------------------------------------------------------------------
constexpr int kBlock = 256;
constexpr int kQR = 16;   // rows per thread

template <int VEC, bool SR>
__global__ __launch_bounds__(kBlock) void k_quantize(const float* __restrict__ x, int64_t M, int64_t C,
                                                     int64_t ld, const uint8_t* __restrict__ group,
                                                     const sq_scale* __restrict__ scale, QuantCfg cfg, int tc4n,
                                                     int8_t* __restrict__ q_fold, int64_t ld_fold,
                                                     int8_t* __restrict__ q_t, int64_t ld_t,
                                                     const int32_t* __restrict__ layout) {
    const int tid = threadIdx.x;
    const int tc4 = tid & (tc4n - 1), tr = tid / tc4n;
    const int rows_per_tile = kQR * (kBlock / tc4n);
    const int64_t c0 = (int64_t)blockIdx.x * 4 * tc4n + 4 * tc4;
    const int64_t row_tiles = (M + rows_per_tile - 1) / rows_per_tile;

    const sq_scale sc = *scale;
    const bool zero = sc.flags != 0u;
    const float Qf = (float)cfg.Q;

    float s[4];
    int t[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int64_t c = c0 + j;
        const int g = (group && c < C) ? (int)group[c] : 0;
        s[j] = __fmul_rn(sc.inv, pow2f(g));
        t[j] = group ? min(cfg.num_groups - 1 - g, cfg.T) : 0;
    }
    const bool sr_vec = SR && ((C & 3) == 0);   // 4 channels share one Philox block

    for (int64_t rt = blockIdx.y; rt < row_tiles; rt += gridDim.y) {
        const int64_t m_base = rt * rows_per_tile + (int64_t)kQR * tr;
        if (c0 < C && m_base < M) {
            float v[kQR][4];
#pragma unroll
            for (int i = 0; i < kQR; ++i) {
                const int64_t m = m_base + i;
                v[i][0] = v[i][1] = v[i][2] = v[i][3] = 0.f;
                if (m < M) {
                    bool done = false;
                    if constexpr (VEC == 4) {
                        if (c0 + 4 <= C) {
                            const float4 f = *reinterpret_cast<const float4*>(x + m * ld + c0);
                            v[i][0] = f.x; v[i][1] = f.y; v[i][2] = f.z; v[i][3] = f.w;
                            done = true;
                        }
                    }
                    if (!done) {
#pragma unroll
                        for (int j = 0; j < 4; ++j)
                            if (c0 + j < C) v[i][j] = x[m * ld + c0 + j];
                    }
                }
            }
            uint32_t colw[4][kQR / 4];   // channel j, rows 4w .. 4w + 3 packed little-endian
#pragma unroll
            for (int j = 0; j < 4; ++j)
#pragma unroll
                for (int w = 0; w < kQR / 4; ++w) colw[j][w] = 0u;
#pragma unroll
            for (int i = 0; i < kQR; ++i) {
                const int64_t m = m_base + i;
                uint32_t u[4] = {0u, 0u, 0u, 0u};
                if (SR && m < M) {
                    if (sr_vec) {
                        const U4 w = philox_block((uint64_t)(m * C + c0) >> 2, cfg);
                        u[0] = w.x >> 8; u[1] = w.y >> 8; u[2] = w.z >> 8; u[3] = w.w >> 8;
                    } else {
#pragma unroll
                        for (int j = 0; j < 4; ++j) u[j] = sr_uniform24((uint64_t)(m * C + c0 + j), cfg);
                    }
                }
                int code[4];
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    code[j] = (zero || m >= M || c0 + j >= C) ? 0 : quant_one<SR>(v[i][j], s[j], Qf, u[j]);
                    colw[j][i / 4] |= (uint32_t)(uint8_t)code[j] << (8 * (i % 4));
                }
                if (q_fold && m < M) {
                    int8_t* dst = q_fold + m * ld_fold + c0;
                    if (c0 + 4 <= C) {
                        *reinterpret_cast<uint32_t*>(dst) = ((uint32_t)(uint8_t)(code[0] * (1 << t[0]))) |
                                                            ((uint32_t)(uint8_t)(code[1] * (1 << t[1])) << 8) |
                                                            ((uint32_t)(uint8_t)(code[2] * (1 << t[2])) << 16) |
                                                            ((uint32_t)(uint8_t)(code[3] * (1 << t[3])) << 24);
                    } else {
#pragma unroll
                        for (int j = 0; j < 4; ++j)
                            if (c0 + j < C) dst[j] = (int8_t)(code[j] * (1 << t[j]));
                    }
                }
            }
            if (q_t) {
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    if (c0 + j >= C) continue;
                    int8_t* dst = q_t + (c0 + j) * ld_t + m_base;
                    if (m_base + kQR <= M) {
                        *reinterpret_cast<uint4*>(dst) = make_uint4(colw[j][0], colw[j][1], colw[j][2], colw[j][3]);
                    } else {
                        for (int i = 0; i < (int)(M - m_base); ++i)
                            dst[i] = (int8_t)(colw[j][i / 4] >> (8 * (i % 4)));
                    }
                }
            }
        }

        // Appended fold columns (dgrad operand only), written by the blocks of
        // the first channel tile for their rows.
        if (q_fold && layout && blockIdx.x == 0) {
            const int D = layout[1];
            const int64_t base = layout[2];
            const int32_t* ext = layout + kLayoutHeader;
            const int64_t m_tile = rt * rows_per_tile;
            const int64_t n_el = (int64_t)rows_per_tile * D;
            for (int64_t idx = tid; idx < n_el; idx += kBlock) {
                const int64_t rr = idx / D, j = idx % D;
                const int64_t m = m_tile + rr;
                if (m >= M) continue;
                const int ch = ext[j];
                int val = 0;
                if (ch >= 0 && !zero) {
                    const int g = (int)group[ch];
                    const float sc_ch = __fmul_rn(sc.inv, pow2f(g));
                    const uint32_t u = SR ? sr_uniform24((uint64_t)(m * C + ch), cfg) : 0u;
                    const int tt = min(cfg.num_groups - 1 - g, cfg.T);
                    val = quant_one<SR>(x[m * ld + ch], sc_ch, Qf, u) * (1 << tt);
                }
                q_fold[m * ld_fold + base + j] = (int8_t)val;
            }
        }
    }
}

}  // namespace

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
ColmaxPlan colmax_plan(int64_t M, int64_t C, bool vec) {
    ColmaxPlan p{};
    const int VEC = vec ? 4 : 1;
    const int64_t units = (C + VEC - 1) / VEC;
    int tpr = 1;
    while (tpr < units && tpr < 64) tpr <<= 1;
    const int nrl = kColThreads / tpr;
    p.vec = VEC;
    p.tpr = tpr;
    p.chunks = std::max<int64_t>(1, (units + tpr - 1) / tpr);
    // about 1024 blocks (four per CU), each slab at least 8 row passes deep
    int64_t slabs = std::max<int64_t>(1, 1024 / p.chunks);
    const int64_t min_rows = 8 * (int64_t)nrl;
    slabs = std::min<int64_t>(slabs, std::max<int64_t>(1, (M + min_rows - 1) / min_rows));
    slabs = std::min<int64_t>(slabs, 65535);
    p.rows_per_slab = std::max<int64_t>(1, (M + slabs - 1) / slabs);
    p.slabs = M > 0 ? (M + p.rows_per_slab - 1) / p.rows_per_slab : 0;
    return p;
}

int64_t colmax_reduce_blocks(int64_t C) { return C >= kFinThreads ? (C + kRedThreads - 1) / kRedThreads : 0; }

int64_t colmax_workspace_words(int64_t M, int64_t C) {
    // worst case over both vector widths: slab maxima + channel ranges + block maxima
    const ColmaxPlan a = colmax_plan(M, C, true), b = colmax_plan(M, C, false);
    return std::max(a.slabs, b.slabs) * C + C + colmax_reduce_blocks(C);
}

hipError_t launch_colmax(const float* x, int64_t M, int64_t C, int64_t ld, uint32_t* partial, int64_t* slabs,
                         hipStream_t s) {
    *slabs = 0;
    if (M <= 0 || C <= 0) return hipSuccess;
    const bool vec = ((ld & 3) == 0) && ((reinterpret_cast<uintptr_t>(x) & 15) == 0);
    const ColmaxPlan p = colmax_plan(M, C, vec);
    *slabs = p.slabs;
    dim3 grid((unsigned)p.chunks, (unsigned)p.slabs);
    if (vec)
        hipLaunchKernelGGL(k_colmax<4>, grid, dim3(kColThreads), 0, s, x, M, C, ld, p.tpr, p.rows_per_slab, partial);
    else
        hipLaunchKernelGGL(k_colmax<1>, grid, dim3(kColThreads), 0, s, x, M, C, ld, p.tpr, p.rows_per_slab, partial);
    return hipGetLastError();
}

static hipError_t launch_reduce(const uint32_t* partial, int64_t slabs, int64_t C, uint32_t* rbits, uint32_t* bmax,
                                hipStream_t s) {
    const int64_t nb = colmax_reduce_blocks(C);
    if (nb == 0) return hipSuccess;
    hipLaunchKernelGGL(k_colmax_reduce, dim3((unsigned)nb), dim3(kRedThreads), 0, s, partial, slabs, C, rbits, bmax);
    return hipGetLastError();
}

hipError_t launch_finalize_grad(const uint32_t* partial, int64_t slabs, int64_t C, const QuantCfg& cfg,
                                uint32_t* rbits, uint8_t* group, sq_scale* scale, int32_t* layout, hipStream_t s) {
    uint32_t* bmax = rbits + C;
    const hipError_t e = launch_reduce(partial, slabs, C, rbits, bmax, s);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_finalize_grad, dim3(1), dim3(kFinThreads), 0, s, partial, slabs, C, cfg, rbits, bmax,
                       colmax_reduce_blocks(C), group, scale, layout);
    return hipGetLastError();
}

hipError_t launch_finalize_tensor(const uint32_t* partial, int64_t slabs, int64_t C, int Q, uint32_t* rbits,
                                  sq_scale* scale, hipStream_t s) {
    uint32_t* bmax = rbits + C;
    const hipError_t e = launch_reduce(partial, slabs, C, rbits, bmax, s);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_finalize_tensor, dim3(1), dim3(kFinThreads), 0, s, partial, slabs, C, Q, bmax,
                       colmax_reduce_blocks(C), scale);
    return hipGetLastError();
}

hipError_t launch_quantize(const float* x, int64_t M, int64_t C, int64_t ld, const uint8_t* group,
                           const sq_scale* scale, const QuantCfg& cfg, int8_t* q_fold, int64_t ld_fold,
                           int8_t* q_t, int64_t ld_t, const int32_t* layout, hipStream_t s) {
    if (M <= 0 || C <= 0) return hipSuccess;
    const bool vec = ((ld & 3) == 0) && ((reinterpret_cast<uintptr_t>(x) & 15) == 0);
    const bool sr = cfg.round_mode == SQ_ROUND_STOCHASTIC;
    int tc4n = 1;
    while (tc4n < 32 && 4 * tc4n < C) tc4n <<= 1;
    const int64_t rows_per_tile = kQR * (kBlock / tc4n);
    dim3 grid((unsigned)((C + 4 * tc4n - 1) / (4 * tc4n)),
              (unsigned)std::min<int64_t>((M + rows_per_tile - 1) / rows_per_tile, 65535));
    if (vec && sr)
        hipLaunchKernelGGL((k_quantize<4, true>), grid, dim3(kBlock), 0, s, x, M, C, ld, group, scale, cfg, tc4n,
                           q_fold, ld_fold, q_t, ld_t, layout);
    else if (vec)
        hipLaunchKernelGGL((k_quantize<4, false>), grid, dim3(kBlock), 0, s, x, M, C, ld, group, scale, cfg, tc4n,
                           q_fold, ld_fold, q_t, ld_t, layout);
    else if (sr)
        hipLaunchKernelGGL((k_quantize<1, true>), grid, dim3(kBlock), 0, s, x, M, C, ld, group, scale, cfg, tc4n,
                           q_fold, ld_fold, q_t, ld_t, layout);
    else
        hipLaunchKernelGGL((k_quantize<1, false>), grid, dim3(kBlock), 0, s, x, M, C, ld, group, scale, cfg, tc4n,
                           q_fold, ld_fold, q_t, ld_t, layout);
    return hipGetLastError();
}

}  // namespace sq
