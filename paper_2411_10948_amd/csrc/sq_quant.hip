// ShiftQuant quantizer kernels for gfx950.
//
// Three stream-ordered passes (the tensor range r_max is global, so the
// gradient is read twice):
//   k_colmax    per-channel abs-max r_c (Sec. 3.1) as unsigned bit patterns,
//               coalesced float4 row loads, one maximum per channel per slab
//   k_finalize  one block: combines the slab maxima into r_c and r_max, group
//               ids (power-of-two thresholds, Sec. 3.1), scales, flags, and
//               the fold layout for the dgrad
//   k_quantize  scale, round (ties-to-even or Philox stochastic rounding,
//               App. B Eq. "sq"), clamp, write the shift-folded dgrad operand
//               row-major and the codes transposed (LDS 4x4-byte transposes)
//
// All fp32 arithmetic is IEEE with round-to-nearest-even and no contraction
// (the library is built with -ffp-contract=off; the products below also use
// the _rn intrinsics), so the codes are a bit-exact function of the inputs.
#include <algorithm>

#include "sq_internal.h"

namespace sq {

namespace {

constexpr int kBlock = 256;

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

// ---------------------------------------------------------------------------
// ---------------------------------------------------------------------------
// Per-channel abs-max, first level.  The rows are cut into slabs; block
// (chunk, slab) reduces its slab for the chunk's channels and stores the
// slab maxima to partial[slab * C + c] (plain stores: same-address atomics
// from many blocks serialise, so the slabs are combined by the finalize
// kernel instead).  Thread (rl, tc) covers VEC channels starting at
// (chunk * tpr + tc) * VEC and rows rl, rl + kColThreads / tpr, ...
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
                for (; m + 3 * (int64_t)nrl < m_end; m += 4 * (int64_t)nrl) {
                    float4 v[4];
#pragma unroll
                    for (int u = 0; u < 4; ++u)
                        v[u] = *reinterpret_cast<const float4*>(x + (m + u * (int64_t)nrl) * ld + c0);
#pragma unroll
                    for (int u = 0; u < 4; ++u) {
                        best[0] = max(best[0], __float_as_uint(v[u].x) & 0x7FFFFFFFu);
                        best[1] = max(best[1], __float_as_uint(v[u].y) & 0x7FFFFFFFu);
                        best[2] = max(best[2], __float_as_uint(v[u].z) & 0x7FFFFFFFu);
                        best[3] = max(best[3], __float_as_uint(v[u].w) & 0x7FFFFFFFu);
                    }
                }
                for (; m < m_end; m += nrl) {
                    const float4 v = *reinterpret_cast<const float4*>(x + m * ld + c0);
                    best[0] = max(best[0], __float_as_uint(v.x) & 0x7FFFFFFFu);
                    best[1] = max(best[1], __float_as_uint(v.y) & 0x7FFFFFFFu);
                    best[2] = max(best[2], __float_as_uint(v.z) & 0x7FFFFFFFu);
                    best[3] = max(best[3], __float_as_uint(v.w) & 0x7FFFFFFFu);
                }
            }
        }
        for (; m < m_end; m += nrl) {   // scalar path (and the ragged last vector)
#pragma unroll
            for (int j = 0; j < VEC; ++j)
                if (c0 + j < C)
                    best[j] = max(best[j], __float_as_uint(x[m * ld + c0 + j]) & 0x7FFFFFFFu);
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
// Block-wide reductions for the single-block finalize kernels.
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

// Exclusive prefix of a 0/1 flag over the block, plus the block total.
__device__ int block_excl_scan_flag(bool flag, int* sh, int* total) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
    const uint64_t mask = __ballot(flag);
    const int before_in_wave = __popcll(mask & ((1ull << lane) - 1ull));
    __syncthreads();
    if (lane == 0) sh[w] = __popcll(mask);
    __syncthreads();
    int base = 0, tot = 0;
    for (int i = 0; i < nw; ++i) {
        if (i < w) base += sh[i];
        tot += sh[i];
    }
    __syncthreads();
    *total = tot;
    return base + before_in_wave;
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

// ---------------------------------------------------------------------------
// Finalize for the gradient quantizer (one block).  Thread tid owns the
// channels c = tid + k * kFinThreads; for k < kFinRegs their ranges and
// excess shifts stay in registers, beyond that they are re-read from rbits
// (written by the same thread).
// ---------------------------------------------------------------------------
constexpr int kFinThreads = 1024, kFinRegs = 16;

__global__ __launch_bounds__(kFinThreads) void k_finalize_grad(const uint32_t* __restrict__ partial, int64_t S,
                                                               int64_t C, QuantCfg cfg,
                                                               uint32_t* __restrict__ rbits,
                                                               uint8_t* __restrict__ group,
                                                               sq_scale* __restrict__ scale,
                                                               int32_t* __restrict__ layout) {
    __shared__ uint32_t shu[16];
    __shared__ int shi[16];
    const int tid = threadIdx.x;

    // channel ranges and r_max
    uint32_t rr[kFinRegs];
#pragma unroll
    for (int k = 0; k < kFinRegs; ++k) rr[k] = 0u;
    uint32_t mb = 0u;
    if (C < kFinThreads) {
        // few channels, many slabs: W channels x L slab lanes, then combine
        // the lanes through LDS
        __shared__ uint32_t lanes[kFinThreads];
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
        if (tid < C) {
            uint32_t r = 0u;
            for (int l = 0; l < L; ++l) r = max(r, lanes[l * W + tid]);
            rr[0] = r;
            rbits[tid] = r;
            mb = r;
        }
    } else {
        // many channels, few slabs: independent loads across the channels a
        // thread owns
        for (int64_t sl = 0; sl < S; ++sl) {
#pragma unroll
            for (int k = 0; k < kFinRegs; ++k) {
                const int64_t c = tid + (int64_t)k * kFinThreads;
                if (c < C) rr[k] = max(rr[k], partial[sl * C + c]);
            }
        }
#pragma unroll
        for (int k = 0; k < kFinRegs; ++k) {
            const int64_t c = tid + (int64_t)k * kFinThreads;
            if (c < C) rbits[c] = rr[k];
            mb = max(mb, rr[k]);
        }
        for (int64_t c = tid + (int64_t)kFinRegs * kFinThreads; c < C; c += kFinThreads) {
            const uint32_t r = reduce_slabs(partial, S, C, c);
            rbits[c] = r;
            mb = max(mb, r);
        }
    }
    mb = block_max_u32(mb, shu);
    const float r_max = __uint_as_float(mb);
    uint32_t flags = 0u;
    if (mb >= 0x7F800000u) flags = SQ_FLAG_NONFINITE;
    else if (r_max < pow2f(-96)) flags = SQ_FLAG_ZERO;

    const float Qf = (float)cfg.Q;
    if (tid == 0) {
        sq_scale s;
        s.r_max = r_max;
        s.inv = flags ? 0.0f : __fdiv_rn(Qf, r_max);
        s.step = flags ? 0.0f : __fdiv_rn(r_max, Qf);
        s.flags = flags;
        *scale = s;
    }

    // group ids and excess shifts
    uint8_t ee[kFinRegs];
    int emax = 0;
#pragma unroll
    for (int k = 0; k < kFinRegs; ++k) {
        const int64_t c = tid + (int64_t)k * kFinThreads;
        int e = 0;
        if (c < C) {
            const int g = flags ? cfg.num_groups - 1 : group_of(__uint_as_float(rr[k]), r_max, cfg.num_groups);
            group[c] = (uint8_t)g;
            e = excess_of(g, cfg);
        }
        ee[k] = (uint8_t)e;
        emax = max(emax, e);
    }
    for (int64_t c = tid + (int64_t)kFinRegs * kFinThreads; c < C; c += kFinThreads) {
        const int g = flags ? cfg.num_groups - 1 : group_of(__uint_as_float(rbits[c]), r_max, cfg.num_groups);
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
        int written = 0;
#pragma unroll
        for (int k = 0; k < kFinRegs; ++k) {
            const int64_t c_base = (int64_t)k * kFinThreads;
            if (c_base < C) {      // uniform across the block
                const int64_t c = c_base + tid;
                const bool member = c < C && (int)ee[k] > j;
                int chunk_total = 0;
                const int pos = block_excl_scan_flag(member, shi, &chunk_total);
                if (member) ext[start + written + pos] = (int32_t)c;
                written += chunk_total;
            }
        }
        for (int64_t c_base = (int64_t)kFinRegs * kFinThreads; c_base < C; c_base += kFinThreads) {
            const int64_t c = c_base + tid;
            bool member = false;
            if (c < C)
                member = excess_of(group_of(__uint_as_float(rbits[c]), r_max, cfg.num_groups), cfg) > j;
            int chunk_total = 0;
            const int pos = block_excl_scan_flag(member, shi, &chunk_total);
            if (member) ext[start + written + pos] = (int32_t)c;
            written += chunk_total;
        }
        const int padded = (int)round_up(written, kFoldPad);
        for (int i = written + tid; i < padded; i += kFinThreads) ext[start + i] = -1;
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

// ---------------------------------------------------------------------------
// Finalize for per-tensor quantization (one block): the maximum of all slab
// maxima is the tensor's absolute maximum.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kFinThreads) void k_finalize_tensor(const uint32_t* __restrict__ partial, int64_t S,
                                                                 int64_t C, int Q, sq_scale* __restrict__ scale) {
    __shared__ uint32_t shu[16];
    uint32_t mb = 0u;
    for (int64_t c = threadIdx.x; c < C; c += kFinThreads) mb = max(mb, reduce_slabs(partial, S, C, c));
    mb = block_max_u32(mb, shu);
    if (threadIdx.x == 0) {
        const float a = __uint_as_float(mb);
        uint32_t flags = 0u;
        if (mb >= 0x7F800000u) flags = SQ_FLAG_NONFINITE;
        else if (a < pow2f(-96)) flags = SQ_FLAG_ZERO;
        sq_scale s;
        s.r_max = a;
        s.inv = flags ? 0.0f : __fdiv_rn((float)Q, a);
        s.step = flags ? 0.0f : __fdiv_rn(a, (float)Q);
        s.flags = flags;
        *scale = s;
    }
}

// ---------------------------------------------------------------------------
// Quantize.  A block covers a tile of kTM rows x kTC channels; thread
// (tr4, tc4) handles 4x4 sub-blocks: rows tr4*4 .. +3 of each 64-row half,
// channels tc4*4 .. +3.  Codes go to q_fold row-major (shift-folded) and,
// through an LDS transpose, to q_t channel-major.
// ---------------------------------------------------------------------------
constexpr int kTM = 128, kTC = 64, kTS = kTM + 16;   // LDS row stride (bytes)

template <int VEC, bool SR>
__global__ __launch_bounds__(kBlock) void k_quantize(const float* __restrict__ x, int64_t M, int64_t C,
                                                     int64_t ld, const uint8_t* __restrict__ group,
                                                     const sq_scale* __restrict__ scale, QuantCfg cfg,
                                                     int8_t* __restrict__ q_fold, int64_t ld_fold,
                                                     int8_t* __restrict__ q_t, int64_t ld_t,
                                                     const int32_t* __restrict__ layout) {
    __shared__ __attribute__((aligned(16))) uint8_t sT[kTC * kTS];
    const int tid = threadIdx.x;
    const int tc4 = tid & 15, tr4 = tid >> 4;
    const int64_t c_tile = (int64_t)blockIdx.x * kTC;
    const int64_t row_tiles = (M + kTM - 1) / kTM;
    const int64_t c0 = c_tile + tc4 * 4;

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
        const int sh = cfg.num_groups - 1 - g;
        t[j] = group ? min(sh, cfg.T) : 0;
    }
    const bool sr_vec = SR && ((C & 3) == 0);   // 4 channels share one Philox block

    // grid-stride over row tiles (gridDim.y is capped by the launcher)
    for (int64_t rt = blockIdx.y; rt < row_tiles; rt += gridDim.y) {
        const int64_t m_tile = rt * kTM;
#pragma unroll
        for (int half = 0; half < 2; ++half) {
            int code[4][4];   // [row i][channel j]
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int64_t m = m_tile + half * 64 + tr4 * 4 + i;
                float v[4] = {0.f, 0.f, 0.f, 0.f};
                if (m < M) {
                    bool done = false;
                    if constexpr (VEC == 4) {
                        if (c0 + 4 <= C) {
                            const float4 f = *reinterpret_cast<const float4*>(x + m * ld + c0);
                            v[0] = f.x; v[1] = f.y; v[2] = f.z; v[3] = f.w;
                            done = true;
                        }
                    }
                    if (!done) {
#pragma unroll
                        for (int j = 0; j < 4; ++j)
                            if (c0 + j < C) v[j] = x[m * ld + c0 + j];
                    }
                }
                uint32_t u[4] = {0u, 0u, 0u, 0u};
                if (SR && m < M && c0 < C) {
                    if (sr_vec) {
                        const U4 w = philox_block((uint64_t)(m * C + c0) >> 2, cfg);
                        u[0] = w.x >> 8; u[1] = w.y >> 8; u[2] = w.z >> 8; u[3] = w.w >> 8;
                    } else {
#pragma unroll
                        for (int j = 0; j < 4; ++j) {
                            const uint64_t idx = (uint64_t)(m * C + c0 + j);
                            u[j] = pick(philox_block(idx >> 2, cfg), (int)(idx & 3u)) >> 8;
                        }
                    }
                }
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    code[i][j] = (zero || m >= M || c0 + j >= C) ? 0 : quant_one<SR>(v[j], s[j], Qf, u[j]);

                if (q_fold && m < M && c0 < C) {
                    int8_t* dst = q_fold + m * ld_fold + c0;
                    if (c0 + 4 <= C) {
                        const uint32_t packed = ((uint32_t)(uint8_t)(code[i][0] * (1 << t[0]))) |
                                                ((uint32_t)(uint8_t)(code[i][1] * (1 << t[1])) << 8) |
                                                ((uint32_t)(uint8_t)(code[i][2] * (1 << t[2])) << 16) |
                                                ((uint32_t)(uint8_t)(code[i][3] * (1 << t[3])) << 24);
                        *reinterpret_cast<uint32_t*>(dst) = packed;
                    } else {
#pragma unroll
                        for (int j = 0; j < 4; ++j)
                            if (c0 + j < C) dst[j] = (int8_t)(code[i][j] * (1 << t[j]));
                    }
                }
            }
            if (q_t) {
                // 4x4 byte transpose: word j holds channel j of rows i = 0..3
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const uint32_t w = ((uint32_t)(uint8_t)code[0][j]) | ((uint32_t)(uint8_t)code[1][j] << 8) |
                                       ((uint32_t)(uint8_t)code[2][j] << 16) | ((uint32_t)(uint8_t)code[3][j] << 24);
                    *reinterpret_cast<uint32_t*>(&sT[(tc4 * 4 + j) * kTS + half * 64 + tr4 * 4]) = w;
                }
            }
        }

        if (q_t) {
            __syncthreads();
#pragma unroll
            for (int k = 0; k < 2; ++k) {
                const int id = tid + k * kBlock;
                const int ch = id >> 3, seg = id & 7;
                const int64_t c = c_tile + ch;
                const int64_t m = m_tile + seg * 16;
                if (c < C && m < M) {
                    const uint4 w = *reinterpret_cast<const uint4*>(&sT[ch * kTS + seg * 16]);
                    int8_t* dst = q_t + c * ld_t + m;
                    if (m + 16 <= M) {
                        *reinterpret_cast<uint4*>(dst) = w;
                    } else {
                        const uint8_t* b = &sT[ch * kTS + seg * 16];
                        for (int e = 0; e < (int)(M - m); ++e) dst[e] = (int8_t)b[e];
                    }
                }
            }
        }

        // Appended fold columns (dgrad operand only), written by the blocks of the
        // first channel tile for their rows.
        if (q_fold && layout && blockIdx.x == 0) {
            const int D = layout[1];
            const int64_t base = layout[2];
            const int32_t* ext = layout + kLayoutHeader;
            for (int idx = tid; idx < kTM * D; idx += kBlock) {
                const int rr = idx / D, j = idx % D;
                const int64_t m = m_tile + rr;
                if (m >= M) continue;
                const int ch = ext[j];
                int val = 0;
                if (ch >= 0 && !zero) {
                    const int g = (int)group[ch];
                    const float sc_ch = __fmul_rn(sc.inv, pow2f(g));
                    uint32_t u = 0u;
                    if (SR) {
                        const uint64_t e_idx = (uint64_t)(m * C + ch);
                        u = pick(philox_block(e_idx >> 2, cfg), (int)(e_idx & 3u)) >> 8;
                    }
                    const int tt = min(cfg.num_groups - 1 - g, cfg.T);
                    val = quant_one<SR>(x[m * ld + ch], sc_ch, Qf, u) * (1 << tt);
                }
                q_fold[m * ld_fold + base + j] = (int8_t)val;
            }
        }
        __syncthreads();   // sT is reused by the next row tile
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
    // about 512 blocks (two per CU), each slab at least 4 row passes deep
    int64_t slabs = std::max<int64_t>(1, 512 / p.chunks);
    const int64_t min_rows = 4 * (int64_t)nrl;
    slabs = std::min<int64_t>(slabs, std::max<int64_t>(1, (M + min_rows - 1) / min_rows));
    slabs = std::min<int64_t>(slabs, 65535);
    p.rows_per_slab = std::max<int64_t>(1, (M + slabs - 1) / slabs);
    p.slabs = M > 0 ? (M + p.rows_per_slab - 1) / p.rows_per_slab : 0;
    return p;
}

int64_t colmax_workspace_words(int64_t M, int64_t C) {
    // worst case over both vector widths: partial maxima + channel ranges
    const ColmaxPlan a = colmax_plan(M, C, true), b = colmax_plan(M, C, false);
    return std::max(a.slabs, b.slabs) * C + C;
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

hipError_t launch_finalize_grad(const uint32_t* partial, int64_t slabs, int64_t C, const QuantCfg& cfg,
                                uint32_t* rbits, uint8_t* group, sq_scale* scale, int32_t* layout, hipStream_t s) {
    hipLaunchKernelGGL(k_finalize_grad, dim3(1), dim3(kFinThreads), 0, s, partial, slabs, C, cfg, rbits, group,
                       scale, layout);
    return hipGetLastError();
}

hipError_t launch_finalize_tensor(const uint32_t* partial, int64_t slabs, int64_t C, int Q, sq_scale* scale,
                                  hipStream_t s) {
    hipLaunchKernelGGL(k_finalize_tensor, dim3(1), dim3(kFinThreads), 0, s, partial, slabs, C, Q, scale);
    return hipGetLastError();
}

hipError_t launch_quantize(const float* x, int64_t M, int64_t C, int64_t ld, const uint8_t* group,
                           const sq_scale* scale, const QuantCfg& cfg, int8_t* q_fold, int64_t ld_fold,
                           int8_t* q_t, int64_t ld_t, const int32_t* layout, hipStream_t s) {
    if (M <= 0 || C <= 0) return hipSuccess;
    const bool vec = ((ld & 3) == 0) && ((reinterpret_cast<uintptr_t>(x) & 15) == 0);
    const bool sr = cfg.round_mode == SQ_ROUND_STOCHASTIC;
    dim3 grid((unsigned)((C + kTC - 1) / kTC), (unsigned)std::min<int64_t>((M + kTM - 1) / kTM, 65535));
    if (vec && sr)
        hipLaunchKernelGGL((k_quantize<4, true>), grid, dim3(kBlock), 0, s, x, M, C, ld, group, scale, cfg,
                           q_fold, ld_fold, q_t, ld_t, layout);
    else if (vec)
        hipLaunchKernelGGL((k_quantize<4, false>), grid, dim3(kBlock), 0, s, x, M, C, ld, group, scale, cfg,
                           q_fold, ld_fold, q_t, ld_t, layout);
    else if (sr)
        hipLaunchKernelGGL((k_quantize<1, true>), grid, dim3(kBlock), 0, s, x, M, C, ld, group, scale, cfg,
                           q_fold, ld_fold, q_t, ld_t, layout);
    else
        hipLaunchKernelGGL((k_quantize<1, false>), grid, dim3(kBlock), 0, s, x, M, C, ld, group, scale, cfg,
                           q_fold, ld_fold, q_t, ld_t, layout);
    return hipGetLastError();
}

}  // namespace sq
