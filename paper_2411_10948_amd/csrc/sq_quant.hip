// ShiftQuant quantizer kernels for gfx950.
//
// Stream-ordered passes (the tensor range r_max is global, so the gradient is
// read twice):
//   k_colmax         per-channel abs-max r_c (Sec. 3.1) as unsigned bit
//                    patterns: coalesced float4 row loads, one maximum per
//                    channel per row slab (plain stores, no atomics) and one
//                    per block
//   finalize         r_max, group ids (power-of-two thresholds, Sec. 3.1),
//                    scales, flags, and the fold layout for dgrad: one block
//                    (k_finalize_grad) for few channels, else the group kernel
//                    (k_final_groups_slabs, which also combines the slabs per
//                    channel) and the placement kernel (k_final_place);
//                    k_colmax_reduce + k_final_groups serve channel ranges
//                    that come from the producer of dY
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

// The 16-bit uniform of the element with logical index idx = m * C + c: one
// Philox block per 8 consecutive indices, half idx % 2 (low first) of word
// (idx / 2) % 4.
__device__ __forceinline__ uint32_t sr_uniform16(uint64_t idx, const QuantCfg& cfg) {
    return (pick(philox_block(idx >> 3, cfg), (int)((idx >> 1) & 3u)) >> (16u * (uint32_t)(idx & 1u))) & 0xFFFFu;
}

// One code: v = fl(x * s); round; clamp to [-Q, Q].  u16 is the 16-bit
// uniform used only by stochastic rounding.
template <bool SR>
__device__ __forceinline__ int quant_one(float x, float s, float Qf, uint32_t u16) {
    const float v = __fmul_rn(x, s);
    float qf;
    if (SR) {
        const float l = floorf(v);
        const float f = __fsub_rn(v, l);
        qf = ((float)u16 < __fmul_rn(f, 65536.0f)) ? __fadd_rn(l, 1.0f) : l;
    } else {
        qf = rintf(v);
    }
    qf = fminf(fmaxf(qf, -Qf), Qf);
    return (int)qf;
}

// The same code as a float (an exact integer in [-Q, Q]).
template <bool SR>
__device__ __forceinline__ float quant_onef(float x, float s, float Qf, uint32_t u16) {
    const float v = __fmul_rn(x, s);
    float qf;
    if (SR) {
        const float l = floorf(v);
        const float f = __fsub_rn(v, l);
        qf = ((float)u16 < __fmul_rn(f, 65536.0f)) ? __fadd_rn(l, 1.0f) : l;
    } else {
        qf = rintf(v);
    }
    return fminf(fmaxf(qf, -Qf), Qf);
}

__device__ __forceinline__ uint32_t absbits(float x) { return __float_as_uint(x) & 0x7FFFFFFFu; }

// ---------------------------------------------------------------------------
// Per-channel abs-max, first level.  The rows are cut into slabs; block
// (chunk, slab) reduces its slab for the chunk's channels and stores the
// slab maxima to partial[slab * C + c] (plain stores: same-address atomics
// from many blocks serialise, so the slabs are combined in a second step).
// Thread (rl, tc) covers VEC channels starting at (chunk * tpr + tc) * VEC and
// rows rl, rl + kColThreads / tpr, ... of the slab, 8 loads in flight.
// NT: nontemporal loads, for gradients larger than the last-level cache (see
// launch_colmax).
// ---------------------------------------------------------------------------
constexpr uint64_t kLastLevelCacheBytes = 256ull << 20;   // MI355X last-level (memory-side) cache
constexpr int kColThreads = 512;
typedef float v4f __attribute__((ext_vector_type(4)));

template <int VEC, bool NT>
__global__ __launch_bounds__(kColThreads) void k_colmax(const float* __restrict__ x, int64_t M, int64_t C,
                                                        int64_t ld, int tpr, int64_t rows_per_slab,
                                                        uint32_t* __restrict__ partial,
                                                        uint32_t* __restrict__ block_max) {
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
                // batches of 8 rows, the next batch in flight while one is
                // reduced.  Rows past the slab re-read its last row (the
                // maximum is unchanged): no branch between the loads, so the
                // wait before a batch's reduction leaves the next batch in flight.
                const int64_t step = nrl;
                auto load8 = [&](int64_t mm, float4 (&v)[8]) {
#pragma unroll
                    for (int u = 0; u < 8; ++u) {
                        const int64_t row = min(mm + u * step, m_end - 1);
                        if (NT) {
                            const v4f t = __builtin_nontemporal_load(reinterpret_cast<const v4f*>(x + row * ld + c0));
                            v[u] = make_float4(t.x, t.y, t.z, t.w);
                        } else {
                            v[u] = *reinterpret_cast<const float4*>(x + row * ld + c0);
                        }
                    }
                };
                auto reduce8 = [&](const float4 (&v)[8]) {
#pragma unroll
                    for (int u = 0; u < 8; ++u) {
                        best[0] = max(best[0], absbits(v[u].x));
                        best[1] = max(best[1], absbits(v[u].y));
                        best[2] = max(best[2], absbits(v[u].z));
                        best[3] = max(best[3], absbits(v[u].w));
                    }
                };
                if (m < m_end) {
                    float4 va[8], vb[8];
                    load8(m, va);
                    for (; m < m_end; m += 16 * step) {
                        load8(m + 8 * step, vb);
                        reduce8(va);
                        load8(m + 16 * step, va);
                        reduce8(vb);
                    }
                }
                m = m_end;
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
    // the block's maximum over its channels (the rl == 0 threads, tid < tpr,
    // all in wave 0), so that r_max needs no pass over the channel ranges
    if (block_max && tid < 64) {
        uint32_t mb = 0u;
        if (rl == 0 && c0 < C)
#pragma unroll
            for (int j = 0; j < VEC; ++j)
                if (c0 + j < C) mb = max(mb, best[j]);
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) mb = max(mb, (uint32_t)__shfl_xor((int)mb, o, 64));
        if (tid == 0) block_max[(int64_t)blockIdx.y * gridDim.x + blockIdx.x] = mb;
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

// Second level for many channels: rbits[c] = max over slabs, and the block's
// maximum in bmax[blockIdx.x].
constexpr int kRedThreads = 256;

// kRedLanes threads per channel share its slabs (slab s goes to lane s mod
// kRedLanes), combined in LDS: a block of kRedThreads channels uses
// kRedLanes * kRedThreads threads.
constexpr int kRedLanes = 4;
__global__ __launch_bounds__(kRedThreads * kRedLanes) void k_colmax_reduce(const uint32_t* __restrict__ partial,
                                                                           int64_t S, int64_t C,
                                                                           uint32_t* __restrict__ rbits,
                                                                           uint32_t* __restrict__ bmax) {
    __shared__ uint32_t lanes[kRedLanes][kRedThreads];
    __shared__ uint32_t shu[kRedThreads * kRedLanes / 64];
    const int ch = threadIdx.x % kRedThreads, ln = threadIdx.x / kRedThreads;
    const int64_t c = (int64_t)blockIdx.x * kRedThreads + ch;
    uint32_t a[4] = {0u, 0u, 0u, 0u};
    if (c < C) {
        int64_t s = ln;
        for (; s + 3 * kRedLanes < S; s += 4 * kRedLanes) {
#pragma unroll
            for (int u = 0; u < 4; ++u) a[u] = max(a[u], partial[(s + u * kRedLanes) * C + c]);
        }
        for (; s < S; s += kRedLanes) a[0] = max(a[0], partial[s * C + c]);
    }
    lanes[ln][ch] = max(max(a[0], a[1]), max(a[2], a[3]));
    __syncthreads();
    uint32_t r = 0u;
    if (ln == 0) {
#pragma unroll
        for (int l = 0; l < kRedLanes; ++l) r = max(r, lanes[l][ch]);
        if (c < C) rbits[c] = r;
    }
    r = block_max_u32(r, shu);
    if (threadIdx.x == 0) bmax[blockIdx.x] = r;
}

// Channel ranges for fewer channels than threads: W channel units x L slab
// lanes, combined through LDS (lanes holds 4 * kFinThreads words).  A unit is
// 4 channels read as one 16-byte load when C is a multiple of 4, else 1.
// Thread tid < C returns r_{tid}; the others 0.
constexpr int kFinThreads = 1024;

__device__ uint32_t small_channel_ranges(const uint32_t* __restrict__ partial, int64_t S, int64_t C,
                                         uint32_t* lanes) {
    const int tid = threadIdx.x;
    const bool v4 = (C & 3) == 0;
    const int units = v4 ? (int)(C / 4) : (int)C;
    int W = 1;
    while (W < units) W <<= 1;
    const int L = kFinThreads / W;
    const int cl = tid % W, lane = tid / W;
    uint32_t a[4] = {0u, 0u, 0u, 0u};
    if (cl < units) {
        if (v4) {
            const uint32_t* base = partial + 4 * (int64_t)cl;
            int64_t sl = lane;
            for (; sl + 7 * (int64_t)L < S; sl += 8 * (int64_t)L) {
                uint4 v[8];
#pragma unroll
                for (int u = 0; u < 8; ++u) v[u] = *reinterpret_cast<const uint4*>(base + (sl + u * (int64_t)L) * C);
#pragma unroll
                for (int u = 0; u < 8; ++u) {
                    a[0] = max(a[0], v[u].x); a[1] = max(a[1], v[u].y);
                    a[2] = max(a[2], v[u].z); a[3] = max(a[3], v[u].w);
                }
            }
            for (; sl < S; sl += L) {
                const uint4 v = *reinterpret_cast<const uint4*>(base + sl * C);
                a[0] = max(a[0], v.x); a[1] = max(a[1], v.y); a[2] = max(a[2], v.z); a[3] = max(a[3], v.w);
            }
        } else {
            uint32_t b[8] = {0u, 0u, 0u, 0u, 0u, 0u, 0u, 0u};
            int64_t sl = lane;
            for (; sl + 7 * (int64_t)L < S; sl += 8 * (int64_t)L) {
#pragma unroll
                for (int u = 0; u < 8; ++u) b[u] = max(b[u], partial[(sl + u * (int64_t)L) * C + cl]);
            }
            for (; sl < S; sl += L) b[0] = max(b[0], partial[sl * C + cl]);
#pragma unroll
            for (int u = 0; u < 8; ++u) a[0] = max(a[0], b[u]);
        }
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) lanes[4 * tid + k] = a[k];
    __syncthreads();
    uint32_t r = 0u;
    if (tid < C) {
        const int q = v4 ? tid / 4 : tid, k = v4 ? tid % 4 : 0;
        for (int l = 0; l < L; ++l) r = max(r, lanes[4 * (l * W + q) + k]);
    }
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

// Shift windows of the fold (the layout is documented in sq_internal.h),
// computed by one thread from the number of channels at each shift.
struct FoldPlan {
    int nr, main_r, D, H, F;
    int win_of[kMaxRegions];      // region of each shift value
    int base[kMaxRegions];        // lowest shift of each region
    int cnt[kMaxRegions];         // channels of each region
    int ext_start[kMaxRegions];   // first appended column (non-main regions)
    int flat[kMaxRegions];        // first flat K column
    int run[kMaxRegions];         // channels ranked so far
};

// The plan is computed by one thread in registers (every loop has a
// compile-time bound of kMaxRegions shift values) and stored to LDS once.
// Window of shift value s: key 0 for the main window [B*, B* + T], key j > 0
// for [B* + j (T + 1), ...] above it, key -j for the j-th window below it
// (its base clipped at 0).  Regions are the non-empty windows (and always the
// main one) in descending key order, which is descending base.
__device__ void make_fold_plan(const int* n_lds, int S, int T, int64_t C, FoldPlan& P) {
    int n[kMaxRegions];
#pragma unroll
    for (int s = 0; s < kMaxRegions; ++s) n[s] = s <= S ? n_lds[s] : 0;
    // the window [B, B + T] holding the most channels (lowest B on ties)
    int bstar = 0, best = -1;
#pragma unroll
    for (int B = 0; B < kMaxRegions; ++B) {
        if (B > (S - T > 0 ? S - T : 0)) break;
        int c = 0;
#pragma unroll
        for (int s = 0; s < kMaxRegions; ++s) c += (s >= B && s <= B + T) ? n[s] : 0;
        if (c > best) { best = c; bstar = B; }
    }
    auto key_of = [&](int s) { return s >= bstar ? (s - bstar) / (T + 1) : -1 - (bstar - 1 - s) / (T + 1); };
    // channels per key, keys -7 .. 7
    int kc[2 * kMaxRegions - 1];
#pragma unroll
    for (int k = 0; k < 2 * kMaxRegions - 1; ++k) kc[k] = 0;
#pragma unroll
    for (int s = 0; s < kMaxRegions; ++s) {
        const int key = key_of(s) + (kMaxRegions - 1);
#pragma unroll
        for (int k = 0; k < 2 * kMaxRegions - 1; ++k) kc[k] += (k == key && s <= S) ? n[s] : 0;
    }
    // regions in descending key order
    int nr = 0, main_r = 0, flat = 0, ext = 0, H = 0;
    int region_of_key[2 * kMaxRegions - 1];
#pragma unroll
    for (int k = 2 * kMaxRegions - 2; k >= 0; --k) {
        const int key = k - (kMaxRegions - 1);
        region_of_key[k] = -1;
        if (!(kc[k] > 0 || key == 0)) continue;
        const int lo = key >= 0 ? bstar + key * (T + 1) : max(0, bstar + key * (T + 1));
        const int r = nr++;
        region_of_key[k] = r;
        P.base[r] = lo;
        P.cnt[r] = kc[k];
        P.flat[r] = flat;
        P.run[r] = 0;
        if (key == 0) {
            main_r = r;
            P.ext_start[r] = -1;
            H = ext;
            flat += (int)round_up(C, kFoldPad);
        } else {
            P.ext_start[r] = ext;
            ext += (int)round_up(kc[k], kFoldPad);
            flat += (int)round_up(kc[k], kFoldPad);
        }
    }
#pragma unroll
    for (int s = 0; s < kMaxRegions; ++s) {
        const int k = key_of(s) + (kMaxRegions - 1);
        int r = 0;
#pragma unroll
        for (int kk = 0; kk < 2 * kMaxRegions - 1; ++kk) r = kk == k ? region_of_key[kk] : r;
        P.win_of[s] = s <= S ? r : 0;
    }
    P.nr = nr;
    P.main_r = main_r;
    P.D = ext;
    P.H = H;
    P.F = P.base[nr - 1];
}

__device__ __forceinline__ int wave_sum(int v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

// ---------------------------------------------------------------------------
// Finalize for the gradient quantizer (one block): r_max, scales and flags,
// the group of every channel (channel c handled by thread c mod kFinThreads),
// the shift windows of the fold, and each channel's place in q_fold.  The
// appended columns of a region list its channels in ascending order; a
// channel's rank comes from wave ballots plus per-wave totals in LDS.
// ---------------------------------------------------------------------------
constexpr int kFinWaves = kFinThreads / 64;
constexpr int kChunk = 16;   // rounds of kFinThreads channels whose loads are batched

__global__ __launch_bounds__(kFinThreads) void k_finalize_grad(const uint32_t* __restrict__ partial, int64_t S,
                                                               int64_t C, QuantCfg cfg,
                                                               const uint32_t* __restrict__ rbits,
                                                               const uint32_t* __restrict__ bmax, int64_t nb,
                                                               uint8_t* __restrict__ group,
                                                               sq_scale* __restrict__ scale,
                                                               int32_t* __restrict__ layout, int64_t ext_max) {
    __shared__ uint32_t shu[16];
    __shared__ int cnt[kChunk][kFinWaves][kMaxRegions];
    __shared__ int pre[kChunk][kFinWaves][kMaxRegions];
    __shared__ int tot[kChunk][kMaxRegions];
    __shared__ int roundpre[kChunk][kMaxRegions];
    __shared__ uint32_t lanes[4 * kFinThreads];
    __shared__ FoldPlan P;
    __shared__ int nsh[kMaxRegions];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int Sh = cfg.num_groups - 1;   // largest shift

    uint32_t mb = 0u, r_small = 0u;
    if (C < kFinThreads) {
        r_small = small_channel_ranges(partial, S, C, lanes);
        mb = r_small;
    } else {
        for (int64_t i = tid; i < nb; i += kFinThreads) mb = max(mb, bmax[i]);
    }
    mb = block_max_u32(mb, shu);
    const sq_scale sc = make_scale(mb, (float)cfg.Q);
    if (tid == 0) *scale = sc;
    const bool flagged = sc.flags != 0u;

    int32_t* ext = layout + kLayoutHeader;
    int32_t* desc = ext + ext_max;
    if (ext_max == 0) {
        // every shift fits int8 (N_G - 1 <= T): one window at base 0, the
        // code of channel c stored as code << sh_c in its own column
        for (int64_t c = tid; c < C; c += kFinThreads) {
            const uint32_t rb = C < kFinThreads ? r_small : rbits[c];
            const int g = flagged ? Sh : group_of(__uint_as_float(rb), sc.r_max, cfg.num_groups);
            group[c] = (uint8_t)g;
            desc[c] = Sh - g;
        }
        if (tid < kLayoutHeader) {
            int v = 0;
            if (tid == kLayNR) v = 1;
            else if (tid == kLayBase) v = (int)fold_ext_base(C);
            else if (tid > kLayStart && tid < kLayStart + kMaxRegions) v = 0x7FFFFFFF;
            layout[tid] = v;
        }
        return;
    }

    // Channel c = k * kFinThreads + tid is handled by this thread in round k;
    // rounds are processed in chunks of kChunk with their loads batched.
    const int64_t rounds = (C + kFinThreads - 1) / kFinThreads;

    // groups and the number of channels at each shift
    int hist[kMaxRegions];
#pragma unroll
    for (int s = 0; s < kMaxRegions; ++s) hist[s] = 0;
    for (int64_t k0 = 0; k0 < rounds; k0 += kChunk) {
        uint32_t rb[kChunk];
#pragma unroll
        for (int k = 0; k < kChunk; ++k) {
            const int64_t c = (k0 + k) * kFinThreads + tid;
            rb[k] = c < C ? (C < kFinThreads ? r_small : rbits[c]) : 0u;
        }
#pragma unroll
        for (int k = 0; k < kChunk; ++k) {
            const int64_t c = (k0 + k) * kFinThreads + tid;
            if (c >= C) continue;
            const int g = flagged ? Sh : group_of(__uint_as_float(rb[k]), sc.r_max, cfg.num_groups);
            group[c] = (uint8_t)g;
#pragma unroll
            for (int s = 0; s < kMaxRegions; ++s) hist[s] += (Sh - g) == s;
        }
    }
#pragma unroll
    for (int s = 0; s < kMaxRegions; ++s) {
        const int v = wave_sum(hist[s]);
        if (lane == 0) cnt[0][wave][s] = v;
    }
    __syncthreads();
    if (tid < kMaxRegions) {
        int v = 0;
        for (int w = 0; w < kFinWaves; ++w) v += cnt[0][w][tid];
        nsh[tid] = v;
    }
    __syncthreads();
    if (tid == 0) make_fold_plan(nsh, Sh, cfg.T, C, P);
    __syncthreads();

    // place of every channel: descriptor ((pos + 1) << 4) | t, and the
    // appended-column list.  Appended channels are ranked per round with wave
    // ballots; cnt[k][w][q] counts those of region q in wave w of round k,
    // and pre[k][w][q] is the number of region-q channels before that wave
    // (earlier chunks, earlier rounds, earlier waves).
    const int nr = P.nr, main_r = P.main_r;
    const uint64_t below = (1ull << lane) - 1ull;
    for (int64_t k0 = 0; k0 < rounds; k0 += kChunk) {
        uint8_t gk[kChunk];
#pragma unroll
        for (int k = 0; k < kChunk; ++k) {
            const int64_t c = (k0 + k) * kFinThreads + tid;
            gk[k] = c < C ? group[c] : (uint8_t)0;   // written by this thread above
        }
        int code_r[kChunk], rank[kChunk];
#pragma unroll
        for (int k = 0; k < kChunk; ++k) {
            const int64_t c = (k0 + k) * kFinThreads + tid;
            int r = main_r;
            if (c < C) r = P.win_of[Sh - (int)gk[k]];
            code_r[k] = r;
            const bool is_ext = c < C && r != main_r;
            rank[k] = 0;
            if (k0 + k >= rounds) continue;   // uniform: no channel of this round exists
            for (int q = 0; q < nr; ++q) {
                const uint64_t m = __ballot(is_ext && r == q);
                if (is_ext && r == q) rank[k] = __popcll(m & below);
                if (lane == 0) cnt[k][wave][q] = __popcll(m);
            }
        }
        __syncthreads();
        // thread (k, q): exclusive prefix over the waves of round k
        if (tid < kChunk * kMaxRegions) {
            const int k = tid / kMaxRegions, q = tid % kMaxRegions;
            int acc = 0;
            if (q < nr && k0 + k < rounds)
                for (int w = 0; w < kFinWaves; ++w) {
                    pre[k][w][q] = acc;
                    acc += cnt[k][w][q];
                }
            tot[k][q] = acc;
        }
        __syncthreads();
        // thread q: prefix over the rounds, plus the channels of earlier chunks
        if (tid < nr) {
            int acc = P.run[tid];
            for (int k = 0; k < kChunk && k0 + k < rounds; ++k) {
                roundpre[k][tid] = acc;
                acc += tot[k][tid];
            }
            P.run[tid] = acc;
        }
        __syncthreads();
#pragma unroll
        for (int k = 0; k < kChunk; ++k) {
            const int64_t c = (k0 + k) * kFinThreads + tid;
            if (c >= C) continue;
            const int r = code_r[k];
            const int t = (Sh - (int)gk[k]) - P.base[r];
            int pos = -1;
            if (r != main_r) {
                pos = P.ext_start[r] + roundpre[k][r] + pre[k][wave][r] + rank[k];
                ext[pos] = (int32_t)c;
            }
            desc[c] = ((pos + 1) << 4) | t;
        }
        __syncthreads();   // cnt / pre / roundpre free for the next chunk
    }
    for (int r = 0; r < nr; ++r) {
        if (r == main_r) continue;
        const int padded = (int)round_up(P.cnt[r], kFoldPad);
        for (int i = P.cnt[r] + tid; i < padded; i += kFinThreads) ext[P.ext_start[r] + i] = -1;
    }
    if (tid < kLayoutHeader) {
        int v = 0;
        if (tid == kLayNR) v = nr;
        else if (tid == kLayD) v = P.D;
        else if (tid == kLayBase) v = (int)fold_ext_base(C);
        else if (tid == kLayF) v = P.F;
        else if (tid == kLayH) v = P.H;
        else if (tid >= kLayStart && tid < kLayStart + kMaxRegions)
            v = tid - kLayStart < nr ? P.flat[tid - kLayStart] : 0x7FFFFFFF;
        else if (tid >= kLayShift && tid < kLayShift + kMaxRegions) {
            const int r = tid - kLayShift;
            v = (r > 0 && r < nr) ? P.base[r - 1] - P.base[r] : 0;
        }
        layout[tid] = v;
    }
}

// ---------------------------------------------------------------------------
// Finalize for many channels (C >= kFinThreads), spread over the blocks of
// the second reduction level (kRedThreads channels each) in two kernels:
//   k_final_groups: r_max from the per-block maxima (every block), the group
//     of each of its channels, and the block's count of channels per shift;
//     with one fold window the descriptors and the header too;
//   k_final_place:  every block plans the windows from the summed counts
//     (the same plan everywhere), takes its region offsets from the counts
//     of the blocks before it, and ranks its appended channels with wave
//     ballots; block 0 writes the header and the region padding.
// ---------------------------------------------------------------------------
// Groups of the block's channels (thread t < kRedThreads: channel
// blockIdx.x * kRedThreads + t with range bits rb; the other threads pass
// nothing), the descriptors and header with one fold window, else the
// block's count of channels per shift.  Every thread of the block calls it.
__device__ void final_groups_body(int64_t c, uint32_t rb, const sq_scale& sc, int64_t C, const QuantCfg& cfg,
                                  uint8_t* __restrict__ group, int32_t* __restrict__ layout, int64_t ext_max,
                                  int32_t* __restrict__ hist, int* cnt) {
    const int tid = threadIdx.x;
    const int Sh = cfg.num_groups - 1;
    int sh = -1;
    if (tid < kRedThreads && c < C) {
        const int g = sc.flags ? Sh : group_of(__uint_as_float(rb), sc.r_max, cfg.num_groups);
        group[c] = (uint8_t)g;
        sh = Sh - g;
    }
    if (ext_max == 0) {
        // one window at base 0: the code of channel c is stored as code << sh_c in its own column
        int32_t* desc = layout + kLayoutHeader;
        if (tid < kRedThreads && c < C) desc[c] = sh;
        if (blockIdx.x == 0 && tid < kLayoutHeader) {
            int v = 0;
            if (tid == kLayNR) v = 1;
            else if (tid == kLayBase) v = (int)fold_ext_base(C);
            else if (tid > kLayStart && tid < kLayStart + kMaxRegions) v = 0x7FFFFFFF;
            layout[tid] = v;
        }
        return;
    }
    if (tid < kMaxRegions) cnt[tid] = 0;
    __syncthreads();
#pragma unroll
    for (int q = 0; q < kMaxRegions; ++q) {
        const uint64_t m = __ballot(sh == q);
        if ((tid & 63) == 0 && m) atomicAdd(&cnt[q], __popcll(m));
    }
    __syncthreads();
    if (tid < kMaxRegions) hist[blockIdx.x * kMaxRegions + tid] = cnt[tid];
}

__global__ __launch_bounds__(kRedThreads) void k_final_groups(const uint32_t* __restrict__ rbits,
                                                               const uint32_t* __restrict__ bmax, int64_t nb,
                                                               int64_t C, QuantCfg cfg, uint8_t* __restrict__ group,
                                                               sq_scale* __restrict__ scale, int32_t* __restrict__ layout,
                                                               int64_t ext_max, int32_t* __restrict__ hist) {
    __shared__ uint32_t shu[kRedThreads / 64];
    __shared__ int cnt[kMaxRegions];
    const int tid = threadIdx.x;
    uint32_t mb = 0u;
    for (int64_t i = tid; i < nb; i += kRedThreads) mb = max(mb, bmax[i]);
    mb = block_max_u32(mb, shu);
    const sq_scale sc = make_scale(mb, (float)cfg.Q);
    if (blockIdx.x == 0 && tid == 0) *scale = sc;
    const int64_t c = (int64_t)blockIdx.x * kRedThreads + tid;
    final_groups_body(c, c < C ? rbits[c] : 0u, sc, C, cfg, group, layout, ext_max, hist, cnt);
}

// The same from the abs-max pass's outputs directly: r_max from its block
// maxima, and each channel's range from its slab maxima (kRedLanes threads
// per channel, as k_colmax_reduce), one launch fewer.
__global__ __launch_bounds__(kRedThreads * kRedLanes) void k_final_groups_slabs(
    const uint32_t* __restrict__ partial, int64_t S, const uint32_t* __restrict__ block_max, int64_t nbm, int64_t C,
    QuantCfg cfg, uint8_t* __restrict__ group, sq_scale* __restrict__ scale, int32_t* __restrict__ layout,
    int64_t ext_max, int32_t* __restrict__ hist) {
    __shared__ uint32_t lanes[kRedLanes][kRedThreads];
    __shared__ uint32_t shu[kRedThreads * kRedLanes / 64];
    __shared__ int cnt[kMaxRegions];
    const int tid = threadIdx.x;
    const int ch = tid % kRedThreads, ln = tid / kRedThreads;
    const int64_t c = (int64_t)blockIdx.x * kRedThreads + ch;
    uint32_t a[4] = {0u, 0u, 0u, 0u};
    if (c < C) {
        int64_t s = ln;
        for (; s + 3 * kRedLanes < S; s += 4 * kRedLanes) {
#pragma unroll
            for (int u = 0; u < 4; ++u) a[u] = max(a[u], partial[(s + u * kRedLanes) * C + c]);
        }
        for (; s < S; s += kRedLanes) a[0] = max(a[0], partial[s * C + c]);
    }
    uint32_t mb = 0u;
    for (int64_t i = tid; i < nbm; i += kRedThreads * kRedLanes) mb = max(mb, block_max[i]);
    mb = block_max_u32(mb, shu);
    lanes[ln][ch] = max(max(a[0], a[1]), max(a[2], a[3]));
    __syncthreads();
    uint32_t rb = 0u;
    if (ln == 0) {
#pragma unroll
        for (int l = 0; l < kRedLanes; ++l) rb = max(rb, lanes[l][ch]);
    }
    const sq_scale sc = make_scale(mb, (float)cfg.Q);
    if (blockIdx.x == 0 && tid == 0) *scale = sc;
    final_groups_body(c, rb, sc, C, cfg, group, layout, ext_max, hist, cnt);
}

__global__ __launch_bounds__(kRedThreads) void k_final_place(const uint8_t* __restrict__ group,
                                                              const int32_t* __restrict__ hist, int64_t nb, int64_t C,
                                                              QuantCfg cfg, int32_t* __restrict__ layout,
                                                              int64_t ext_max) {
    __shared__ int tot[kMaxRegions], before[kMaxRegions];
    __shared__ int wcnt[kRedThreads / 64][kMaxRegions];
    __shared__ FoldPlan P;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int Sh = cfg.num_groups - 1;
    // channels per shift: all blocks, and the blocks before this one (thread
    // t sums shift t % 8 over the blocks b = t / 8 (mod 32), then LDS atomics)
    if (tid < kMaxRegions) { tot[tid] = 0; before[tid] = 0; }
    __syncthreads();
    {
        const int s = tid % kMaxRegions;
        int vt = 0, vb = 0;
        for (int64_t b = tid / kMaxRegions; b < nb; b += kRedThreads / kMaxRegions) {
            const int h = hist[b * kMaxRegions + s];
            vt += h;
            vb += b < (int64_t)blockIdx.x ? h : 0;
        }
        if (vt) atomicAdd(&tot[s], vt);
        if (vb) atomicAdd(&before[s], vb);
    }
    __syncthreads();
    if (tid == 0) make_fold_plan(tot, Sh, cfg.T, C, P);
    __syncthreads();
    const int nr = P.nr, main_r = P.main_r;
    int32_t* ext = layout + kLayoutHeader;
    int32_t* desc = ext + ext_max;
    const int64_t c = (int64_t)blockIdx.x * kRedThreads + tid;
    const int sh = c < C ? Sh - (int)group[c] : 0;
    const int r = c < C ? P.win_of[sh] : main_r;
    const bool is_ext = c < C && r != main_r;
    int rank = 0;
    const uint64_t below = (1ull << lane) - 1ull;
    for (int q = 0; q < nr; ++q) {
        const uint64_t m = __ballot(is_ext && r == q);
        if (is_ext && r == q) rank = __popcll(m & below);
        if (lane == 0) wcnt[wave][q] = __popcll(m);
    }
    __syncthreads();
    if (c < C) {
        int pos = -1;
        if (is_ext) {
            // region offset: appended channels of region r in earlier blocks and waves
            int off = 0;
#pragma unroll
            for (int s2 = 0; s2 < kMaxRegions; ++s2)
                if (s2 <= Sh && P.win_of[s2] == r) off += before[s2];
            for (int w = 0; w < wave; ++w) off += wcnt[w][r];
            pos = P.ext_start[r] + off + rank;
            ext[pos] = (int32_t)c;
        }
        desc[c] = ((pos + 1) << 4) | (sh - P.base[r]);
    }
    if (blockIdx.x != 0) return;
    for (int q = 0; q < nr; ++q) {
        if (q == main_r) continue;
        const int padded = (int)round_up(P.cnt[q], kFoldPad);
        for (int i = P.cnt[q] + tid; i < padded; i += kRedThreads) ext[P.ext_start[q] + i] = -1;
    }
    if (tid < kLayoutHeader) {
        int v = 0;
        if (tid == kLayNR) v = nr;
        else if (tid == kLayD) v = P.D;
        else if (tid == kLayBase) v = (int)fold_ext_base(C);
        else if (tid == kLayF) v = P.F;
        else if (tid == kLayH) v = P.H;
        else if (tid >= kLayStart && tid < kLayStart + kMaxRegions)
            v = tid - kLayStart < nr ? P.flat[tid - kLayStart] : 0x7FFFFFFF;
        else if (tid >= kLayShift && tid < kLayShift + kMaxRegions) {
            const int q = tid - kLayShift;
            v = (q > 0 && q < nr) ? P.base[q - 1] - P.base[q] : 0;
        }
        layout[tid] = v;
    }
}

// Finalize for per-tensor quantization (one block): the tensor's absolute
// maximum is the maximum over all slab maxima.
__global__ __launch_bounds__(kFinThreads) void k_finalize_tensor(const uint32_t* __restrict__ partial, int64_t S,
                                                                 int64_t C, int Q, const uint32_t* __restrict__ bmax,
                                                                 int64_t nb, sq_scale* __restrict__ scale) {
    __shared__ uint32_t shu[16];
    __shared__ uint32_t lanes[4 * kFinThreads];
    uint32_t mb = 0u;
    if (C < kFinThreads) mb = small_channel_ranges(partial, S, C, lanes);
    else
        for (int64_t i = threadIdx.x; i < nb; i += kFinThreads) mb = max(mb, bmax[i]);
    mb = block_max_u32(mb, shu);
    if (threadIdx.x == 0) *scale = make_scale(mb, (float)Q);
}

// ---------------------------------------------------------------------------
// Quantize.  A block quantizes tiles of TR rows x TC channels (64 or 128 each,
// smaller where the tensor would give too few tiles to fill the chip),
// striding over the tiles; neighbouring
// channel tiles of a row tile go to consecutive blocks.  Thread (rq, cq)
// handles, in each pass over the tile, the 4 consecutive rows 4 rq .. 4 rq + 3
// of the channel quad 4 cq .. 4 cq + 3: one 16-byte load per row, the row's 4
// shift-folded codes as one 4-byte store into q_fold (a wave writes whole
// row segments), and each channel's 4 codes as one word into an LDS tile
// [channel][row], from which the block writes q_t as 16-byte chunks, so a
// 128-row tile completes whole 128-byte lines of q_t.  Low register use keeps many
// waves per SIMD in flight to hide the memory latency.
// ---------------------------------------------------------------------------
constexpr int kBlock = 256;

template <int TC, int kTR, int VEC, bool SR>
__global__ __launch_bounds__(kBlock) void k_quantize(const float* __restrict__ x, int64_t M, int64_t C,
                                                     int64_t ld, const uint8_t* __restrict__ group,
                                                     const sq_scale* __restrict__ scale, QuantCfg cfg,
                                                     int8_t* __restrict__ q_fold, int64_t ld_fold,
                                                     int8_t* __restrict__ q_t, int64_t ld_t,
                                                     const int32_t* __restrict__ desc, int64_t ext_base,
                                                     PadGrid pg, int tiled) {
    constexpr int QD = TC / 4;            // channel quads per tile
    constexpr int RQ = kBlock / QD;       // row quads per pass
    constexpr int RP = 4 * RQ;            // rows per pass
    constexpr int PASSES = kTR / RP;
    constexpr int TW = kTR / 4 + 1;       // LDS words per channel row (padded)
    __shared__ uint32_t tq[TC * TW];
    const int tid = threadIdx.x, cq = tid % QD, rq = tid / QD;
    const int64_t ctiles = (C + TC - 1) / TC, rtiles = (M + kTR - 1) / kTR;

    const sq_scale sc = *scale;
    const bool zero = sc.flags != 0u;
    const float Qf = (float)cfg.Q;
    // C a multiple of 8: the channel quads 2k and 2k + 1 of a row share one
    // Philox block; the two lanes (adjacent) each run it for two of their four
    // rows and swap the halves the other needs
    const bool sr_pair = SR && ((C & 7) == 0);
    const int par = cq & 1;

    for (int64_t tile = blockIdx.x; tile < ctiles * rtiles; tile += gridDim.x) {
        const int64_t ct = tile % ctiles, rt = tile / ctiles;
        const int64_t c0 = ct * TC + 4 * cq, m_tile = rt * kTR;
        const bool full_vec = VEC == 4 && c0 + 4 <= C;
        float s[4];
        int t[4], pos[4];   // fold: code << t in main column c (pos < 0) or appended column pos
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int64_t c = c0 + j;
            const int g = (group && c < C) ? (int)group[c] : 0;
            s[j] = __fmul_rn(sc.inv, pow2f(g));
            const int d = (desc && c < C) ? desc[c] : 0;
            t[j] = d & 15;
            pos[j] = (d >> 4) - 1;
        }
        // passes unrolled, except under stochastic rounding (its Philox words
        // make an unrolled body too large for the compiler)
        constexpr int kUnrollPasses = SR ? 1 : PASSES;
#pragma unroll kUnrollPasses
        for (int p = 0; p < PASSES; ++p) {
            const int r0 = p * RP + 4 * rq;   // first of this thread's rows within the tile
            float v[4][4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int64_t m = m_tile + r0 + i;
                v[i][0] = v[i][1] = v[i][2] = v[i][3] = 0.f;
                if (m < M && c0 < C) {
                    if (full_vec) {
                        const float4 f = *reinterpret_cast<const float4*>(x + m * ld + c0);
                        v[i][0] = f.x; v[i][1] = f.y; v[i][2] = f.z; v[i][3] = f.w;
                    } else {
#pragma unroll
                        for (int j = 0; j < 4; ++j)
                            if (c0 + j < C) v[i][j] = x[m * ld + c0 + j];
                    }
                }
            }
            uint32_t colw[4] = {0u, 0u, 0u, 0u};   // channel j: rows r0 .. r0 + 3, little-endian
            // this lane's two Philox words (its quad's 4 halves) for each of its 4 rows
            uint32_t sw[4][2];
            if (SR && sr_pair) {
                const int64_t cpair = c0 & ~(int64_t)7;
                uint32_t mine[2][4];
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    const int64_t m = m_tile + r0 + 2 * par + h;
                    const U4 w = philox_block((uint64_t)(m * C + cpair) >> 3, cfg);
                    mine[h][0] = w.x; mine[h][1] = w.y; mine[h][2] = w.z; mine[h][3] = w.w;
                }
                // own rows 2 par + h: words 2 par, 2 par + 1; the partner's rows
                // come through a lane swap of the words 2 par, 2 par + 1 it computed
#pragma unroll
                for (int h = 0; h < 2; ++h)
#pragma unroll
                    for (int k = 0; k < 2; ++k) {
                        const uint32_t give = mine[h][2 * (1 - par) + k];
                        const uint32_t got = (uint32_t)__shfl_xor((int)give, 1, 64);
                        sw[2 * par + h][k] = mine[h][2 * par + k];
                        sw[2 * (1 - par) + h][k] = got;
                    }
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int64_t m = m_tile + r0 + i;
                uint32_t u[4] = {0u, 0u, 0u, 0u};
                if (SR && m < M && c0 < C) {
                    if (sr_pair) {
#pragma unroll
                        for (int j = 0; j < 4; ++j) u[j] = (sw[i][j >> 1] >> (16 * (j & 1))) & 0xFFFFu;
                    } else {
#pragma unroll
                        for (int j = 0; j < 4; ++j)
                            if (c0 + j < C) u[j] = sr_uniform16((uint64_t)(m * C + c0 + j), cfg);
                    }
                }
                int code[4];
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    code[j] = (zero || m >= M || c0 + j >= C) ? 0 : quant_one<SR>(v[i][j], s[j], Qf, u[j]);
                    colw[j] |= (uint32_t)(uint8_t)code[j] << (8 * i);
                }
                if (q_fold && m < M && c0 < C && !tiled) {
                    int8_t* row = q_fold + m * ld_fold;
                    uint32_t word = 0u;
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        const uint32_t f = (uint32_t)(uint8_t)(code[j] * (1 << t[j]));
                        if (pos[j] < 0) word |= f << (8 * j);
                        else if (c0 + j < C) row[ext_base + pos[j]] = (int8_t)f;
                    }
                    if (c0 + 4 <= C) {
                        *reinterpret_cast<uint32_t*>(row + c0) = word;
                    } else {
#pragma unroll
                        for (int j = 0; j < 4; ++j)
                            if (c0 + j < C) row[c0 + j] = (int8_t)(word >> (8 * j));
                    }
                } else if (q_fold && m < M && c0 < ext_base && tiled) {
                    // tile-major: the quad's 4 bytes are contiguous; codes of
                    // channels >= C (K padding of the main columns) are 0
                    uint32_t word = 0u;
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        const uint32_t f = (uint32_t)(uint8_t)(code[j] * (1 << t[j]));
                        if (pos[j] < 0) word |= f << (8 * j);
                        else if (c0 + j < C) q_fold[tiled_off(m, ext_base + pos[j], ld_fold)] = (int8_t)f;
                    }
                    *reinterpret_cast<uint32_t*>(q_fold + tiled_off(m, c0, ld_fold)) = word;
                }
            }
            if (q_t) {
#pragma unroll
                for (int j = 0; j < 4; ++j) tq[(4 * cq + j) * TW + r0 / 4] = colw[j];
            }
        }
        if (q_t) {
            __syncthreads();
            // channel row ch of the tile: kTR bytes = kTR / 16 chunks of 16
            // bytes; this thread writes chunk `part` of the channel rows ch0,
            // ch0 + kBlock / CPR, ..., so its pixels (and their place on a
            // padded grid) are the same for every row it writes
            constexpr int CPR = kTR / 16;
            static_assert((TC * CPR) % kBlock == 0 && kBlock % CPR == 0, "whole passes over the tile");
            const int part = tid % CPR, ch0 = tid / CPR;
            const int64_t m = m_tile + 16 * part;
            // padded pixel grid: pixel m = (n, oh, ow) at n HpWp + oh Wp + ow;
            // 16 pixels in one image row as one 16-byte store, else two 8-byte
            // halves (which never cross an image row when Wo % 8 == 0)
            const bool grid_fast = pg.Wo && pg.Wo % 8 == 0 && (pg.off & 7) == 0 && m + 16 <= M;
            int64_t d0 = 0, d1 = 0;
            bool whole = false;
            if (grid_fast) {
                const uint32_t m0 = (uint32_t)m;
                const uint32_t n = m0 / pg.HoWo, rem = m0 - n * pg.HoWo, oh = rem / pg.Wo;
                const uint32_t ow = rem - oh * pg.Wo;
                d0 = (int64_t)n * pg.HpWp + (int64_t)oh * pg.Wp + ow + pg.off;
                whole = ow + 16 <= pg.Wo && (d0 & 15) == 0;
                const uint32_t mh = m0 + 8;
                const uint32_t n1 = mh / pg.HoWo, rem1 = mh - n1 * pg.HoWo, oh1 = rem1 / pg.Wo;
                d1 = (int64_t)n1 * pg.HpWp + (int64_t)oh1 * pg.Wp + (rem1 - oh1 * pg.Wo) + pg.off;
            }
            // kept rolled: unrolled, the 64-channel tiles measured 1.5 us slower
#pragma unroll 1
            for (int it = 0; it < TC * CPR / kBlock; ++it) {
                const int ch = ch0 + it * (kBlock / CPR);
                const int64_t c = ct * TC + ch;
                if (tiled) {
                    // tile-major: 16 codes of a channel row are contiguous;
                    // rows past M hold 0 (K padding up to a multiple of 64)
                    if (c < C && m < round_up(M, 64)) {
                        const uint32_t* src = &tq[ch * TW + 4 * part];
                        *reinterpret_cast<uint4*>(q_t + tiled_off(c, m, ld_t)) =
                            make_uint4(src[0], src[1], src[2], src[3]);
                    }
                    continue;
                }
                if (c >= C || m >= M) continue;
                const uint32_t* src = &tq[ch * TW + 4 * part];
                int8_t* row = q_t + c * ld_t;
                if (grid_fast) {
                    if (whole) {
                        *reinterpret_cast<uint4*>(row + d0) = make_uint4(src[0], src[1], src[2], src[3]);
                    } else {
                        *reinterpret_cast<uint2*>(row + d0) = make_uint2(src[0], src[1]);
                        *reinterpret_cast<uint2*>(row + d1) = make_uint2(src[2], src[3]);
                    }
                } else if (pg.Wo) {
                    for (int i = 0; i < 16 && m + i < M; ++i) {
                        const uint32_t mi = (uint32_t)(m + i);
                        const uint32_t n = mi / pg.HoWo, rem = mi - n * pg.HoWo, oh = rem / pg.Wo;
                        const uint32_t ow = rem - oh * pg.Wo;
                        row[(int64_t)n * pg.HpWp + (int64_t)oh * pg.Wp + ow + pg.off] =
                            (int8_t)(src[i / 4] >> (8 * (i % 4)));
                    }
                } else if (m + 16 <= M) {
                    *reinterpret_cast<uint4*>(row + m) = make_uint4(src[0], src[1], src[2], src[3]);
                } else {
                    for (int i = 0; i < (int)(M - m); ++i) row[m + i] = (int8_t)(src[i / 4] >> (8 * (i % 4)));
                }
            }
            __syncthreads();
        }
    }
}

// ---------------------------------------------------------------------------
// Quantize, 8-channel form: the same codes and layouts as k_quantize for
// 16-byte aligned inputs with C a multiple of 8 (no padded pixel grid).  A
// thread quantizes 8 consecutive channels of 4 consecutive rows; the 8
// elements of a row form one Philox block (indices m C + c0 .. + 7 with c0 a
// multiple of 8), so each thread draws its own uniforms and no lane exchange
// is needed.  Tiles of 128 rows x 64 channels; the codes of a tile are
// transposed through LDS (4 rows per word) for q_t.  Each row's 8
// shift-folded codes leave as one 8-byte store.
// ---------------------------------------------------------------------------
template <bool SR, bool TL>
__global__ __launch_bounds__(kBlock) void k_quantize8(const float* __restrict__ x, int64_t M, int64_t C, int64_t ld,
                                                      const uint8_t* __restrict__ group,
                                                      const sq_scale* __restrict__ scale, QuantCfg cfg,
                                                      int8_t* __restrict__ q_fold, int64_t ld_fold,
                                                      int8_t* __restrict__ q_t, int64_t ld_t,
                                                      const int32_t* __restrict__ desc, int64_t ext_base,
                                                      int meta_vec, PadGrid pg) {
    constexpr int TR = 128, TC = 64, TW = TR / 4 + 1;   // LDS words per channel row (padded)
    __shared__ uint32_t tq[TC * TW];
    const int tid = threadIdx.x, g8 = tid & 7, rq = tid >> 3;
    const int64_t ctiles = (C + TC - 1) / TC, rtiles = (M + TR - 1) / TR;
    const sq_scale sc = *scale;
    const bool zero = sc.flags != 0u;
    const float Qf = (float)cfg.Q;
    // q_t rows written: the codes, and with the tile-major layout their zero
    // padding up to a multiple of 64
    const int64_t m_t = TL ? round_up(M, 64) : M;
    auto at_fold = [&](int64_t m, int64_t k) { return TL ? tiled_off(m, k, ld_fold) : m * ld_fold + k; };

    for (int64_t tile = blockIdx.x; tile < ctiles * rtiles; tile += gridDim.x) {
        const int64_t ct = tile % ctiles, rt = tile / ctiles;
        const int64_t c0 = ct * TC + 8 * g8, m0 = rt * TR + 4 * rq;
        const bool cin = c0 < C;   // C % 8 == 0: all 8 channels or none
        // per channel: scale, fold factor 2^t in its main column (0 for an
        // appended channel, whose main column holds 0), appended position
        uint32_t gw[2] = {0u, 0u};
        int32_t dw[8] = {0, 0, 0, 0, 0, 0, 0, 0};
        if (cin) {
            if (meta_vec) {
                if (group) {
                    const uint2 g2 = *reinterpret_cast<const uint2*>(group + c0);
                    gw[0] = g2.x; gw[1] = g2.y;
                }
                if (desc) {
                    const int4 d0 = *reinterpret_cast<const int4*>(desc + c0);
                    const int4 d1 = *reinterpret_cast<const int4*>(desc + c0 + 4);
                    dw[0] = d0.x; dw[1] = d0.y; dw[2] = d0.z; dw[3] = d0.w;
                    dw[4] = d1.x; dw[5] = d1.y; dw[6] = d1.z; dw[7] = d1.w;
                }
            } else {
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    if (group) gw[j >> 2] |= (uint32_t)group[c0 + j] << (8 * (j & 3));
                    if (desc) dw[j] = desc[c0 + j];
                }
            }
        }
        float s[8], tf[8];
        bool any_ext = false;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            s[j] = __fmul_rn(sc.inv, pow2f((int)((gw[j >> 2] >> (8 * (j & 3))) & 0xFFu)));
            const int pos = (dw[j] >> 4) - 1;
            tf[j] = pos < 0 ? pow2f(dw[j] & 15) : 0.0f;
            any_ext |= pos >= 0;
        }
        // the bytes below are built as code + 128 (unsigned), then flipped
        // back to two's complement with one xor per word
        uint32_t colw[8] = {0u, 0u, 0u, 0u, 0u, 0u, 0u, 0u};   // channel j, rows m0 .. m0 + 3
        const bool rows_in = rt * TR + TR <= M;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int64_t m = m0 + i;
            const bool ok = cin && !zero && (rows_in || m < M);
            float v[8];
            if (ok) {
                const float4 a = *reinterpret_cast<const float4*>(x + m * ld + c0);
                const float4 b = *reinterpret_cast<const float4*>(x + m * ld + c0 + 4);
                v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w; v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
            } else {
#pragma unroll
                for (int j = 0; j < 8; ++j) v[j] = 0.f;
            }
            U4 w{0u, 0u, 0u, 0u};
            if (SR && ok) w = philox_block((uint64_t)(m * C + c0) >> 3, cfg);
            uint32_t lo = 0u, hi = 0u;
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const uint32_t u = SR ? (pick(w, j >> 1) >> (16 * (j & 1))) & 0xFFFFu : 0u;
                const float q = ok ? quant_onef<SR>(v[j], s[j], Qf, u) : 0.0f;
                colw[j] = __builtin_amdgcn_cvt_pk_u8_f32(__fadd_rn(q, 128.0f), i, colw[j]);
                const float qf = __fadd_rn(__fmul_rn(q, tf[j]), 128.0f);
                if (j < 4) lo = __builtin_amdgcn_cvt_pk_u8_f32(qf, j, lo);
                else hi = __builtin_amdgcn_cvt_pk_u8_f32(qf, j - 4, hi);
            }
            if (q_fold && (rows_in || m < M)) {
                if (cin) {
                    if (any_ext) {
#pragma unroll
                        for (int j = 0; j < 8; ++j) {
                            const int pos = (dw[j] >> 4) - 1;
                            if (pos >= 0) {
                                const int code = (int)((colw[j] >> (8 * i)) & 0xFFu) - 128;
                                q_fold[at_fold(m, ext_base + pos)] = (int8_t)(code * (1 << (dw[j] & 15)));
                            }
                        }
                    }
                    *reinterpret_cast<uint2*>(q_fold + at_fold(m, c0)) = make_uint2(lo ^ 0x80808080u, hi ^ 0x80808080u);
                } else if (TL && c0 < ext_base) {
                    // K padding of the main columns
                    *reinterpret_cast<uint2*>(q_fold + at_fold(m, c0)) = make_uint2(0u, 0u);
                }
            }
        }
        if (q_t) {
#pragma unroll
            for (int j = 0; j < 8; ++j) tq[(8 * g8 + j) * TW + rq] = colw[j] ^ 0x80808080u;
            __syncthreads();
            // channel row ch of the tile, rows 32 part .. + 31 (two 16-byte chunks)
            const int ch = tid >> 2, part = tid & 3;
            const int64_t c = ct * TC + ch, mm = rt * TR + 32 * part;
            if (c < C && mm < m_t) {
                const uint32_t* src = &tq[ch * TW + 8 * part];
                const uint4 a = make_uint4(src[0], src[1], src[2], src[3]);
                const uint4 b = make_uint4(src[4], src[5], src[6], src[7]);
                if (TL) {
                    *reinterpret_cast<uint4*>(q_t + tiled_off(c, mm, ld_t)) = a;
                    *reinterpret_cast<uint4*>(q_t + tiled_off(c, mm + 16, ld_t)) = b;
                } else if (pg.Wo && (pg.off & 7) != 0) {
                    // padded pixel grid at an offset that is not a multiple of 8
                    // (a conv input: pixel (n, ih, iw) at n HpWp + (ih + PH) Wp +
                    // iw + PW).  A group of 8 pixels then straddles two aligned
                    // 8-byte words; each word that holds codes is written whole,
                    // once, by the group whose last codes open it: its bytes
                    // are that group's tail and the next group's head, or zeros
                    // where the image row ends.  A row's first group also writes
                    // the word before it (zeros, then its head).  The head of the
                    // next tile's first group is quantized again here from x
                    // (per-tensor codes, round to nearest: the same value).
                    const int sa = 8 * (int)(pg.off & 7);
                    const uint32_t m0 = (uint32_t)mm;
                    uint32_t n = m0 / pg.HoWo, rem = m0 - n * pg.HoWo, oh = rem / pg.Wo, ow = rem - oh * pg.Wo;
                    int8_t* row = q_t + c * ld_t;
                    auto word = [&](int w) {   // codes of 8 pixels: tile word pair w of this channel row
                        return (uint64_t)tq[ch * TW + 2 * w] | ((uint64_t)tq[ch * TW + 2 * w + 1] << 32);
                    };
#pragma unroll
                    for (int g = 0; g < 4; ++g) {
                        if (mm + 8 * g < M) {
                            const uint64_t cur = word(4 * part + g);
                            uint64_t nxt = 0;
                            if (ow + 8 < pg.Wo) {
                                if (part < 3 || g < 3) {
                                    nxt = word(4 * part + g + 1);
                                } else if (!zero) {
                                    const int64_t mn = mm + 8 * g + 8;
                                    const float sn = __fmul_rn(sc.inv, pow2f(0));
#pragma unroll
                                    for (int k = 0; k < 8; ++k)
                                        nxt |= (uint64_t)(uint8_t)quant_one<false>(x[(mn + k) * ld + c], sn, Qf, 0u)
                                               << (8 * k);
                                }
                            }
                            const int64_t d = (int64_t)n * pg.HpWp + (int64_t)oh * pg.Wp + ow + pg.off - sa / 8;
                            if (ow == 0) *reinterpret_cast<uint64_t*>(row + d) = cur << sa;
                            *reinterpret_cast<uint64_t*>(row + d + 8) = (cur >> (64 - sa)) | (nxt << sa);
                        }
                        ow += 8;
                        if (ow == pg.Wo) {
                            ow = 0;
                            if (++oh * pg.Wo == pg.HoWo) {
                                oh = 0;
                                ++n;
                            }
                        }
                    }
                } else if (pg.Wo) {
                    // padded pixel grid (Wo % 8 == 0, offset a multiple of 8):
                    // pixel m = (n, oh, ow) at n HpWp + oh Wp + ow + off; the 4
                    // groups of 8 pixels never cross an image row, so each is one
                    // 8-byte store (16-byte stores of aligned pairs, behind a
                    // branch, measured slower)
                    const uint32_t m0 = (uint32_t)mm;
                    uint32_t n = m0 / pg.HoWo, rem = m0 - n * pg.HoWo, oh = rem / pg.Wo, ow = rem - oh * pg.Wo;
                    int8_t* row = q_t + c * ld_t + pg.off;
#pragma unroll
                    for (int g = 0; g < 4; ++g) {
                        if (mm + 8 * g < M)
                            *reinterpret_cast<uint2*>(row + (int64_t)n * pg.HpWp + (int64_t)oh * pg.Wp + ow) =
                                make_uint2(src[2 * g], src[2 * g + 1]);
                        ow += 8;
                        if (ow == pg.Wo) {
                            ow = 0;
                            if (++oh * pg.Wo == pg.HoWo) {
                                oh = 0;
                                ++n;
                            }
                        }
                    }
                } else if (mm + 32 <= M) {
                    *reinterpret_cast<uint4*>(q_t + c * ld_t + mm) = a;
                    *reinterpret_cast<uint4*>(q_t + c * ld_t + mm + 16) = b;
                } else {
                    for (int r = 0; r < (int)(M - mm); ++r)
                        q_t[c * ld_t + mm + r] = (int8_t)(src[r / 4] >> (8 * (r % 4)));
                }
            }
            __syncthreads();
        }
    }
}

}  // namespace

// ---------------------------------------------------------------------------
// Per-channel quantization of a weight matrix (one scale per row or per
// column; the forward pass quantizes weights per output channel and loss
// propagation per input channel, Sec. 5.1).  Weights are quantized once per
// step, off the backward hot path, so these kernels are plain.
// ---------------------------------------------------------------------------
// column scales from the colmax slab maxima
__global__ void k_channel_scales_cols(const uint32_t* __restrict__ partial, int64_t S, int64_t C, int Q,
                                      sq_scale* __restrict__ scales) {
    for (int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; c < C; c += (int64_t)gridDim.x * blockDim.x)
        scales[c] = make_scale(reduce_slabs(partial, S, C, c), (float)Q);
}

// row scales: one wave per row
__global__ void k_channel_scales_rows(const float* __restrict__ x, int64_t rows, int64_t cols, int64_t ld, int Q,
                                      sq_scale* __restrict__ scales) {
    const int lane = threadIdx.x & 63;
    const int64_t wave = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
    const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) >> 6;
    for (int64_t r = wave; r < rows; r += nwaves) {
        uint32_t m = 0u;
        for (int64_t c = lane; c < cols; c += 64) m = max(m, absbits(x[r * ld + c]));
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) m = max(m, (uint32_t)__shfl_xor((int)m, o, 64));
        if (lane == 0) scales[r] = make_scale(m, (float)Q);
    }
}

// code = clamp(rint(fl(x * inv_ch)), -Q, Q), 0 in a flagged channel
__global__ void k_quantize_channels(const float* __restrict__ x, int64_t rows, int64_t cols, int64_t ld, int axis,
                                    const sq_scale* __restrict__ scales, int Q, int8_t* __restrict__ q, int64_t ld_q,
                                    int transpose) {
    const float Qf = (float)Q;
    const int64_t n = rows * cols;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n; e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t i = transpose ? e % rows : e / cols, j = transpose ? e / rows : e % cols;
        const sq_scale sc = scales[axis == 0 ? i : j];
        int code = 0;
        if (sc.flags == 0u) code = (int)fminf(fmaxf(rintf(__fmul_rn(x[i * ld + j], sc.inv)), -Qf), Qf);
        if (transpose) q[j * ld_q + i] = (int8_t)code;
        else q[i * ld_q + j] = (int8_t)code;
    }
}

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
    // about 512 blocks (two per CU), each slab at least 8 row passes deep:
    // fewer slab maxima for the finalize to reduce (1024 blocks cost the
    // 64-channel conv gradient 3 us more, measured)
    int64_t slabs = std::max<int64_t>(1, 512 / p.chunks);
    const int64_t min_rows = 8 * (int64_t)nrl;
    slabs = std::min<int64_t>(slabs, std::max<int64_t>(1, (M + min_rows - 1) / min_rows));
    slabs = std::min<int64_t>(slabs, 65535);
    p.rows_per_slab = std::max<int64_t>(1, (M + slabs - 1) / slabs);
    p.slabs = M > 0 ? (M + p.rows_per_slab - 1) / p.rows_per_slab : 0;
    return p;
}

int64_t colmax_reduce_blocks(int64_t C) { return C >= kFinThreads ? (C + kRedThreads - 1) / kRedThreads : 0; }

int64_t colmax_workspace_words(int64_t M, int64_t C) {
    // worst case over both vector widths: slab maxima, channel ranges, the
    // second level's block maxima and shift counts, the abs-max blocks' maxima
    int64_t w = 0;
    for (const bool vec : {true, false}) {
        const ColmaxPlan p = colmax_plan(M, C, vec);
        w = std::max(w, p.slabs * C + C + (1 + kMaxRegions) * colmax_reduce_blocks(C) + p.chunks * p.slabs);
    }
    return w;
}

hipError_t launch_colmax(const float* x, int64_t M, int64_t C, int64_t ld, uint32_t* partial, int64_t* slabs,
                         hipStream_t s, uint32_t* block_max, int64_t* n_block_max) {
    *slabs = 0;
    if (n_block_max) *n_block_max = 0;
    if (M <= 0 || C <= 0) return hipSuccess;
    const bool vec = ((ld & 3) == 0) && ((reinterpret_cast<uintptr_t>(x) & 15) == 0);
    const ColmaxPlan p = colmax_plan(M, C, vec);
    *slabs = p.slabs;
    if (n_block_max) *n_block_max = p.chunks * p.slabs;
    dim3 grid((unsigned)p.chunks, (unsigned)p.slabs);
    // A tensor larger than the 256 MB last-level cache cannot stay there for
    // the quantize pass's second read; streaming it through without
    // allocating leaves other lines in place, in particular dirty ones, which
    // would otherwise be written back during this read (large linear layer,
    // 360 MB: this pass 78.7 -> 55.6 us, the step 741 -> 730 us).  Smaller
    // tensors keep ordinary loads (their second read hits the cache).
    const bool nt = (uint64_t)M * (uint64_t)ld * sizeof(float) > kLastLevelCacheBytes;
    if (vec && nt)
        hipLaunchKernelGGL((k_colmax<4, true>), grid, dim3(kColThreads), 0, s, x, M, C, ld, p.tpr, p.rows_per_slab,
                           partial, block_max);
    else if (vec)
        hipLaunchKernelGGL((k_colmax<4, false>), grid, dim3(kColThreads), 0, s, x, M, C, ld, p.tpr, p.rows_per_slab,
                           partial, block_max);
    else
        hipLaunchKernelGGL((k_colmax<1, false>), grid, dim3(kColThreads), 0, s, x, M, C, ld, p.tpr, p.rows_per_slab,
                           partial, block_max);
    return hipGetLastError();
}

static hipError_t launch_reduce(const uint32_t* partial, int64_t slabs, int64_t C, uint32_t* rbits, uint32_t* bmax,
                                hipStream_t s) {
    const int64_t nb = colmax_reduce_blocks(C);
    if (nb == 0) return hipSuccess;
    hipLaunchKernelGGL(k_colmax_reduce, dim3((unsigned)nb), dim3(kRedThreads * kRedLanes), 0, s, partial, slabs, C,
                       rbits, bmax);
    return hipGetLastError();
}

hipError_t launch_finalize_grad(const uint32_t* partial, int64_t slabs, int64_t C, const QuantCfg& cfg,
                                uint32_t* rbits, uint8_t* group, sq_scale* scale, int32_t* layout,
                                int64_t ext_max, hipStream_t s) {
    uint32_t* bmax = rbits + C;
    const hipError_t e = launch_reduce(partial, slabs, C, rbits, bmax, s);
    if (e != hipSuccess) return e;
    const int64_t nb = colmax_reduce_blocks(C);
    if (nb > 0) {
        // many channels: groups and placement spread over nb blocks
        int32_t* hist = reinterpret_cast<int32_t*>(bmax + nb);
        hipLaunchKernelGGL(k_final_groups, dim3((unsigned)nb), dim3(kRedThreads), 0, s, rbits, bmax, nb, C, cfg, group,
                           scale, layout, ext_max, hist);
        if (ext_max > 0)
            hipLaunchKernelGGL(k_final_place, dim3((unsigned)nb), dim3(kRedThreads), 0, s, group, hist, nb, C, cfg,
                               layout, ext_max);
        return hipGetLastError();
    }
    hipLaunchKernelGGL(k_finalize_grad, dim3(1), dim3(kFinThreads), 0, s, partial, slabs, C, cfg, rbits, bmax, nb, group,
                       scale, layout, ext_max);
    return hipGetLastError();
}

hipError_t launch_colmax_finalize_grad(const float* x, int64_t M, int64_t C, int64_t ld, const QuantCfg& cfg,
                                       uint32_t* ws, uint8_t* group, sq_scale* scale, int32_t* layout,
                                       int64_t ext_max, hipStream_t s) {
    const int64_t nb = colmax_reduce_blocks(C);
    if (nb == 0 || M <= 0) {
        int64_t slabs = 0;
        hipError_t e = launch_colmax(x, M, C, ld, ws, &slabs, s);
        if (e != hipSuccess) return e;
        return launch_finalize_grad(ws, slabs, C, cfg, ws + slabs * C, group, scale, layout, ext_max, s);
    }
    // many channels: the abs-max pass also leaves its blocks' maxima, and the
    // group kernel reduces the slab maxima itself (no k_colmax_reduce)
    const ColmaxPlan p = colmax_plan(M, C, ((ld & 3) == 0) && ((reinterpret_cast<uintptr_t>(x) & 15) == 0));
    uint32_t* rbits = ws + p.slabs * C;
    int32_t* hist = reinterpret_cast<int32_t*>(rbits + C + nb);
    uint32_t* bm = rbits + C + (1 + kMaxRegions) * nb;
    int64_t slabs = 0, nbm = 0;
    hipError_t e = launch_colmax(x, M, C, ld, ws, &slabs, s, bm, &nbm);
    if (e != hipSuccess) return e;
    if (slabs != p.slabs) return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_final_groups_slabs, dim3((unsigned)nb), dim3(kRedThreads * kRedLanes), 0, s, ws, slabs, bm,
                       nbm, C, cfg, group, scale, layout, ext_max, hist);
    if (ext_max > 0)
        hipLaunchKernelGGL(k_final_place, dim3((unsigned)nb), dim3(kRedThreads), 0, s, group, hist, nb, C, cfg,
                           layout, ext_max);
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

constexpr int64_t kQuantMaxBlocks = 4096;   // grid-stride beyond this
constexpr int64_t kQuantMinTiles = 1024;    // four blocks per CU

hipError_t launch_quantize(const float* x, int64_t M, int64_t C, int64_t ld, const uint8_t* group,
                           const sq_scale* scale, const QuantCfg& cfg, int8_t* q_fold, int64_t ld_fold,
                           int8_t* q_t, int64_t ld_t, const int32_t* desc, hipStream_t s, PadGrid pg, bool tiled) {
    if (M <= 0 || C <= 0) return hipSuccess;
    if (tiled && (pg.Wo || (q_fold && ld_fold % 64) || (q_t && ld_t % 64))) return hipErrorInvalidValue;
    const bool vec = ((ld & 3) == 0) && ((reinterpret_cast<uintptr_t>(x) & 15) == 0);
    const bool sr = cfg.round_mode == SQ_ROUND_STOCHASTIC;
    // 128 x 128 tiles where the tensor gives enough of them to fill the chip
    auto n_tiles = [&](int64_t tc, int64_t tr) { return ((C + tc - 1) / tc) * ((M + tr - 1) / tr); };
    // stochastic rounding keeps the 64-channel tile: the Philox words of a
    // 128-channel tile's passes need about 180 registers (2 waves per SIMD)
    int tc = (C <= 64 || sr) ? 64 : 128, tr = 128;
    if (n_tiles(tc, tr) < kQuantMinTiles) tr = 64;
    if (n_tiles(tc, tr) < kQuantMinTiles) tc = 64;
    const int64_t eb = fold_ext_base(C);
    // a grid offset that is not a multiple of 8 takes the 8-channel kernel
    // only for per-tensor round-to-nearest codes (it quantizes a few codes of
    // the next tile again), else the byte stores of k_quantize
    const bool grid8 = !pg.Wo || (pg.Wo % 8 == 0 && !tiled &&
                                  ((pg.off & 7) == 0 || (!sr && !group && !desc)));
    if (vec && C % 8 == 0 && grid8) {
        // 8-channel form: one Philox block per thread and row; the groups
        // (8 bytes) and descriptors (2 x 16 bytes) of a thread's channels
        // load as vectors when aligned
        const int mv = ((reinterpret_cast<uintptr_t>(group) & 7) == 0 && (reinterpret_cast<uintptr_t>(desc) & 15) == 0);
        const dim3 g8((unsigned)std::min<int64_t>(((C + 63) / 64) * ((M + 127) / 128), kQuantMaxBlocks));
        if (sr && tiled) hipLaunchKernelGGL((k_quantize8<true, true>), g8, dim3(kBlock), 0, s, x, M, C, ld, group, scale,
                                            cfg, q_fold, ld_fold, q_t, ld_t, desc, eb, mv, pg);
        else if (sr) hipLaunchKernelGGL((k_quantize8<true, false>), g8, dim3(kBlock), 0, s, x, M, C, ld, group, scale,
                                        cfg, q_fold, ld_fold, q_t, ld_t, desc, eb, mv, pg);
        else if (tiled) hipLaunchKernelGGL((k_quantize8<false, true>), g8, dim3(kBlock), 0, s, x, M, C, ld, group,
                                           scale, cfg, q_fold, ld_fold, q_t, ld_t, desc, eb, mv, pg);
        else hipLaunchKernelGGL((k_quantize8<false, false>), g8, dim3(kBlock), 0, s, x, M, C, ld, group, scale, cfg,
                                q_fold, ld_fold, q_t, ld_t, desc, eb, mv, pg);
        return hipGetLastError();
    }
    const dim3 grid((unsigned)std::min<int64_t>(n_tiles(tc, tr), kQuantMaxBlocks));
#define SQ_LAUNCH_QUANT(TC, TR)                                                                                  \
    do {                                                                                                         \
        if (vec && sr) hipLaunchKernelGGL((k_quantize<TC, TR, 4, true>), grid, dim3(kBlock), 0, s, x, M, C, ld,  \
                                          group, scale, cfg, q_fold, ld_fold, q_t, ld_t, desc, eb, pg, (int)tiled);              \
        else if (vec) hipLaunchKernelGGL((k_quantize<TC, TR, 4, false>), grid, dim3(kBlock), 0, s, x, M, C, ld,  \
                                         group, scale, cfg, q_fold, ld_fold, q_t, ld_t, desc, eb, pg, (int)tiled);               \
        else if (sr) hipLaunchKernelGGL((k_quantize<TC, TR, 1, true>), grid, dim3(kBlock), 0, s, x, M, C, ld,    \
                                        group, scale, cfg, q_fold, ld_fold, q_t, ld_t, desc, eb, pg, (int)tiled);                \
        else hipLaunchKernelGGL((k_quantize<TC, TR, 1, false>), grid, dim3(kBlock), 0, s, x, M, C, ld, group,    \
                                scale, cfg, q_fold, ld_fold, q_t, ld_t, desc, eb, pg, (int)tiled);                               \
    } while (0)
    if (tc == 64 && tr == 64) SQ_LAUNCH_QUANT(64, 64);
    else if (tc == 64) SQ_LAUNCH_QUANT(64, 128);
    else if (tr == 64) SQ_LAUNCH_QUANT(128, 64);
    else SQ_LAUNCH_QUANT(128, 128);
#undef SQ_LAUNCH_QUANT
    return hipGetLastError();
}

hipError_t launch_quantize_channels(const float* x, int64_t rows, int64_t cols, int64_t ld, int bits, int axis,
                                   int transpose, int8_t* q, int64_t ld_q, sq_scale* scales, uint32_t* partial,
                                   hipStream_t s) {
    if (rows <= 0 || cols <= 0) return hipSuccess;
    const int Q = (1 << (bits - 1)) - 1;
    if (axis == 1) {
        int64_t slabs = 0;
        const hipError_t e = launch_colmax(x, rows, cols, ld, partial, &slabs, s);
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(k_channel_scales_cols, dim3((unsigned)std::min<int64_t>((cols + 255) / 256, 4096)), dim3(256),
                           0, s, partial, slabs, cols, Q, scales);
    } else {
        hipLaunchKernelGGL(k_channel_scales_rows, dim3((unsigned)std::min<int64_t>((rows + 3) / 4, 8192)), dim3(256), 0,
                           s, x, rows, cols, ld, Q, scales);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_quantize_channels, dim3((unsigned)std::min<int64_t>((rows * cols + 255) / 256, 16384)),
                       dim3(256), 0, s, x, rows, cols, ld, axis, scales, Q, q, ld_q, transpose);
    return hipGetLastError();
}

}  // namespace sq
