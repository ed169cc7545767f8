// Integer GEMMs of the ShiftQuant backward pass for gfx950.
//
// One kernel template serves both products as C[i, j] = sum_k A[i, k] * B[j, k]
// with both operands K-contiguous int8:
//   dgrad: A = shift-folded gradient codes [M, C_out(+appended)],
//          B = W^T codes [C_in, C_out]              -> dX [M, C_in]
//   wgrad: A = transposed gradient codes [C_out, M],
//          B = X^T codes [C_in, M]                   -> dW [C_out, C_in]
// int32 accumulation on the matrix cores (v_mfma_i32_32x32x32_i8 or
// v_mfma_i32_16x16x64_i8), block tiles of WM x WN waves, K tiles of BK bytes
// double-buffered in LDS (rows padded by 16 bytes, which keeps the 16-byte
// fragment reads free of bank conflicts), and the dequantization of
// Eq. "dq_mm_f" fused into the epilogue.
//
// ShiftMM (Sec. 3.2) shifts every product by the shift of its inner index
// before accumulation.  The quantizer stores each channel's code already
// shifted within a window of shifts that fits int8; channels of the windows
// other than the main one sit in appended K columns.  This kernel visits the
// windows in descending order and shifts the accumulator left by the
// difference of window bases at each window start and by the last base at the
// end (Horner's rule), so the result equals sum_c code * w << (N_G - 1 - g_c)
// exactly.
#include <algorithm>
#include <type_traits>

#include "sq_internal.h"

namespace sq {

namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

// Tile configuration: BM x BN outputs per block, WM x WN waves, BK bytes of
// K per LDS stage, MF = 32 (32x32x32 MFMA) or 16 (16x16x64 MFMA).
template <int BM_, int BN_, int BK_, int WM_, int WN_, int MF_>
struct TileCfg {
    static constexpr int BM = BM_, BN = BN_, BK = BK_, WM = WM_, WN = WN_, MF = MF_;
    static constexpr int kThreads = 64 * WM * WN;
    static constexpr int TM = BM / WM, TN = BN / WN;      // wave tile
    static constexpr int FM = TM / MF, FN = TN / MF;      // MFMA blocks per wave
    static constexpr int KS = MF == 32 ? 32 : 64;         // K bytes per MFMA
    static constexpr int NACC = MF == 32 ? 16 : 4;        // int32 results per lane per MFMA
    static constexpr int LS = BK + 16;                    // LDS row stride in bytes
    static constexpr int CPR = BK / 16;                   // 16-byte chunks per row
    static constexpr int LA = BM * CPR / kThreads;        // chunks per thread per stage
    static constexpr int LB = BN * CPR / kThreads;
    static constexpr int kSmem = 2 * (BM + BN) * LS;
    static_assert(MF == 32 || MF == 16, "MFMA shape");
    static_assert(TM % MF == 0 && TN % MF == 0, "wave tile must hold whole MFMA blocks");
    static_assert(BK % KS == 0, "K tile must hold whole MFMA steps");
    static_assert(LA * kThreads == BM * CPR && LB * kThreads == BN * CPR, "even load split");
};

// The configurations the library launches.
using CfgSmall = TileCfg<128, 128, 64, 2, 2, 32>;   // small/skinny outputs, split-K
using CfgLarge = TileCfg<256, 256, 64, 4, 2, 16>;   // large products (matrix-core bound)

// Zero the bytes of a 16-byte chunk at positions >= nvalid (0 < nvalid < 16).
__device__ __forceinline__ uint4 mask_tail(uint4 v, int nvalid) {
    uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int keep = nvalid - 4 * i;
        const uint32_t m = keep >= 4 ? 0xFFFFFFFFu : (keep <= 0 ? 0u : ((1u << (8 * keep)) - 1u));
        w[i] &= m;
    }
    return make_uint4(w[0], w[1], w[2], w[3]);
}

// Blocks are dispatched to the 8 XCDs of the chip round-robin.  Give each XCD
// a contiguous range of tiles, then walk that range in groups of kGroupM tile
// rows so neighbouring blocks share operand panels in their XCD's L2.
constexpr int64_t kXcds = 8, kGroupM = 8;

__device__ __forceinline__ void tile_coords(int64_t b, int64_t tiles_m, int64_t tiles_n, int64_t& tm, int64_t& tn) {
    const int64_t nt = tiles_m * tiles_n;
    const int64_t x = b % kXcds, i = b / kXcds, q = nt / kXcds, r = nt % kXcds;
    const int64_t t = x * q + min(x, r) + i;
    const int64_t per_group = kGroupM * tiles_n;
    const int64_t first_m = (t / per_group) * kGroupM;
    const int64_t gsz = min(tiles_m - first_m, kGroupM);
    const int64_t w = t % per_group;
    tm = first_m + w % gsz;
    tn = w / gsz;
}

// Position in the K sequence of the implicit-im2col convolution: flat fold
// tile f, tap tau = r * KW + s of the window.
struct TapCursor {
    int f = 0, tau = 0, r = 0, s = 0;
    __device__ void next(int taps, int kw) {
        ++tau;
        if (++s == kw) { s = 0; ++r; }
        if (tau == taps) { tau = 0; r = 0; s = 0; ++f; }
    }
};

template <int MF>
struct Mfma;
template <>
struct Mfma<32> {
    typedef v16i acc_t;
    static __device__ __forceinline__ acc_t run(v4i a, v4i b, acc_t c) {
        return __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, c, 0, 0, 0);
    }
};
template <>
struct Mfma<16> {
    typedef v4i acc_t;
    static __device__ __forceinline__ acc_t run(v4i a, v4i b, acc_t c) {
        return __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, c, 0, 0, 0);
    }
};

// fp32 outputs of the weight gradient go out with nontemporal stores: the
// optimizer consumes dW, not the next kernel of the backward pass, so its lines
// should not sit dirty in the last-level cache, where the next reads of a
// gradient would first have to write them back (large linear layer: the next
// abs-max pass 95 -> 81 us, the step 761 -> 749 us)
typedef float v4f __attribute__((ext_vector_type(4)));
__device__ __forceinline__ void store_f4(float* dst, float a, float b, float c, float d, bool nt) {
    if (nt) __builtin_nontemporal_store(v4f{a, b, c, d}, reinterpret_cast<v4f*>(dst));
    else *reinterpret_cast<float4*>(dst) = make_float4(a, b, c, d);
}
__device__ __forceinline__ void store_f1(float* dst, float a, bool nt) {
    if (nt) __builtin_nontemporal_store(a, dst);
    else *dst = a;
}

// The dgrad's flat K sequence (fold layout in sq_internal.h): appended
// columns [0, H), the main segment, appended columns [H, D).  Tile t is
// appended when it lies outside the main segment's n_main tiles.
struct FoldView {
    int n_ext = 0, h_tiles = 0, fshift = 0, bk = 64;
    __device__ bool is_ext(int t, int n_main) const { return t < h_tiles || t >= h_tiles + n_main; }
    __device__ int64_t ext_col(int t, int n_main) const { return (int64_t)(t < h_tiles ? t : t - n_main) * bk; }
};

__device__ __forceinline__ FoldView fold_view(const GemmArgs& p, int bk) {
    FoldView v;
    v.bk = bk;
    if (p.layout) {
        v.n_ext = p.extA ? p.layout[kLayD] / bk : 0;
        v.h_tiles = p.layout[kLayH] / bk;
        v.fshift = p.layout[kLayF];
    }
    return v;
}

// Output-column scale of epi_mode 2 (one weight scale per output column):
// fl(fl(step_G * step_W[n]) * 2^-(N_G - 1)).
__device__ __forceinline__ float col_scale(const GemmArgs& p, float gstep, int64_t n) {
    return __fmul_rn(__fmul_rn(gstep, p.os[n].step), pow2f(-(p.num_groups - 1)));
}

// Region starts of the flat K sequence, in order; at each one the
// accumulator is shifted left by the base difference to the region before
// (Horner's rule).  The schedule is read once into registers, so the K loop
// itself touches no memory but its operand tiles.  col is the flat K column
// of the next start.
struct HornerSteps {
    int next = 1, nr = 1;
    int64_t col = INT64_MAX;
    uint32_t shifts = 0u;                                          // 4 bits per region
    int s1 = 0, s2 = 0, s3 = 0, s4 = 0, s5 = 0, s6 = 0, s7 = 0;   // region starts
    __device__ explicit HornerSteps(const GemmArgs& p) {
        static_assert(kMaxRegions == 8, "one start per region after the first");
        if (p.layout) {
            const int32_t* L = p.layout;
            nr = L[kLayNR];
            s1 = L[kLayStart + 1]; s2 = L[kLayStart + 2]; s3 = L[kLayStart + 3]; s4 = L[kLayStart + 4];
            s5 = L[kLayStart + 5]; s6 = L[kLayStart + 6]; s7 = L[kLayStart + 7];
#pragma unroll
            for (int r = 1; r < kMaxRegions; ++r) shifts |= (uint32_t)(L[kLayShift + r] & 15) << (4 * r);
            if (nr > 1) col = s1;
        }
    }
    // the starts are consumed in order: shift the queue instead of indexing
    // it (an indexed member would be placed in scratch memory)
    __device__ int advance() {
        const int sft = (int)((shifts >> (4 * next)) & 15u);
        ++next;
        col = next < nr ? (int64_t)s2 : INT64_MAX;
        s2 = s3; s3 = s4; s4 = s5; s5 = s6; s6 = s7;
        return sft;
    }
};

template <class T>
__global__ __launch_bounds__(T::kThreads) void k_gemm(GemmArgs p, int64_t tiles_m, int64_t tiles_n,
                                                      int64_t k_per_split) {
    __shared__ __attribute__((aligned(16))) int8_t smem[T::kSmem];
    using MF = Mfma<T::MF>;
    using acc_t = typename MF::acc_t;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / T::WN, wn = wave % T::WN;
    int64_t tm, tn;
    tile_coords(blockIdx.x, tiles_m, tiles_n, tm, tn);
    const int64_t m0 = tm * T::BM, n0 = tn * T::BN;

    // K tiles: this split's slice of the main segment, with the appended
    // fold columns (dgrad) around it.
    const FoldView fv = fold_view(p, T::BK);
    const int64_t kbeg = (int64_t)blockIdx.y * k_per_split;
    const int64_t kend = min(p.K, kbeg + k_per_split);
    const int n_main = kend > kbeg ? (int)((kend - kbeg + T::BK - 1) / T::BK) : 0;
    const int n_tiles = fv.n_ext + n_main;

    acc_t acc[T::FM][T::FN];
#pragma unroll
    for (int i = 0; i < T::FM; ++i)
#pragma unroll
        for (int j = 0; j < T::FN; ++j)
#pragma unroll
            for (int r = 0; r < T::NACC; ++r) acc[i][j][r] = 0;

    uint4 ra[T::LA], rb[T::LB];

    auto load = [&](int t) {
        const int8_t *Ab, *Bb;
        int64_t la, lb, k0, klim;
        if (fv.is_ext(t, n_main)) {
            Ab = p.extA; la = p.ld_extA; Bb = p.extB; lb = p.ld_extB;
            k0 = fv.ext_col(t, n_main); klim = (int64_t)fv.n_ext * T::BK;
        } else {
            Ab = p.A; la = p.lda; Bb = p.B; lb = p.ldb;
            k0 = kbeg + (int64_t)(t - fv.h_tiles) * T::BK; klim = kend;
        }
#pragma unroll
        for (int i = 0; i < T::LA; ++i) {
            const int id = tid + i * T::kThreads;
            const int row = id / T::CPR, c16 = (id % T::CPR) * 16;
            const int64_t kk = k0 + c16, gm = m0 + row;
            uint4 v = make_uint4(0u, 0u, 0u, 0u);
            if (kk < klim && gm < p.Mg) {
                v = *reinterpret_cast<const uint4*>(Ab + gm * la + kk);
                if (kk + 16 > klim) v = mask_tail(v, (int)(klim - kk));
            }
            ra[i] = v;
        }
#pragma unroll
        for (int i = 0; i < T::LB; ++i) {
            const int id = tid + i * T::kThreads;
            const int row = id / T::CPR, c16 = (id % T::CPR) * 16;
            const int64_t kk = k0 + c16, gn = n0 + row;
            uint4 v = make_uint4(0u, 0u, 0u, 0u);
            if (kk < klim && gn < p.Ng) {
                v = *reinterpret_cast<const uint4*>(Bb + gn * lb + kk);
                if (kk + 16 > klim) v = mask_tail(v, (int)(klim - kk));
            }
            rb[i] = v;
        }
    };
    auto store = [&](int buf) {
        int8_t* sA = smem + buf * (T::BM + T::BN) * T::LS;
        int8_t* sB = sA + T::BM * T::LS;
#pragma unroll
        for (int i = 0; i < T::LA; ++i) {
            const int id = tid + i * T::kThreads;
            *reinterpret_cast<uint4*>(&sA[(id / T::CPR) * T::LS + (id % T::CPR) * 16]) = ra[i];
        }
#pragma unroll
        for (int i = 0; i < T::LB; ++i) {
            const int id = tid + i * T::kThreads;
            *reinterpret_cast<uint4*>(&sB[(id / T::CPR) * T::LS + (id % T::CPR) * 16]) = rb[i];
        }
    };
    auto compute = [&](int buf) {
        const int8_t* sA = smem + buf * (T::BM + T::BN) * T::LS;
        const int8_t* sB = sA + T::BM * T::LS;
        const int lrow = lane % T::MF, lk = (lane / T::MF) * 16;
#pragma unroll
        for (int ks = 0; ks < T::BK / T::KS; ++ks) {
            v4i a[T::FM], b[T::FN];
#pragma unroll
            for (int i = 0; i < T::FM; ++i)
                a[i] = *reinterpret_cast<const v4i*>(
                    &sA[(wm * T::TM + i * T::MF + lrow) * T::LS + ks * T::KS + lk]);
#pragma unroll
            for (int j = 0; j < T::FN; ++j)
                b[j] = *reinterpret_cast<const v4i*>(
                    &sB[(wn * T::TN + j * T::MF + lrow) * T::LS + ks * T::KS + lk]);
            // The B tile feeds the matrix-core A operand, so each lane's
            // results run along an output row (4 consecutive columns).
#pragma unroll
            for (int i = 0; i < T::FM; ++i)
#pragma unroll
                for (int j = 0; j < T::FN; ++j) acc[i][j] = MF::run(b[j], a[i], acc[i][j]);
        }
    };

    if (n_tiles > 0) {
        load(0);
        store(0);
        __syncthreads();
        HornerSteps hs(p);
        for (int t = 0; t < n_tiles; ++t) {
            if (t + 1 < n_tiles) load(t + 1);
            if ((int64_t)t * T::BK == hs.col) {
                const int sft = hs.advance();
#pragma unroll
                for (int i = 0; i < T::FM; ++i)
#pragma unroll
                    for (int j = 0; j < T::FN; ++j) acc[i][j] = acc[i][j] << sft;
            }
            compute(t & 1);
            if (t + 1 < n_tiles) store((t + 1) & 1);
            __syncthreads();
        }
    }

    if (fv.fshift) {
#pragma unroll
        for (int i = 0; i < T::FM; ++i)
#pragma unroll
            for (int j = 0; j < T::FN; ++j) acc[i][j] = acc[i][j] << fv.fshift;
    }

    // ---- epilogue ----
    float base = 0.0f, alpha = 0.0f, gstep = 0.0f;
    if (p.out && !p.part) {
        const sq_scale gs = *p.gs, os = *p.os;
        gstep = gs.step;
        base = __fmul_rn(gs.step, os.step);
        alpha = __fmul_rn(base, pow2f(-(p.num_groups - 1)));
    }
    const bool vec_acc = p.acc && ((p.ld_acc & 3) == 0) && ((reinterpret_cast<uintptr_t>(p.acc) & 15) == 0);
    const bool vec_out = p.out && ((p.ld_out & 3) == 0) && ((reinterpret_cast<uintptr_t>(p.out) & 15) == 0);
    const bool vec_part = p.part && ((p.Ng & 3) == 0) && ((reinterpret_cast<uintptr_t>(p.part) & 15) == 0);
    constexpr int kQuads = T::NACC / 4;   // groups of 4 consecutive columns per lane and MFMA block
    // epi_mode 2: this lane's output columns are the same for every row
    float cs[T::FN][kQuads][4];
#pragma unroll
    for (int j = 0; j < T::FN; ++j)
#pragma unroll
        for (int q = 0; q < kQuads; ++q) {
            const int64_t jj = n0 + wn * T::TN + j * T::MF + (T::MF == 32 ? q * 8 + (lane / 32) * 4 : (lane / 16) * 4);
#pragma unroll
            for (int e = 0; e < 4; ++e)
                cs[j][q][e] = (p.epi_mode == 2 && p.out && !p.part && jj + e < p.Ng) ? col_scale(p, gstep, jj + e) : 0.0f;
        }
#pragma unroll
    for (int i = 0; i < T::FM; ++i) {
        const int64_t ii = m0 + wm * T::TM + i * T::MF + lane % T::MF;
        if (ii >= p.Mg) continue;
        float sc = alpha;
        if (p.out && !p.part && p.epi_mode == 1) sc = __fmul_rn(base, pow2f(-(int)p.group[ii]));
#pragma unroll
        for (int j = 0; j < T::FN; ++j) {
#pragma unroll
            for (int q = 0; q < kQuads; ++q) {
                // 32x32: register quartet q covers columns 8q + 4 * (lane / 32) + 0..3
                // 16x16: columns 4 * (lane / 16) + 0..3
                const int64_t jj = n0 + wn * T::TN + j * T::MF +
                                   (T::MF == 32 ? q * 8 + (lane / 32) * 4 : (lane / 16) * 4);
                if (jj >= p.Ng) continue;
                const int v0 = acc[i][j][q * 4 + 0], v1 = acc[i][j][q * 4 + 1];
                const int v2 = acc[i][j][q * 4 + 2], v3 = acc[i][j][q * 4 + 3];
                const int vv[4] = {v0, v1, v2, v3};
                const bool full = jj + 4 <= p.Ng;
                if (p.part) {
                    // split-K: this split's partial tile, dense [splits, Mg, Ng]
                    int32_t* dst = p.part + (int64_t)blockIdx.y * p.Mg * p.Ng + ii * p.Ng + jj;
                    if (vec_part && full) {
                        *reinterpret_cast<int4*>(dst) = make_int4(v0, v1, v2, v3);
                    } else {
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            if (jj + e < p.Ng) dst[e] = vv[e];
                    }
                    continue;
                }
                if (p.acc) {
                    int32_t* dst = p.acc + ii * p.ld_acc + jj;
                    if (vec_acc && full) {
                        *reinterpret_cast<int4*>(dst) = make_int4(v0, v1, v2, v3);
                    } else {
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            if (jj + e < p.Ng) dst[e] = vv[e];
                    }
                }
                if (p.out) {
                    float* dst = p.out + ii * p.ld_out + jj;
                    float s4[4] = {sc, sc, sc, sc};
                    if (p.epi_mode == 2)
#pragma unroll
                        for (int e = 0; e < 4; ++e) s4[e] = cs[j][q][e];
                    const float f0 = __fmul_rn((float)v0, s4[0]), f1 = __fmul_rn((float)v1, s4[1]);
                    const float f2 = __fmul_rn((float)v2, s4[2]), f3 = __fmul_rn((float)v3, s4[3]);
                    if (vec_out && full) {
                        store_f4(dst, f0, f1, f2, f3, p.epi_mode == 1);
                    } else {
                        const float ff[4] = {f0, f1, f2, f3};
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            if (jj + e < p.Ng) store_f1(dst + e, ff[e], p.epi_mode == 1);
                    }
                }
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Pipelined variant for K-aligned operands: 64-byte K tiles move from global
// memory straight into a ring of STAGES LDS buffers with the gfx950 direct
// loads (buffer_load_dwordx4 ... lds, 16 bytes per lane, a fixed per-lane
// offset and a scalar K offset), so STAGES - 1 tiles are in flight without
// holding registers or address arithmetic.  Each wave instruction fills 1 KB of
// LDS = 16 rows x 64 bytes in lane order; the 16-byte chunk c of row r is
// stored at chunk c ^ swz(r), which keeps the fragment reads conflict-free.
// Synchronisation is explicit: a wave waits (vmcnt) for its own loads of
// tile t, a barrier publishes them to the block, and a stage is refilled only
// after the barrier that follows every wave's reads of it.  The MFMA operands
// are double-buffered in registers: the LDS reads of tile t + 1 are issued
// before the MFMAs of tile t, so they complete while the matrix cores work.
// HORNER = false compiles out the accumulator shifts of the fold (wgrad, and
// dgrads whose fold has one window), which lets the accumulators live in the
// matrix-core registers for the whole loop.
// Requirements (checked by the launcher): every K segment a multiple of 64,
// lda/ldb multiples of 16, 16-byte aligned operands, offsets below 2^31.
// ---------------------------------------------------------------------------
template <int BM_, int BN_, int WM_, int WN_, int MF_, int STAGES_>
struct PipeCfg {
    static constexpr int BM = BM_, BN = BN_, BK = 64, WM = WM_, WN = WN_, MF = MF_, STAGES = STAGES_;
    static constexpr int kThreads = 64 * WM * WN, kWaves = WM * WN;
    static constexpr int TM = BM / WM, TN = BN / WN;
    static constexpr int FM = TM / MF, FN = TN / MF;
    static constexpr int KS = MF == 32 ? 32 : 64;
    static constexpr int KSTEPS = BK / KS;                // MFMA k-steps per K tile
    static constexpr int NACC = MF == 32 ? 16 : 4;
    static constexpr int kStage = (BM + BN) * BK;         // bytes per stage
    static constexpr int IA = BM / 16 / kWaves;           // A load instructions per wave per stage
    static constexpr int IB = BN / 16 / kWaves;
    static constexpr int kLoads = IA + IB;
    static constexpr int kSmem = STAGES * kStage;
    static_assert(IA * 16 * kWaves == BM && IB * 16 * kWaves == BN, "rows split evenly over waves");
    static_assert(TM % MF == 0 && TN % MF == 0, "wave tile must hold whole MFMA blocks");
    static_assert(STAGES >= 3 && STAGES <= 4 && (STAGES - 2) * kLoads <= 63, "vmcnt range");
};

using PipeLarge = PipeCfg<256, 256, 4, 2, 16, 4>;   // 128 KB of LDS, one block per CU
using PipeWide = PipeCfg<256, 256, 2, 2, 16, 4>;    // 4 waves of 128 x 128: half the LDS reads per MFMA
using PipeSmall = PipeCfg<128, 128, 2, 2, 16, 4>;   // 64 KB of LDS
using PipeSkinny = PipeCfg<64, 192, 2, 2, 16, 4>;   // at most 64 output rows (wgrad of narrow layers)
using PipeTall = PipeCfg<128, 384, 2, 4, 16, 4>;    // 8 waves of 64 x 96: more tiles where 256 x 256 leaves CUs idle
using PipeNarrow = PipeCfg<256, 64, 4, 1, 16, 4>;   // at most 64 output columns (conv dgrad), 80 KB of LDS

typedef __attribute__((address_space(3))) void lds_void_t;

// chunk swizzle of a 64-byte LDS row (conflict-free for 8- and 16-lane phases)
[[maybe_unused]] __device__ __forceinline__ int swz(int r) { return ((r >> 1) ^ (r >> 2)) & 3; }

// s_waitcnt vmcnt(n) leaving the other counters unconstrained (gfx9 encoding)
template <int N>
__device__ __forceinline__ void wait_vm() {
    __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// Maximum over the 16 lanes of a DPP row (lanes 16 r .. 16 r + 15), in every
// lane of the row: swaps within quads (xor 1, xor 2), then the mirrors of
// each 8-lane half and of the whole row.  Every lane of the wave must be active.
[[maybe_unused]] __device__ __forceinline__ uint32_t row16_max(uint32_t v) {
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xF, 0xF, false));    // quad_perm [1,0,3,2]
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xF, 0xF, false));    // quad_perm [2,3,0,1]
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x141, 0xF, 0xF, false));   // row_half_mirror
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x140, 0xF, 0xF, false));   // row_mirror
    return v;
}

template <class T, bool HORNER, bool CONV = false, bool RANGES = false>
__global__ __launch_bounds__(T::kThreads) void k_gemm_pipe(GemmArgs p, int64_t tiles_m, int64_t tiles_n,
                                                           int64_t k_per_split) {
#if defined(__HIP_DEVICE_COMPILE__)   // buffer resources exist in the device pass only
    __shared__ __attribute__((aligned(1024))) int8_t smem[T::kSmem];
    using MF = Mfma<T::MF>;
    using acc_t = typename MF::acc_t;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / T::WN, wn = wave % T::WN;
    // Split-K launches are one-dimensional, over (split, tile) items taken
    // split-major.  Blocks go to the XCDs round-robin (block L to XCD L mod 8),
    // so XCD x is given the contiguous run of items after those of XCDs
    // 0 .. x-1: its CUs work on the tiles of one or two K splits at a time and
    // share its L2 (the MLP layer's 7-split wgrad: 184 -> 87 MB fetched past
    // the L2, 52.4 -> 50.5 us).  Within the run, tiles go in the grouped raster.
    int64_t bt = blockIdx.x, split = blockIdx.y;
    int64_t tm, tn;
    if (p.splits > 1) {
        const int64_t nt = tiles_m * tiles_n, total = nt * p.splits, L = blockIdx.x;
        const int64_t x = L & 7, j = L >> 3;
        int64_t start = 0;   // items of XCDs 0 .. x-1: ceil((total - y) / 8) each
        for (int64_t y = 0; y < x; ++y) start += (total - y + 7) >> 3;
        const int64_t i = start + j;
        split = i / nt;
        bt = i - split * nt;
        const int64_t per_group = kGroupM * tiles_n, first_m = (bt / per_group) * kGroupM;
        const int64_t gsz = min(tiles_m - first_m, (int64_t)kGroupM), w = bt % per_group;
        tm = first_m + w % gsz;
        tn = w / gsz;
    } else {
        tile_coords(bt, tiles_m, tiles_n, tm, tn);
    }
    const int64_t m0 = tm * T::BM, n0 = tn * T::BN;

    const FoldView fv = fold_view(p, T::BK);
    int64_t koff = 0, Kd = p.K;   // K range: [0, K), or a device-side segment
    if (p.kseg) { koff = p.kseg[0]; Kd = p.kseg[1]; }
    const int64_t kbeg = split * k_per_split;
    const int64_t kend = min(Kd, kbeg + k_per_split);
    const int n_main = kend > kbeg ? (int)((kend - kbeg) / T::BK) : 0;
    // a convolution visits the flat fold sequence once per tap: tile t is
    // flat tile t / taps of tap t % taps
    const int taps = CONV ? p.taps : 1;
    const int n_tiles = (fv.n_ext + n_main) * taps;

    // Operand tiles come in with buffer loads straight to LDS: each lane's
    // 32-bit byte offset (row of its load instruction, logical chunk
    // (lane % 4) ^ swz(r)) is fixed for the whole K loop, and the K offset of
    // the tile is a scalar.  Rows past the end of an operand read its last
    // row (their results are never stored).  The launcher guarantees that
    // every offset fits in 31 bits.
    const int wv = __builtin_amdgcn_readfirstlane(wave);
    const int lr = lane >> 2;
    constexpr int kRsrcFlags = 0x00020000;   // raw byte buffer, gfx9 data format
    auto rsrc = [&](const int8_t* base, int64_t rows, int64_t ld) {
        return __builtin_amdgcn_make_buffer_rsrc(const_cast<int8_t*>(base), (short)0, (int)min(rows * ld, (int64_t)0x7FFFFFFF),
                                                 kRsrcFlags);
    };
    // tile-major operands (p.tiled) hold whole 16-row groups
    const int64_t rows_a = CONV ? p.a_rows : (p.tiled ? round_up(p.Mg, 16) : p.Mg);
    const int64_t rows_b = p.tiled ? round_up(p.Ng, 16) : p.Ng;
    const __amdgpu_buffer_rsrc_t rA = rsrc(p.A, rows_a, p.lda), rB = rsrc(p.B, rows_b, p.ldb);
    // Row-major: row r at r ld.  Tile-major: the 16 rows of this load
    // instruction form one contiguous 1 KB tile per K tile, and the K offset
    // of a tile (scalar) is its index times 1 KB.
    auto lane_off = [&](int i, int64_t first, int64_t rows, int64_t ld) {
        const int r = (i * T::kWaves + wv) * 16 + lr;
        const int64_t rr = min(first + r, rows - 1);
        const int chunk = 16 * ((lane & 3) ^ swz(r));
        if (p.tiled) return (uint32_t)(tiled_off(rr, 0, ld) + chunk);
        return (uint32_t)(rr * ld + chunk);
    };
    auto kbytes = [&](int64_t col) { return (int)(p.tiled ? (col >> 6) << 10 : col); };
    uint32_t offA[T::IA], offB[T::IB];
#pragma unroll
    for (int i = 0; i < T::IA; ++i) offA[i] = lane_off(i, m0, p.Mg, p.lda);
#pragma unroll
    for (int i = 0; i < T::IB; ++i) offB[i] = lane_off(i, n0, p.Ng, p.ldb);
    // Convolution: the input pixel (n, ih, iw) of each of this lane's A rows;
    // tap (r, s) reads output pixel (n, ih + PH - r, iw + PW - s) of q_fold,
    // or, outside the output grid, an offset past the end of the buffer,
    // which the buffer load's range check turns into zeros.
    int cv_ih[CONV ? T::IA : 1], cv_iw[CONV ? T::IA : 1], cv_row0[CONV ? T::IA : 1];
    uint32_t cv_chunk[CONV ? T::IA : 1];
    if constexpr (CONV) {
#pragma unroll
        for (int i = 0; i < T::IA; ++i) {
            const int r = (i * T::kWaves + wv) * 16 + lr;
            const int64_t pix = min(m0 + r, p.Mg - 1);
            const int64_t n = pix / (p.cv_H * p.cv_W), hw = pix - n * p.cv_H * p.cv_W;
            cv_ih[i] = (int)(hw / p.cv_W);
            cv_iw[i] = (int)(hw - (int64_t)cv_ih[i] * p.cv_W);
            cv_row0[i] = (int)(n * p.cv_Ho * p.cv_Wo);
            cv_chunk[i] = 16u * (uint32_t)((lane & 3) ^ swz(r));
        }
    }
    auto conv_off = [&](int i, int tr, int ts) -> uint32_t {
        const int oh = cv_ih[i] + p.cv_PH - tr, ow = cv_iw[i] + p.cv_PW - ts;
        const bool ok = (uint32_t)oh < (uint32_t)p.cv_Ho && (uint32_t)ow < (uint32_t)p.cv_Wo;
        return ok ? (uint32_t)((cv_row0[i] + oh * (int)p.cv_Wo + ow) * (int)p.lda) + cv_chunk[i] : 0x80000000u;
    };

    // (flat tile, tap) of the next tile to issue and of the next tile to
    // compute; issue() and step() each visit t = 0, 1, 2, ... in order
    TapCursor icur, hcur;
    auto issue = [&](int t) {
        int8_t* st = smem + (t % T::STAGES) * T::kStage;
        if constexpr (CONV) {
            const int f = icur.f, tr = icur.r, ts = icur.s;
            icur.next(taps, p.cv_KW);
            const bool ext = HORNER && fv.is_ext(f, n_main);
            const int k0 = ext ? (int)fv.ext_col(f, n_main) : (f - fv.h_tiles) * T::BK;
            const __amdgpu_buffer_rsrc_t ra = ext ? rsrc(p.extA, p.a_rows, p.ld_extA) : rA;
#pragma unroll
            for (int i = 0; i < T::IA; ++i)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (lds_void_t*)(st + (i * T::kWaves + wv) * 1024), 16,
                                                         conv_off(i, tr, ts), k0, 0, 0);
#pragma unroll
            for (int i = 0; i < T::IB; ++i)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(rB, (lds_void_t*)(st + T::BM * T::BK + (i * T::kWaves + wv) * 1024),
                                                         16, offB[i], t * T::BK, 0, 0);
            return;
        }
        if (HORNER && fv.is_ext(t, n_main)) {
            // appended fold columns (a few tiles): offsets computed here
            const __amdgpu_buffer_rsrc_t rAe = rsrc(p.extA, p.tiled ? round_up(p.Mg, 16) : p.Mg, p.ld_extA),
                                         rBe = rsrc(p.extB, p.tiled ? round_up(p.Ng, 16) : p.Ng, p.ld_extB);
            const int64_t col = fv.ext_col(t, n_main);
            const int k0a = kbytes(p.ext_koff + col), k0b = kbytes(col);
#pragma unroll
            for (int i = 0; i < T::IA; ++i)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(rAe, (lds_void_t*)(st + (i * T::kWaves + wv) * 1024), 16,
                                                         lane_off(i, m0, p.Mg, p.ld_extA), k0a, 0, 0);
#pragma unroll
            for (int i = 0; i < T::IB; ++i)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(
                    rBe, (lds_void_t*)(st + T::BM * T::BK + (i * T::kWaves + wv) * 1024), 16,
                    lane_off(i, n0, p.Ng, p.ld_extB), k0b, 0, 0);
            return;
        }
        const int k0 = kbytes(koff + kbeg + (int64_t)(t - fv.h_tiles) * T::BK);
#pragma unroll
        for (int i = 0; i < T::IA; ++i)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rA, (lds_void_t*)(st + (i * T::kWaves + wv) * 1024), 16, offA[i],
                                                     k0, 0, 0);
#pragma unroll
        for (int i = 0; i < T::IB; ++i)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rB, (lds_void_t*)(st + T::BM * T::BK + (i * T::kWaves + wv) * 1024),
                                                     16, offB[i], k0, 0, 0);
    };

    acc_t acc[T::FM][T::FN];
#pragma unroll
    for (int i = 0; i < T::FM; ++i)
#pragma unroll
        for (int j = 0; j < T::FN; ++j)
#pragma unroll
            for (int r = 0; r < T::NACC; ++r) acc[i][j][r] = 0;

    // MFMA operands of one K tile, double-buffered (buffer index fixed at
    // compile time by the two-step unrolled loop below)
    v4i fa[2][T::KSTEPS][T::FM], fb[2][T::KSTEPS][T::FN];
    const int lrow = lane % T::MF, lc = lane / T::MF;
    // This lane's byte offset in a stage is fixed: r * BK + 16 (c ^ swz(r))
    // depends on r only through r mod 8, which every 16-row fragment shares,
    // so each fragment read is one base register plus a compile-time offset
    // (fragment, operand, stage) once the loop is unrolled over the stages.
    static_assert(T::KSTEPS == 1 && T::MF == 16 && T::TM % 8 == 0 && T::TN % 8 == 0, "fixed-offset fragment reads");
    const int lane_base_a = [&] {
        const int r = wm * T::TM + lrow;
        return r * T::BK + 16 * (lc ^ swz(r));
    }();
    const int lane_base_b = [&] {
        const int r = wn * T::TN + lrow;
        return r * T::BK + 16 * (lc ^ swz(r));
    }();
    auto read_frags_at = [&](auto STG, auto BUF) {
        constexpr int buf = decltype(BUF)::value, stg = decltype(STG)::value;
#pragma unroll
        for (int i = 0; i < T::FM; ++i)
            fa[buf][0][i] = *reinterpret_cast<const v4i*>(smem + stg * T::kStage + lane_base_a + i * T::MF * T::BK);
#pragma unroll
        for (int j = 0; j < T::FN; ++j)
            fb[buf][0][j] = *reinterpret_cast<const v4i*>(smem + stg * T::kStage + T::BM * T::BK + lane_base_b +
                                                           j * T::MF * T::BK);
    };
    auto read_frags = [&](int t, auto BUF) {
        constexpr int buf = decltype(BUF)::value;
        const int8_t* sA = smem + (t % T::STAGES) * T::kStage;
        const int8_t* sB = sA + T::BM * T::BK;
#pragma unroll
        for (int ks = 0; ks < T::KSTEPS; ++ks) {
            const int c = ks * (T::KS / 16) + lc;   // logical 16-byte chunk of this lane
#pragma unroll
            for (int i = 0; i < T::FM; ++i) {
                const int r = wm * T::TM + i * T::MF + lrow;
                fa[buf][ks][i] = *reinterpret_cast<const v4i*>(&sA[r * T::BK + 16 * (c ^ swz(r))]);
            }
#pragma unroll
            for (int j = 0; j < T::FN; ++j) {
                const int r = wn * T::TN + j * T::MF + lrow;
                fb[buf][ks][j] = *reinterpret_cast<const v4i*>(&sB[r * T::BK + 16 * (c ^ swz(r))]);
            }
        }
    };
    // B fragment outer: the first MFMAs of a tile need the A fragments and
    // the first B fragment only, so they start before the later reads land
    auto mfmas = [&](auto BUF) {
        constexpr int buf = decltype(BUF)::value;
#pragma unroll
        for (int ks = 0; ks < T::KSTEPS; ++ks)
#pragma unroll
            for (int j = 0; j < T::FN; ++j)
#pragma unroll
                for (int i = 0; i < T::FM; ++i) acc[i][j] = MF::run(fb[buf][ks][j], fa[buf][ks][i], acc[i][j]);
    };
    // this wave's loads of a tile are complete once at most `later` younger
    // tiles remain in flight
    auto wait_tile = [&](int later) {
        if (later >= 2) wait_vm<2 * T::kLoads>();
        else if (later == 1) wait_vm<T::kLoads>();
        else wait_vm<0>();
    };

    HornerSteps hs(p);
    // one K tile: publish tile t + 1, refill the stage tile t - 1 used, read
    // tile t + 1's operands, then the MFMAs of tile t.  The reads are issued
    // on the last tile too (of a stale stage, never used), which keeps the
    // loop body free of branches around LDS reads, so the compiler's counter
    // waits before the MFMAs leave the new reads in flight.
    auto step = [&](int t, auto CUR, auto NXT, auto STG_NXT) {
        wait_tile(min(T::STAGES - 3, n_tiles - 2 - t));
        __builtin_amdgcn_s_barrier();
        if (t + T::STAGES - 1 < n_tiles) issue(t + T::STAGES - 1);
        const bool region_start = CONV ? hcur.tau == 0 && (int64_t)hcur.f * T::BK == hs.col : (int64_t)t * T::BK == hs.col;
        if constexpr (CONV) hcur.next(taps, p.cv_KW);
        if (HORNER && region_start) {
            const int sft = hs.advance();
#pragma unroll
            for (int i = 0; i < T::FM; ++i)
#pragma unroll
                for (int j = 0; j < T::FN; ++j) acc[i][j] = acc[i][j] << sft;
        }
        read_frags_at(STG_NXT, NXT);
        mfmas(CUR);
        // issue order: the LDS reads of the next tile spread between the
        // MFMAs of this one (each group: a share of MFMAs, then one read), so
        // the matrix cores start on operands that are already in registers
        constexpr int kReads = T::KSTEPS * (T::FM + T::FN);
        constexpr int kMfma = T::KSTEPS * T::FM * T::FN;
        constexpr int kPer = kMfma / kReads;
#pragma unroll
        for (int g = 0; g < kReads; ++g) {
            __builtin_amdgcn_sched_group_barrier(0x008, kPer, 0);   // MFMAs
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);      // one LDS read
        }
        __builtin_amdgcn_sched_group_barrier(0x008, kMfma - kPer * kReads, 0);
    };

    if (n_tiles > 0) {
#pragma unroll
        for (int s = 0; s < T::STAGES - 1; ++s)
            if (s < n_tiles) issue(s);
        wait_tile(min(T::STAGES - 2, n_tiles - 1));
        __builtin_amdgcn_s_barrier();
        read_frags(0, std::integral_constant<int, 0>());
        // unrolled over the 4 stages (tile t + 1 sits in stage (t + 1) % 4)
        using I0 = std::integral_constant<int, 0>;
        using I1 = std::integral_constant<int, 1>;
        using I2 = std::integral_constant<int, 2>;
        using I3 = std::integral_constant<int, 3>;
        static_assert(T::STAGES == 4, "loop unrolled over 4 stages");
        for (int t = 0; t < n_tiles; t += 4) {
            step(t, I0(), I1(), I1());
            if (t + 1 < n_tiles) step(t + 1, I1(), I0(), I2());
            if (t + 2 < n_tiles) step(t + 2, I0(), I1(), I3());
            if (t + 3 < n_tiles) step(t + 3, I1(), I0(), I0());
        }
    }

    // ---- epilogue (as in the register-staged kernel; the fold's final shift
    // is applied per element) ----
    const int fsh = HORNER ? fv.fshift : 0;
    float base = 0.0f, alpha = 0.0f, gstep = 0.0f;
    if (p.out && !p.part) {
        const sq_scale gs = *p.gs, os = *p.os;
        gstep = gs.step;
        base = __fmul_rn(gs.step, os.step);
        alpha = __fmul_rn(base, pow2f(-(p.num_groups - 1)));
    }
    const bool vec_acc = p.acc && ((p.ld_acc & 3) == 0) && ((reinterpret_cast<uintptr_t>(p.acc) & 15) == 0);
    const bool vec_out = p.out && ((p.ld_out & 3) == 0) && ((reinterpret_cast<uintptr_t>(p.out) & 15) == 0);
    const bool vec_part = p.part && ((p.Ng & 3) == 0) && ((reinterpret_cast<uintptr_t>(p.part) & 15) == 0);
    constexpr int kQuads = T::NACC / 4;
    // epi_mode 2: this lane's output columns are the same for every row
    float cs[T::FN][kQuads][4];
#pragma unroll
    for (int j = 0; j < T::FN; ++j)
#pragma unroll
        for (int q = 0; q < kQuads; ++q) {
            const int64_t jj = n0 + wn * T::TN + j * T::MF + (T::MF == 32 ? q * 8 + (lane / 32) * 4 : (lane / 16) * 4);
#pragma unroll
            for (int e = 0; e < 4; ++e)
                cs[j][q][e] = (p.epi_mode == 2 && p.out && !p.part && jj + e < p.Ng) ? col_scale(p, gstep, jj + e) : 0.0f;
        }
    // RANGES: channel maxima of |out| per 32-row slab (two 16-row fragments;
    // every wave's rows are whole slabs), bit patterns with the sign cleared
    static_assert(!RANGES || (T::MF == 16 && T::TM % 32 == 0), "ranges need 16-row fragments and whole slabs");
    uint32_t rm[RANGES ? T::FN : 1][4];
#pragma unroll
    for (int j = 0; j < (RANGES ? T::FN : 1); ++j)
#pragma unroll
        for (int e = 0; e < 4; ++e) rm[j][e] = 0u;
#pragma unroll
    for (int i = 0; i < T::FM; ++i) {
        const int64_t ii = m0 + wm * T::TM + i * T::MF + lane % T::MF;
        if (ii < p.Mg) {
        float sc = alpha;
        if (p.out && !p.part && p.epi_mode == 1) sc = __fmul_rn(base, pow2f(-(int)p.group[ii]));
#pragma unroll
        for (int j = 0; j < T::FN; ++j) {
#pragma unroll
            for (int q = 0; q < kQuads; ++q) {
                const int64_t jj = n0 + wn * T::TN + j * T::MF +
                                   (T::MF == 32 ? q * 8 + (lane / 32) * 4 : (lane / 16) * 4);
                if (jj >= p.Ng) continue;
                const int v0 = acc[i][j][q * 4 + 0] << fsh, v1 = acc[i][j][q * 4 + 1] << fsh;
                const int v2 = acc[i][j][q * 4 + 2] << fsh, v3 = acc[i][j][q * 4 + 3] << fsh;
                const int vv[4] = {v0, v1, v2, v3};
                const bool full = jj + 4 <= p.Ng;
                if (p.part) {
                    int32_t* dst = p.part + split * p.Mg * p.Ng + ii * p.Ng + jj;
                    if (vec_part && full) {
                        *reinterpret_cast<int4*>(dst) = make_int4(v0, v1, v2, v3);
                    } else {
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            if (jj + e < p.Ng) dst[e] = vv[e];
                    }
                    continue;
                }
                if (p.acc) {
                    int32_t* dst = p.acc + ii * p.ld_acc + jj;
                    if (vec_acc && full) {
                        *reinterpret_cast<int4*>(dst) = make_int4(v0, v1, v2, v3);
                    } else {
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            if (jj + e < p.Ng) dst[e] = vv[e];
                    }
                }
                if (p.out) {
                    float* dst = p.out + ii * p.ld_out + jj;
                    float s4[4] = {sc, sc, sc, sc};
                    if (p.epi_mode == 2)
#pragma unroll
                        for (int e = 0; e < 4; ++e) s4[e] = cs[j][q][e];
                    const float f0 = __fmul_rn((float)v0, s4[0]), f1 = __fmul_rn((float)v1, s4[1]);
                    const float f2 = __fmul_rn((float)v2, s4[2]), f3 = __fmul_rn((float)v3, s4[3]);
                    if (vec_out && full) {
                        store_f4(dst, f0, f1, f2, f3, p.epi_mode == 1);
                    } else {
                        const float ff[4] = {f0, f1, f2, f3};
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            if (jj + e < p.Ng) store_f1(dst + e, ff[e], p.epi_mode == 1);
                    }
                    if (RANGES) {
                        const float ff[4] = {f0, f1, f2, f3};
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            if (jj + e < p.Ng)
                                rm[RANGES ? j : 0][e] = max(rm[RANGES ? j : 0][e], __float_as_uint(ff[e]) & 0x7FFFFFFFu);
                    }
                }
            }
        }
        }
        if (RANGES && (i & 1)) {
            // end of a 32-row slab: maximum over the 16 lanes of each column
            // group (same lane / 16), then the group's first lane writes
            const int64_t slab = (m0 + wm * T::TM) / 32 + i / 2;
#pragma unroll
            for (int j = 0; j < (RANGES ? T::FN : 1); ++j)
#pragma unroll
                for (int e = 0; e < 4; ++e) rm[j][e] = row16_max(rm[j][e]);
            if ((lane & 15) == 0 && slab * 32 < p.Mg) {
#pragma unroll
                for (int j = 0; j < (RANGES ? T::FN : 1); ++j) {
                    const int64_t jj = n0 + wn * T::TN + j * T::MF + (lane / 16) * 4;
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        if (jj + e < p.Ng) p.ranges[slab * p.Ng + jj + e] = rm[j][e];
                }
            }
#pragma unroll
            for (int j = 0; j < (RANGES ? T::FN : 1); ++j)
#pragma unroll
                for (int e = 0; e < 4; ++e) rm[j][e] = 0u;
        }
    }
#endif
}

// ---------------------------------------------------------------------------
// Input gradient of a "same" stride-1 convolution (Ho = H, Wo = W) with the
// rows of q_fold staged once per K chunk.  Tap (r, s) of input pixel p reads
// q_fold row p + d, d = (PH - r) W + (PW - s), so the rows a tile of BM
// pixels needs for all taps form the contiguous window [p0 - E, p0 + BM + E),
// E = PH W + PW.  Per 64-column chunk of the fold's flat K sequence the block
// loads that window and the chunk's weights of every tap into LDS once, then
// runs one round of MFMAs per tap on rows of the window shifted by d.  A tap
// whose output pixel lies outside the image (its row belongs to another image
// row or image) adds nothing: that lane's operand fragment is cleared.  The
// K order (chunk-major, tap-minor) and the Horner shifts at region starts are
// those of the per-tap kernel.
// ---------------------------------------------------------------------------
constexpr int kHaloBM = 256, kHaloExtra = 128, kHaloWaves = 4, kHaloMaxTaps = 9;

template <bool HORNER>
__global__ __launch_bounds__(64 * kHaloWaves) void k_conv_halo(GemmArgs p) {
#if defined(__HIP_DEVICE_COMPILE__)
    constexpr int BM = kHaloBM, BN = 64, BK = 64, WR = kHaloBM + kHaloExtra;   // window rows
    constexpr int kA = WR * BK;
    __shared__ __attribute__((aligned(1024))) int8_t smem[kA + kHaloMaxTaps * BN * BK];
    using MF = Mfma<16>;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wv = __builtin_amdgcn_readfirstlane(wave);
    const int64_t m0 = (int64_t)blockIdx.x * BM, n0 = (int64_t)blockIdx.y * BN;
    const int taps = p.taps, KW = p.cv_KW, H = (int)p.cv_H, W = (int)p.cv_W;
    const int E = p.cv_PH * W + p.cv_PW;
    const FoldView fv = fold_view(p, BK);
    const int n_main = (int)(p.K / BK);
    const int n_chunks = fv.n_ext + n_main;

    constexpr int kRsrcFlags = 0x00020000;   // raw byte buffer, gfx9 data format
    auto rsrc = [&](const int8_t* base, int64_t rows, int64_t ld) {
        return __builtin_amdgcn_make_buffer_rsrc(const_cast<int8_t*>(base), (short)0,
                                                 (int)min(rows * ld, (int64_t)0x7FFFFFFF), kRsrcFlags);
    };
    const __amdgpu_buffer_rsrc_t rA = rsrc(p.A, p.a_rows, p.lda), rB = rsrc(p.B, p.Ng, p.ldb);
    const int lr = lane >> 2;
    // window rows: instruction i of this wave fills rows (i * waves + wv) * 16 .. + 15;
    // rows before the tensor get an offset past the end of the buffer (zeros)
    constexpr int kWin = WR / 16 / kHaloWaves;
    uint32_t offW[kWin];
#pragma unroll
    for (int i = 0; i < kWin; ++i) {
        const int w = (i * kHaloWaves + wv) * 16 + lr;
        const int64_t g = m0 - E + w;
        offW[i] = g >= 0 ? (uint32_t)(g * p.lda) + 16u * (uint32_t)((lane & 3) ^ swz(w)) : 0x80000000u;
    }
    // weights: this wave fills rows wv * 16 .. + 15 of each tap's 64-row block
    const int brow = wv * 16 + lr;
    const uint32_t offBw = (uint32_t)(min(n0 + brow, p.Ng - 1) * p.ldb);

    // the input pixel of each of this lane's 4 accumulator rows (one per
    // 16-row MFMA block of the wave's 64 rows)
    const int lrow = lane % 16, lc = lane / 16;
    int ih[4], iw[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int64_t pix = min(m0 + wv * 64 + i * 16 + lrow, p.Mg - 1);
        const int hw = (int)(pix % ((int64_t)H * W));
        ih[i] = hw / W;
        iw[i] = hw - ih[i] * W;
    }

    v4i acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = v4i{0, 0, 0, 0};

    HornerSteps hs(p);
    for (int f = 0; f < n_chunks; ++f) {
        // stage the chunk: the row window of q_fold and every tap's weights
        const bool ext = HORNER && fv.is_ext(f, n_main);
        const int kc = ext ? (int)fv.ext_col(f, n_main) : (f - fv.h_tiles) * BK;
        const __amdgpu_buffer_rsrc_t ra = ext ? rsrc(p.extA, p.a_rows, p.ld_extA) : rA;
        __syncthreads();   // the previous chunk's reads of LDS are done
#pragma unroll
        for (int i = 0; i < kWin; ++i)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (lds_void_t*)(smem + (i * kHaloWaves + wv) * 1024), 16,
                                                     offW[i], kc, 0, 0);
        for (int tau = 0; tau < taps; ++tau) {
            const int row = tau * BN + brow;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                rB, (lds_void_t*)(smem + kA + (tau * BN + wv * 16) * BK), 16,
                offBw + 16u * (uint32_t)((lane & 3) ^ swz(row)), (f * taps + tau) * BK, 0, 0);
        }
        wait_vm<0>();
        __syncthreads();
        if (HORNER && (int64_t)f * BK == hs.col) {
            const int sft = hs.advance();
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = acc[i][j] << sft;
        }
        for (int tau = 0, tr = 0, ts = 0; tau < taps; ++tau) {
            const int d = (p.cv_PH - tr) * W + (p.cv_PW - ts);
            v4i fa[4], fb[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int w = wv * 64 + i * 16 + lrow + E + d;
                const v4i v = *reinterpret_cast<const v4i*>(&smem[w * BK + 16 * (lc ^ swz(w))]);
                const int oh = ih[i] + p.cv_PH - tr, ow = iw[i] + p.cv_PW - ts;
                const bool ok = (unsigned)oh < (unsigned)H && (unsigned)ow < (unsigned)W;
                fa[i] = ok ? v : v4i{0, 0, 0, 0};
            }
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int r = tau * BN + j * 16 + lrow;
                fb[j] = *reinterpret_cast<const v4i*>(&smem[kA + r * BK + 16 * (lc ^ swz(r))]);
            }
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = MF::run(fb[j], fa[i], acc[i][j]);
            if (++ts == KW) { ts = 0; ++tr; }
        }
    }

    // epilogue: alpha = step_G * step_W * 2^-(N_G - 1), the fold's final shift
    const int fsh = HORNER ? fv.fshift : 0;
    float alpha = 0.0f;
    if (p.out) {
        const sq_scale gs = *p.gs, os = *p.os;
        alpha = __fmul_rn(__fmul_rn(gs.step, os.step), pow2f(-(p.num_groups - 1)));
    }
    const bool vec_acc = p.acc && ((p.ld_acc & 3) == 0) && ((reinterpret_cast<uintptr_t>(p.acc) & 15) == 0);
    const bool vec_out = p.out && ((p.ld_out & 3) == 0) && ((reinterpret_cast<uintptr_t>(p.out) & 15) == 0);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int64_t ii = m0 + wv * 64 + i * 16 + lrow;
        if (ii >= p.Mg) continue;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int64_t jj = n0 + j * 16 + lc * 4;
            if (jj >= p.Ng) continue;
            const int vv[4] = {acc[i][j][0] << fsh, acc[i][j][1] << fsh, acc[i][j][2] << fsh, acc[i][j][3] << fsh};
            const bool full = jj + 4 <= p.Ng;
            if (p.acc) {
                int32_t* dst = p.acc + ii * p.ld_acc + jj;
                if (vec_acc && full) *reinterpret_cast<int4*>(dst) = make_int4(vv[0], vv[1], vv[2], vv[3]);
                else
                    for (int e = 0; e < 4; ++e)
                        if (jj + e < p.Ng) dst[e] = vv[e];
            }
            if (p.out) {
                float* dst = p.out + ii * p.ld_out + jj;
                const float ff[4] = {__fmul_rn((float)vv[0], alpha), __fmul_rn((float)vv[1], alpha),
                                     __fmul_rn((float)vv[2], alpha), __fmul_rn((float)vv[3], alpha)};
                if (vec_out && full) *reinterpret_cast<float4*>(dst) = make_float4(ff[0], ff[1], ff[2], ff[3]);
                else
                    for (int e = 0; e < 4; ++e)
                        if (jj + e < p.Ng) dst[e] = ff[e];
            }
        }
    }
#endif
}

// ---------------------------------------------------------------------------
// Streaming variant of the same-size convolution input gradient for one
// 64-column K chunk (C_out <= 64, every shift in one window) and C_in <= 64.
// Each block owns a contiguous range of input pixels and walks it in steps of
// 128 rows (a wave takes rows 16 w .. and 64 + 16 w .. of the step, so each
// weight fragment read feeds two MFMAs).  The weights of every tap (rows
// (r, s, ci) of W^T, read straight from wq_t) stay in LDS; the rows of q_fold
// flow through an LDS ring of 64-row chunks, two per step, loaded kStreamPF
// steps ahead, and a step's outputs go out
// with buffer stores while the next steps compute, so the output stream (the
// bulk of the traffic) does not wait for loads.  A wave's loads and stores
// complete in order on gfx9, so the wait for a chunk also covers the stores
// issued before it: every wave issues the same number of loads and stores per
// step (rows outside the tensor or the block take offsets past the end of the
// buffer, which the range check drops), which keeps the vmcnt waits exact.
// Code columns >= C_out (unwritten padding of q_fold) are cleared in the
// operand registers (FULLK: all 64 columns hold codes, nothing to clear).
// Taps that fall outside the image read a 16-byte zero slot of LDS instead
// of their ring row.
// ---------------------------------------------------------------------------
[[maybe_unused]] constexpr int kStreamRing = 8, kStreamPF = 2, kStreamNW = 4;   // ring chunks, prefetch steps, chunks per step
constexpr int kStreamBlocks = 512;

// Hide a value from the optimizer, so that a memory instruction whose lanes
// take different offsets stays one instruction (not one per branch of a select).
template <class T>
__device__ __forceinline__ void opaque(T& v) { asm volatile("" : "+v"(v)); }

// RANGES: the block also writes max |dX| of each channel over its rows
// (bit patterns, sign cleared) to row blockIdx.x of p.ranges [blocks, Ng]:
// the producer-side channel ranges of the next layer's quantizer.
template <bool ACC, bool FULLK, bool RANGES = false>
__global__ __launch_bounds__(256) void k_conv_stream(GemmArgs p, int64_t rows_per_block) {
#if defined(__HIP_DEVICE_COMPILE__)
    constexpr int BK = 64, kRing = kStreamRing * 64 * BK;
    constexpr int kZero = kRing + kHaloMaxTaps * 64 * BK;   // 16 zero bytes
    constexpr int NS = ACC ? 16 : 8;   // stores per lane and step
    static_assert(kStreamNW + 2 * kStreamPF <= kStreamRing && 2 * NS + 4 <= 63, "ring / vmcnt range");
    __shared__ __attribute__((aligned(1024))) int8_t smem[kZero + 16];
    using MF = Mfma<16>;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
    if (tid == 0) *reinterpret_cast<uint4*>(smem + kZero) = make_uint4(0u, 0u, 0u, 0u);
    __syncthreads();
    const int taps = p.taps, KW = p.cv_KW, H = (int)p.cv_H, W = (int)p.cv_W;
    const int E = p.cv_PH * W + p.cv_PW;
    const int64_t r0 = (int64_t)blockIdx.x * rows_per_block;
    const int64_t r_end = min(p.Mg, r0 + rows_per_block);
    const int steps = (int)((r_end - r0 + 127) / 128);
    const int lr = lane >> 2, lrow = lane % 16, lc = lane / 16;
    constexpr int kRsrcFlags = 0x00020000;
    auto rsrc = [&](const void* base, int64_t bytes) {
        return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0,
                                                 base ? (int)min(bytes, (int64_t)0x7FFFFFFF) : 0, kRsrcFlags);
    };
    const __amdgpu_buffer_rsrc_t rA = rsrc(p.A, p.a_rows * p.lda), rB = rsrc(p.B, (int64_t)taps * p.Ng * p.ldb);
    const __amdgpu_buffer_rsrc_t rO = rsrc(p.out, p.Mg * p.ld_out * 4), rC = rsrc(p.acc, p.Mg * p.ld_acc * 4);

    // scalars first: their loads share the vmcnt counter with the DMA below
    float alpha = 0.0f;
    if (p.out) {
        const sq_scale gs = *p.gs, os = *p.os;
        alpha = __fmul_rn(__fmul_rn(gs.step, os.step), pow2f(-(p.num_groups - 1)));
    }
    const int fsh = p.layout ? p.layout[kLayF] : 0;
    __builtin_amdgcn_s_waitcnt(0);

    // weights: LDS rows tau * 64 + ci <- W^T row tau * C_in + ci; wave wv loads ci = 16 wv .. + 15
    {
        const int ci = wv * 16 + lr;
        const int64_t ci_c = min((int64_t)ci, p.Ng - 1);
        for (int tau = 0; tau < taps; ++tau) {
            const int row = tau * 64 + ci;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                rB, (lds_void_t*)(smem + kRing + (tau * 64 + wv * 16) * BK), 16,
                (uint32_t)(((int64_t)tau * p.Ng + ci_c) * p.ldb) + 16u * (uint32_t)((lane & 3) ^ swz(row)), 0, 0, 0);
        }
    }
    // chunk j of q_fold rows: r0 - E + 64 j .. + 63, in ring slot j mod kStreamRing
    const int64_t win_rows = (r_end - r0) + 2 * E;   // rows of the block's window (chunks past it load nothing)
    auto load_chunk = [&](int j) {
        const int wrow = 64 * j + wv * 16 + lr;             // row of the block's window
        const int slot_row = wrow & (kStreamRing * 64 - 1);
        const int64_t g = r0 - E + wrow;
        uint32_t off = g >= 0 && wrow < win_rows ? (uint32_t)(g * p.lda) + 16u * (uint32_t)((lane & 3) ^ swz(slot_row))
                                                 : 0x80000000u;
        opaque(off);   // one load instruction whatever the lanes' offsets
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rA, (lds_void_t*)(smem + (slot_row - lr) * BK), 16, off, 0, 0, 0);
    };
    // chunks 0 .. 2 PF + NW - 3 before the first step; step k loads chunks
    // 2 k + NW + 2 PF - 2 and + 1 (past the window: loads of nothing, still counted)
#pragma unroll
    for (int j = 0; j < kStreamNW + 2 * kStreamPF - 2; ++j) load_chunk(j);

    const int kvalid = (int)min((int64_t)16, max((int64_t)0, p.K_used - 16 * lc));   // code bytes < C_out
    // image row and column of this lane's two output rows, advanced by 128
    // pixels a step: (hw + 128 mod HW) < 2 HW, so one carry and one wrap
    // suffice (rows past the tensor get a position too; they are not stored)
    const uint32_t HW = (uint32_t)H * (uint32_t)W;
    const uint32_t adv = 128u % HW, adv_h = adv / (uint32_t)W, adv_w = adv - adv_h * (uint32_t)W;
    uint32_t ih[2], iw[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const uint32_t hw = (uint32_t)(r0 + 64 * h + wv * 16 + lrow) % HW;
        ih[h] = hw / (uint32_t)W;
        iw[h] = hw - ih[h] * (uint32_t)W;
    }
    // fp32 only: the fold's final shift goes into the scale, exactly
    // ((float)(v << f) * a == (float)v * (a * 2^f) while neither overflows)
    const float alpha_o = ACC ? alpha : __fmul_rn(alpha, pow2f(fsh));
    uint32_t rmx[RANGES ? 4 : 1][4];   // this lane's maxima of |dX|, columns j * 16 + lc * 4 + e
#pragma unroll
    for (int j = 0; j < (RANGES ? 4 : 1); ++j)
#pragma unroll
        for (int e = 0; e < 4; ++e) rmx[j][e] = 0u;
    for (int k = 0; k < steps; ++k) {
        load_chunk(2 * k + kStreamNW + 2 * kStreamPF - 2);
        load_chunk(2 * k + kStreamNW + 2 * kStreamPF - 1);
        // chunk 2 k + NW - 1, the last this step reads, was issued PF steps
        // back (the prologue's last for k < PF); it has landed once only the
        // younger operations remain: at most two loads per step since, and
        // the stores of the steps in between
        if (k == 0) wait_vm<4>();
        else if (k == 1) wait_vm<NS + 4>();
        else wait_vm<2 * NS + 4>();
        __builtin_amdgcn_s_barrier();   // a plain barrier: the stores stay in flight

        int64_t pix[2];
#pragma unroll
        for (int h = 0; h < 2; ++h) pix[h] = r0 + 128 * k + 64 * h + wv * 16 + lrow;   // this lane's output rows
        v4i acc[2][4];
        // one tap: its two A fragments (zero slot outside the image) times the
        // tap's four weight fragments; the first tap starts from zero
        auto tap = [&](int tau, int tr, int ts, auto FIRST) {
            const int d = (p.cv_PH - tr) * W + (p.cv_PW - ts);
            v4i fa[2];
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int w = (128 * k + 64 * h + wv * 16 + lrow + E + d) & (kStreamRing * 64 - 1);
                const int oh = (int)ih[h] + p.cv_PH - tr, ow = (int)iw[h] + p.cv_PW - ts;
                const bool inside = (unsigned)oh < (unsigned)H && (unsigned)ow < (unsigned)W;
                fa[h] = *reinterpret_cast<const v4i*>(&smem[inside ? w * BK + 16 * (lc ^ swz(w)) : kZero]);
                if (!FULLK && kvalid < 16) {
                    const uint4 m = mask_tail(make_uint4(fa[h][0], fa[h][1], fa[h][2], fa[h][3]), kvalid);
                    fa[h] = v4i{(int)m.x, (int)m.y, (int)m.z, (int)m.w};
                }
            }
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int r = tau * 64 + j * 16 + lrow;
                const v4i fb = *reinterpret_cast<const v4i*>(&smem[kRing + r * BK + 16 * (lc ^ swz(r))]);
#pragma unroll
                for (int h = 0; h < 2; ++h)
                    acc[h][j] = MF::run(fb, fa[h], decltype(FIRST)::value ? v4i{0, 0, 0, 0} : acc[h][j]);
            }
        };
        tap(0, 0, 0, std::true_type());
        for (int tau = 1, tr = KW == 1 ? 1 : 0, ts = KW == 1 ? 0 : 1; tau < taps; ++tau) {
            tap(tau, tr, ts, std::false_type());
            if (++ts == KW) { ts = 0; ++tr; }
        }
        // NS / 2 stores per row half: the fp32 output (a NULL output has an
        // empty range) and, with ACC, the int32 accumulator
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const bool row_ok = pix[h] < r_end;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int col = j * 16 + lc * 4;
                const bool ok = row_ok && col < p.Ng;
                // byte offsets below 2^31 (the output's size is checked on the host)
                const uint32_t prow = (uint32_t)pix[h];
                const int sh = ACC ? fsh : 0;
                const int v0 = acc[h][j][0] << sh, v1 = acc[h][j][1] << sh;
                const int v2 = acc[h][j][2] << sh, v3 = acc[h][j][3] << sh;
                typedef unsigned u4 __attribute__((ext_vector_type(4)));
                const u4 fo = {__float_as_uint(__fmul_rn((float)v0, alpha_o)), __float_as_uint(__fmul_rn((float)v1, alpha_o)),
                               __float_as_uint(__fmul_rn((float)v2, alpha_o)), __float_as_uint(__fmul_rn((float)v3, alpha_o))};
                int oo = ok ? (int)((prow * (uint32_t)p.ld_out + (uint32_t)col) * 4u) : (int)0x80000000;
                opaque(oo);
                __builtin_amdgcn_raw_buffer_store_b128(fo, rO, oo, 0, 0);
                if constexpr (RANGES) {
#pragma unroll
                    for (int e = 0; e < 4; ++e) rmx[j][e] = max(rmx[j][e], ok ? fo[e] & 0x7FFFFFFFu : 0u);
                }
                if constexpr (ACC) {
                    const u4 io = {(unsigned)v0, (unsigned)v1, (unsigned)v2, (unsigned)v3};
                    int oc = ok ? (int)((prow * (uint32_t)p.ld_acc + (uint32_t)col) * 4u) : (int)0x80000000;
                    opaque(oc);
                    __builtin_amdgcn_raw_buffer_store_b128(io, rC, oc, 0, 0);
                }
            }
        }
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            iw[h] += adv_w;
            ih[h] += adv_h;
            if (iw[h] >= (uint32_t)W) { iw[h] -= (uint32_t)W; ++ih[h]; }
            if (ih[h] >= (uint32_t)H) ih[h] -= (uint32_t)H;
        }
        __builtin_amdgcn_s_barrier();   // the ring slots of this step may be refilled
    }
    if constexpr (RANGES) {
        // maximum over the 16 rows of a DPP row (same lc), then over the 4
        // waves through LDS: the weight rows, no longer read after the last
        // barrier and never a target of the ring's prefetches still in flight
        uint32_t* red = reinterpret_cast<uint32_t*>(smem + kRing);   // [4 waves][64 columns]
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int e = 0; e < 4; ++e) rmx[j][e] = row16_max(rmx[j][e]);
        if (lrow == 0) {
#pragma unroll
            for (int j = 0; j < 4; ++j)
#pragma unroll
                for (int e = 0; e < 4; ++e) red[wv * 64 + j * 16 + lc * 4 + e] = rmx[j][e];
        }
        __syncthreads();
        if (tid < 64 && tid < p.Ng) {
            const uint32_t m = max(max(red[tid], red[64 + tid]), max(red[128 + tid], red[192 + tid]));
            p.ranges[(int64_t)blockIdx.x * p.Ng + tid] = m;
        }
    }
#endif
}

// Appended B columns of the dgrad fold: wext[k, j] = W^T code of the channel
// the layout lists for appended column j (0 for padding).
// Tile-major (tiled): both matrices in tiled_off order.
__global__ void k_gather_ext(const int8_t* __restrict__ wq_t, int64_t ld_w, int64_t C_in,
                             const int32_t* __restrict__ layout, int8_t* __restrict__ wext, int64_t ld_ext,
                             int tiled) {
    const int D = layout[1];
    const int32_t* ext = layout + kLayoutHeader;
    for (int64_t k = blockIdx.x; k < C_in; k += gridDim.x)
        for (int j = threadIdx.x; j < D; j += blockDim.x) {
            const int ch = ext[j];
            if (tiled) wext[tiled_off(k, j, ld_ext)] = ch >= 0 ? wq_t[tiled_off(k, ch, ld_w)] : (int8_t)0;
            else wext[k * ld_ext + j] = ch >= 0 ? wq_t[k * ld_w + ch] : (int8_t)0;
        }
}

// Sum of the split-K partial tiles ws [splits, Mg, Ng] (int32 addition is
// exact and order-free), then the same epilogue as the GEMM.  A block of
// kRedThreads covers kRedThreads / lanes groups of 4 consecutive outputs; the
// `lanes` threads of a group (a power of two, about a quarter of the splits,
// at most 16) read every lanes-th split, and are combined in LDS.
constexpr int kRedThreads = 256;

__global__ __launch_bounds__(kRedThreads) void k_splitk_reduce(
    const int32_t* __restrict__ ws, int splits, int lanes, int64_t Mg, int64_t Ng, int32_t* __restrict__ acc,
    int64_t ld_acc, float* __restrict__ out, int64_t ld_out, int epi_mode, const uint8_t* __restrict__ group,
    const sq_scale* __restrict__ gs, const sq_scale* __restrict__ os, int num_groups) {
    __shared__ int4 part[kRedThreads];
    const int64_t plane = Mg * Ng;
    const int items = kRedThreads / lanes;
    const int it = threadIdx.x % items, sl = threadIdx.x / items;
    const int64_t e = 4 * ((int64_t)blockIdx.x * items + it);   // outputs e .. e + 3 of the plane
    const bool vec = (Ng & 3) == 0;
    int4 sum = make_int4(0, 0, 0, 0);
    if (e < plane) {
        if (vec) {
            int s = sl;
            for (; s + 3 * lanes < splits; s += 4 * lanes) {
                int4 v[4];
#pragma unroll
                for (int u = 0; u < 4; ++u) v[u] = *reinterpret_cast<const int4*>(ws + (int64_t)(s + u * lanes) * plane + e);
#pragma unroll
                for (int u = 0; u < 4; ++u) { sum.x += v[u].x; sum.y += v[u].y; sum.z += v[u].z; sum.w += v[u].w; }
            }
            for (; s < splits; s += lanes) {
                const int4 v = *reinterpret_cast<const int4*>(ws + (int64_t)s * plane + e);
                sum.x += v.x; sum.y += v.y; sum.z += v.z; sum.w += v.w;
            }
        } else {
            int t[4] = {0, 0, 0, 0};
            for (int s = sl; s < splits; s += lanes)
#pragma unroll
                for (int u = 0; u < 4; ++u)
                    if (e + u < plane) t[u] += ws[(int64_t)s * plane + e + u];
            sum = make_int4(t[0], t[1], t[2], t[3]);
        }
    }
    if (lanes > 1) {
        part[threadIdx.x] = sum;
        __syncthreads();
        if (sl != 0) return;
        for (int l = 1; l < lanes; ++l) {
            const int4 v = part[l * items + it];
            sum.x += v.x; sum.y += v.y; sum.z += v.z; sum.w += v.w;
        }
    }
    if (e >= plane) return;
    float base = 0.0f, alpha = 0.0f;
    if (out) {
        base = __fmul_rn(gs->step, os->step);
        alpha = __fmul_rn(base, pow2f(-(num_groups - 1)));
    }
    const int t[4] = {sum.x, sum.y, sum.z, sum.w};
    int64_t i = e / Ng, j = e - i * Ng;   // a group of 4 spans two rows only when Ng % 4 != 0
    if (vec) {
        const float sc = out && epi_mode == 1 ? __fmul_rn(base, pow2f(-(int)group[i])) : alpha;
        if (acc) {
            int32_t* dst = acc + i * ld_acc + j;
            if (((ld_acc & 3) == 0) && ((reinterpret_cast<uintptr_t>(acc) & 15) == 0))
                *reinterpret_cast<int4*>(dst) = sum;
            else
                for (int u = 0; u < 4; ++u) dst[u] = t[u];
        }
        if (out) {
            float* dst = out + i * ld_out + j;
            const float f[4] = {__fmul_rn((float)t[0], sc), __fmul_rn((float)t[1], sc), __fmul_rn((float)t[2], sc),
                                __fmul_rn((float)t[3], sc)};
            if (((ld_out & 3) == 0) && ((reinterpret_cast<uintptr_t>(out) & 15) == 0))
                store_f4(dst, f[0], f[1], f[2], f[3], epi_mode == 1);
            else
                for (int u = 0; u < 4; ++u) store_f1(dst + u, f[u], epi_mode == 1);
        }
        return;
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        if (e + u >= plane) break;
        if (acc) acc[i * ld_acc + j] = t[u];
        if (out) {
            const float sc = epi_mode == 1 ? __fmul_rn(base, pow2f(-(int)group[i])) : alpha;
            store_f1(out + i * ld_out + j, __fmul_rn((float)t[u], sc), epi_mode == 1);
        }
        if (++j == Ng) { j = 0; ++i; }
    }
}

__global__ void k_dequant(const int32_t* __restrict__ acc, int64_t rows, int64_t cols, int64_t ld_acc, int kind,
                          const uint8_t* __restrict__ group, const sq_scale* __restrict__ gs,
                          const sq_scale* __restrict__ os, int num_groups, float* __restrict__ out,
                          int64_t ld_out) {
    const float base = __fmul_rn(gs->step, os->step);
    const float alpha = __fmul_rn(base, pow2f(-(num_groups - 1)));
    for (int64_t r = blockIdx.x; r < rows; r += gridDim.x) {
        const float sc = kind == 1 ? __fmul_rn(base, pow2f(-(int)group[r])) : alpha;
        for (int64_t c = threadIdx.x; c < cols; c += blockDim.x) {
            const float s = kind == 2 ? __fmul_rn(__fmul_rn(gs->step, os[c].step), pow2f(-(num_groups - 1))) : sc;
            out[r * ld_out + c] = __fmul_rn((float)acc[r * ld_acc + c], s);
        }
    }
}

// Launch one configuration.  k_per_split is a multiple of T::BK.
template <class T>
hipError_t launch_cfg(const GemmArgs& a, int splits, int64_t k_per_split, hipStream_t s) {
    const int64_t tiles_m = (a.Mg + T::BM - 1) / T::BM, tiles_n = (a.Ng + T::BN - 1) / T::BN;
    if (tiles_m * tiles_n > 0x7FFFFFFF || splits > 65535) return hipErrorInvalidValue;
    if (a.layout && T::BK != kFoldPad) return hipErrorInvalidValue;   // fold regions are whole K tiles
    dim3 grid((unsigned)(tiles_m * tiles_n), (unsigned)splits);
    hipLaunchKernelGGL(k_gemm<T>, grid, dim3(T::kThreads), 0, s, a, tiles_m, tiles_n, k_per_split);
    return hipGetLastError();
}

template <class T, bool HORNER, bool CONV = false, bool RANGES = false>
hipError_t launch_pipe(const GemmArgs& a, int splits, int64_t k_per_split, hipStream_t s) {
    const int64_t tiles_m = (a.Mg + T::BM - 1) / T::BM, tiles_n = (a.Ng + T::BN - 1) / T::BN;
    if (tiles_m * tiles_n * splits > 0x7FFFFFFF || splits > 65535) return hipErrorInvalidValue;
    // split-K: one-dimensional grid, decoded in the kernel (tiles of a split
    // on one XCD); a.splits must equal splits for that decoding
    if (splits > 1 && a.splits != splits) return hipErrorInvalidValue;
    const dim3 grid = splits > 1 ? dim3((unsigned)(tiles_m * tiles_n * splits)) : dim3((unsigned)(tiles_m * tiles_n));
    hipLaunchKernelGGL((k_gemm_pipe<T, HORNER, CONV, RANGES>), grid, dim3(T::kThreads), 0, s, a, tiles_m, tiles_n,
                       k_per_split);
    return hipGetLastError();
}

// The direct-load pipeline needs 64-byte K tiles that never cross the end of a
// segment, 16-byte aligned rows, and byte offsets (rows * ld + K) that fit
// the 31 bits of its buffer loads.
bool pipe_ok(const GemmArgs& a) {
    auto al16 = [](const void* q) { return (reinterpret_cast<uintptr_t>(q) & 15) == 0; };
    auto fits = [&](int64_t rows, int64_t ld, int64_t cols) {
        return (a.tiled ? round_up(rows, 16) : rows) * ld + cols < ((int64_t)1 << 31);
    };
    if (a.K % 64 != 0 || a.lda % 16 != 0 || a.ldb % 16 != 0 || !al16(a.A) || !al16(a.B)) return false;
    if (a.tiled && (a.lda % 64 != 0 || a.ldb % 64 != 0 || (a.extA && (a.ld_extA % 64 || a.ld_extB % 64 ||
                                                                     a.ext_koff % 64))))
        return false;
    if (!fits(a.Mg, a.lda, a.K) || !fits(a.Ng, a.ldb, a.K)) return false;
    if (a.extA) {
        if (a.ld_extA % 16 != 0 || a.ld_extB % 16 != 0 || !al16(a.extA) || !al16(a.extB)) return false;
        if (!fits(a.Mg, a.ld_extA, 0) || !fits(a.Ng, a.ld_extB, 0)) return false;
    }
    return true;
}

// Tile shape of a product: large tiles where there are enough of them (alone,
// or with K split into slices of at least 16 tiles) to fill most of the chip
// and K is long, a 64-row tile for products with at most 64 output rows,
// 128 x 128 otherwise.
enum class Pick { kLarge, kTall, kSmall, kSkinny };

int64_t tiles_of(const GemmArgs& a, int bm, int bn) { return ((a.Mg + bm - 1) / bm) * ((a.Ng + bn - 1) / bn); }

constexpr int64_t kLargeFill = 128;      // large tiles per launch that count as filling the chip
constexpr int64_t kCUs = 256;
constexpr int64_t kMinSplitKTiles = 16;  // K tiles per split of a large-tile split-K

// Split factor that brings large tiles of a short-and-narrow product with a
// long K to at most one block per CU (0: large tiles do not suit this product).
int64_t large_splits(const GemmArgs& a) {
    const int64_t tiles = tiles_of(a, PipeLarge::BM, PipeLarge::BN);
    if (tiles >= kLargeFill) return 1;
    // split only dense tilings (most of each tile inside the product)
    if (a.extA || 4 * a.Mg * a.Ng < 3 * tiles * PipeLarge::BM * PipeLarge::BN) return 0;
    const int64_t ktiles = (a.K + 63) / 64;
    int64_t s = std::min(kCUs / tiles, ktiles / kMinSplitKTiles);
    if (s < 2) return 0;
    const int64_t per = (ktiles + s - 1) / s;   // equal slices, none empty
    s = (ktiles + per - 1) / per;
    return s >= 2 && tiles * s >= kLargeFill ? s : 0;
}

// An unsplit product whose 256 x 256 tiles leave CUs idle takes 128 x 384
// tiles when those fill more CUs (at most one tile per CU, most of each tile
// inside the product): the MLP layer's 16384 x 768 input gradient has 192
// large tiles but 256 tall ones.
bool tall_fits(const GemmArgs& a) {
    const int64_t large = tiles_of(a, PipeLarge::BM, PipeLarge::BN), tall = tiles_of(a, PipeTall::BM, PipeTall::BN);
    return large < kCUs && tall > large && tall <= kCUs &&
           4 * a.Mg * a.Ng >= 3 * tall * PipeTall::BM * PipeTall::BN;
}

// The same split of K over 128 x 384 tiles (0 when it does not apply).  A
// product with few large tiles takes these when they need fewer splits: fewer
// int32 partials to write and sum (the MLP layer's wgrad, 3072 x 768 x 16384:
// 5 splits of 48 tall tiles instead of 7 of 36 large ones, 50.9 -> 47.8 us,
// the partial sums 13.3 -> 10.2 us).
int64_t tall_splits(const GemmArgs& a) {
    const int64_t tiles = tiles_of(a, PipeTall::BM, PipeTall::BN);
    if (tiles >= kCUs || a.extA || 4 * a.Mg * a.Ng < 3 * tiles * PipeTall::BM * PipeTall::BN) return 0;
    const int64_t ktiles = (a.K + 63) / 64;
    int64_t s = std::min(kCUs / tiles, ktiles / kMinSplitKTiles);
    if (s < 2) return 0;
    const int64_t per = (ktiles + s - 1) / s;
    return (ktiles + per - 1) / per;
}
bool tall_split_better(const GemmArgs& a) {
    if (a.K < 1024) return false;
    const int64_t ls = large_splits(a), ts = tall_splits(a);
    return ls > 1 && ts >= 2 && ts < ls;
}

Pick pick(const GemmArgs& a) {
    if (a.splits > 1 && tall_split_better(a) && a.splits == tall_splits(a)) return Pick::kTall;
    const int64_t ls = a.K >= 1024 ? large_splits(a) : 0;
    if (ls == 1 && a.splits <= 1 && tall_fits(a)) return Pick::kTall;
    if (ls > 0 && std::max(a.splits, 1) == ls) return Pick::kLarge;
    if (a.Mg <= 64 && !a.extA) return Pick::kSkinny;
    return Pick::kSmall;
}

}  // namespace

bool gemm_pipe_ok(const GemmArgs& a) { return pipe_ok(a); }

// Channel maxima of |x| per 32-row slab (bit patterns), for products the
// fused epilogue does not take: one thread per (slab, column), coalesced rows.
__global__ __launch_bounds__(256) void k_slab_colmax(const float* __restrict__ x, int64_t M, int64_t N, int64_t ld,
                                                     uint32_t* __restrict__ ranges) {
    const int64_t c = (int64_t)blockIdx.x * 256 + threadIdx.x, slab = blockIdx.y;
    if (c >= N) return;
    uint32_t mx = 0u;
    for (int64_t m = slab * 32; m < min(M, slab * 32 + 32); ++m) mx = max(mx, __float_as_uint(x[m * ld + c]) & 0x7FFFFFFFu);
    ranges[slab * N + c] = mx;
}

hipError_t launch_slab_colmax(const float* x, int64_t M, int64_t N, int64_t ld, uint32_t* ranges, hipStream_t s) {
    const int64_t slabs = (M + 31) / 32;
    if (slabs <= 0 || N <= 0) return hipSuccess;
    if (slabs > 65535) return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_slab_colmax, dim3((unsigned)((N + 255) / 256), (unsigned)slabs), dim3(256), 0, s, x, M, N, ld,
                       ranges);
    return hipGetLastError();
}

// Split-K factor of the weight-gradient product: large tiles with the split
// that fills the chip where that works (large_splits), else enough smaller
// tiles for about one block per CU with at least 8 K tiles per split and no
// empty split.  The partial tiles do not depend on the tile shape.
int wgrad_splits(int64_t M, int64_t C_out, int64_t C_in) {
    GemmArgs probe{};
    probe.Mg = C_out; probe.Ng = C_in; probe.K = M; probe.splits = 1;
    const int64_t ktiles = (M + 63) / 64;
    if (M >= 1024) {
        if (tall_split_better(probe)) return (int)tall_splits(probe);
        const int64_t ls = large_splits(probe);
        if (ls > 0) return (int)ls;
    }
    const bool skinny = C_out <= 64;
    const int64_t tiles = skinny ? tiles_of(probe, PipeSkinny::BM, PipeSkinny::BN)
                                 : tiles_of(probe, PipeSmall::BM, PipeSmall::BN);
    // about one block per CU: more splits only add partial tiles (measured on
    // the ResNet layers: 256 blocks beat 512 and 768 slightly, 128 clearly)
    int64_t splits = (256 + tiles - 1) / tiles;
    splits = std::min(splits, std::max<int64_t>(1, ktiles / 8));
    splits = std::max<int64_t>(1, std::min<int64_t>(splits, 65535));
    const int64_t per = (ktiles + splits - 1) / splits;
    return (int)((ktiles + per - 1) / per);
}

namespace {
// The product restricted to output rows [r0, Mg) (r0 a multiple of 256):
// every row-indexed pointer moves to row r0.
GemmArgs rows_from(const GemmArgs& a, int64_t r0) {
    GemmArgs b = a;
    auto row_ptr = [&](const int8_t* base, int64_t ld) {
        return a.tiled ? base + (r0 / 16) * (ld / 64) * 1024 : base + r0 * ld;
    };
    b.A = row_ptr(a.A, a.lda);
    if (a.extA) b.extA = row_ptr(a.extA, a.ld_extA);
    if (a.acc) b.acc = a.acc + r0 * a.ld_acc;
    if (a.out) b.out = a.out + r0 * a.ld_out;
    if (a.group && a.epi_mode == 1) b.group = a.group + r0;
    b.Mg = a.Mg - r0;
    return b;
}
}  // namespace

hipError_t launch_gemm(const GemmArgs& a, hipStream_t s) {
    if (a.Mg <= 0 || a.Ng <= 0) return hipSuccess;
    const bool pipe = pipe_ok(a);
    // tile-major operands: the pipelined kernel only, no convolution
    if (a.tiled && (!pipe || a.taps || a.kseg)) return hipErrorInvalidValue;
    if (a.kseg && (!pipe || a.splits > 1 || a.layout)) return hipErrorInvalidValue;   // pipelined kernel only
    const Pick p = pick(a);
    if (p == Pick::kLarge && pipe && a.splits <= 1 && !a.ranges && !a.part && !a.taps && !a.kseg) {
        // A last round of large tiles that would leave a quarter or more of
        // the CUs idle: the rows of the full rounds take the large tiles and
        // the remaining rows one round of smaller tiles (two launches).
        const int64_t tn = (a.Ng + PipeLarge::BN - 1) / PipeLarge::BN;
        const int64_t tiles = tn * ((a.Mg + PipeLarge::BM - 1) / PipeLarge::BM);
        const int64_t rounds = tiles / kCUs, rem = tiles - rounds * kCUs;
        const int64_t rows_main = (rounds * kCUs / tn) * PipeLarge::BM;
        if (rounds >= 1 && rem > 0 && 4 * rem <= 3 * kCUs && rows_main > 0 && rows_main < a.Mg) {
            GemmArgs m = a;
            m.Mg = rows_main;
            const hipError_t e = launch_gemm(m, s);
            if (e != hipSuccess) return e;
            return launch_gemm(rows_from(a, rows_main), s);
        }
    }
    const int64_t ktiles = (a.K + 63) / 64;   // every configuration has 64-byte K tiles
    const int splits = std::max(1, a.splits);
    const int64_t per = splits > 1 ? (ktiles + splits - 1) / splits : std::max<int64_t>(ktiles, 1);
    if (splits > 1 && (ktiles + per - 1) / per != splits) return hipErrorInvalidValue;   // wgrad_splits() avoids this
    if (a.ranges) {
        // dX with its channel maxima (producer-side ranges): pipelined kernel, no split
        if (!pipe || splits > 1 || !a.out || a.part) return hipErrorInvalidValue;
        if (p == Pick::kLarge)
            return a.extA ? launch_pipe<PipeLarge, true, false, true>(a, 1, per * 64, s)
                          : launch_pipe<PipeLarge, false, false, true>(a, 1, per * 64, s);
        if (p == Pick::kTall)
            return a.extA ? launch_pipe<PipeTall, true, false, true>(a, 1, per * 64, s)
                          : launch_pipe<PipeTall, false, false, true>(a, 1, per * 64, s);
        if (p == Pick::kSkinny) return launch_pipe<PipeSkinny, false, false, true>(a, 1, per * 64, s);
        return a.extA ? launch_pipe<PipeSmall, true, false, true>(a, 1, per * 64, s)
                      : launch_pipe<PipeSmall, false, false, true>(a, 1, per * 64, s);
    }
    if (p == Pick::kTall && pipe)
        return a.extA ? launch_pipe<PipeTall, true>(a, splits, per * 64, s)
                      : launch_pipe<PipeTall, false>(a, splits, per * 64, s);
    if (p == Pick::kLarge || p == Pick::kTall) {
        if (!pipe) return launch_cfg<CfgLarge>(a, splits, per * 64, s);
        return a.extA ? launch_pipe<PipeLarge, true>(a, splits, per * 64, s)
                      : launch_pipe<PipeLarge, false>(a, splits, per * 64, s);
    }
    if (!pipe) return launch_cfg<CfgSmall>(a, splits, per * 64, s);
    if (p == Pick::kSkinny) return launch_pipe<PipeSkinny, false>(a, splits, per * 64, s);
    return a.extA ? launch_pipe<PipeSmall, true>(a, splits, per * 64, s)
                  : launch_pipe<PipeSmall, false>(a, splits, per * 64, s);
}

// Padded pixel grids of the conv wgrad: a thread writes one aligned 16-byte
// chunk of an output row.  Its 16 grid positions lie in one grid row (Wp is a
// multiple of 16), so they map to a run of consecutive source pixels: two
// aligned 16-byte loads of the source row cover it, and v_alignbyte moves the
// run into place; bytes outside the content are cleared.
__global__ __launch_bounds__(256) void k_grid_pack(const int8_t* __restrict__ in, int64_t ld_in, uint32_t N,
                                                   uint32_t Hc, uint32_t Wc, uint32_t top, uint32_t left, uint32_t Hp,
                                                   uint32_t Wp, int8_t* __restrict__ out, int64_t ld_out,
                                                   uint32_t rows) {
    // every index fits 32 bits (the launcher checks): no 64-bit divisions
    const uint32_t chunks = (uint32_t)(ld_out / 16), img = Hp * Wp, total = rows * chunks;
    for (uint32_t id = blockIdx.x * blockDim.x + threadIdx.x; id < total; id += gridDim.x * blockDim.x) {
        const uint32_t c = id / chunks, G0 = (id - c * chunks) * 16;
        const uint32_t n = G0 / img, rem = G0 - n * img, hp = rem / Wp, wp0 = rem - hp * Wp;
        // grid bytes [e_lo, e_hi) of the chunk hold content pixels
        const int e_lo = (int)max(0, (int)left - (int)wp0), e_hi = (int)min(16, (int)(Wc + left) - (int)wp0);
        uint32_t o[4] = {0u, 0u, 0u, 0u};
        if (n < N && hp >= top && hp - top < Hc && e_lo < e_hi) {
            const int8_t* src = in + (int64_t)c * ld_in;
            // source index of grid byte 0 (before the row start when wp0 < left)
            const int64_t lo = (int64_t)((n * Hc + (hp - top)) * Wc) + (int64_t)wp0 - (int64_t)left;
            const int64_t a16 = lo >= 0 ? (lo & ~(int64_t)15) : -16;
            const int off = (int)(lo - a16);
            uint32_t w[8];
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int64_t at = a16 + 16 * h;
                uint4 v = make_uint4(0u, 0u, 0u, 0u);
                if (at >= 0 && at + 16 <= ld_in) v = *reinterpret_cast<const uint4*>(src + at);
                w[4 * h] = v.x; w[4 * h + 1] = v.y; w[4 * h + 2] = v.z; w[4 * h + 3] = v.w;
            }
            uint32_t sel[5];
            switch (off >> 2) {
                case 0: for (int i = 0; i < 5; ++i) sel[i] = w[i]; break;
                case 1: for (int i = 0; i < 5; ++i) sel[i] = w[i + 1]; break;
                case 2: for (int i = 0; i < 5; ++i) sel[i] = w[i + 2]; break;
                default: for (int i = 0; i < 5; ++i) sel[i] = w[i + 3]; break;
            }
            const uint32_t b = (uint32_t)(off & 3);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int lo_i = min(4, max(0, e_lo - 4 * i)), hi_i = min(4, max(0, e_hi - 4 * i));
                const uint32_t m = hi_i > lo_i ? (0xFFFFFFFFu >> (32 - 8 * (hi_i - lo_i))) << (8 * lo_i) : 0u;
                o[i] = __builtin_amdgcn_alignbyte(sel[i + 1], sel[i], b) & m;
            }
        }
        *reinterpret_cast<uint4*>(out + (int64_t)c * ld_out + G0) = make_uint4(o[0], o[1], o[2], o[3]);
    }
}

hipError_t launch_grid_pack(const int8_t* in, int64_t ld_in, int64_t C, int64_t N, int64_t Hc, int64_t Wc,
                            int64_t top, int64_t left, int64_t Hp, int64_t Wp, int8_t* out, int64_t ld_out,
                            hipStream_t s) {
    if (ld_out % 16 || ld_in % 16 || Wp % 16) return hipErrorInvalidValue;
    const int64_t work = C * (ld_out / 16);
    if (work <= 0) return hipSuccess;
    // 32-bit indices: chunks, grid positions and source pixels
    const int64_t lim = (int64_t)1 << 31;
    if (work >= lim || ld_out >= lim || N * Hp * Wp >= lim || N * Hc * Wc >= lim || C >= lim)
        return hipErrorInvalidValue;
    const dim3 grid((unsigned)std::min<int64_t>((work + 255) / 256, 16384));
    hipLaunchKernelGGL(k_grid_pack, grid, dim3(256), 0, s, in, ld_in, (uint32_t)N, (uint32_t)Hc, (uint32_t)Wc,
                       (uint32_t)top, (uint32_t)left, (uint32_t)Hp, (uint32_t)Wp, out, ld_out, (uint32_t)C);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Implicit-im2col weight gradient of a stride-1 convolution from one copy of
// the input codes on the padded pixel grid:
//   acc[co, (r KW + s) C_in + ci] = sum_P A[co, P] X[ci, P + r Wp + s],
// the third product of the im2col'd conv layer (Fig. "MMs"), whose im2col
// column of tap (r, s) is the grid shifted by r Wp + s bytes.
// A block owns FM x 16 output channels, 16 input channels and RB rows of taps
// (all KW columns of each) for one K split, and walks the split in chunks of
// 16 K tiles: per chunk it stages 1 KB of each of its A rows and 1280 bytes
// of each X row (the chunk and the halo of the row shifts) in a three-deep
// LDS ring, with direct loads whose lane offsets are fixed and whose K offset
// is a scalar.  Wave w of eight (two per SIMD; four for a runtime window)
// takes K tiles w, w + 8 of a chunk; per tile it reads FM A fragments and, per tap row, the 16-byte
// chunk of each X row plus the word after it, from which v_alignbyte forms
// the KW byte-shifted B fragments: one X read feeds KW x FM MFMAs.  Chunk q of an
// LDS row r sits at chunk (q & ~7) | ((q ^ r) & 7), so the 16 rows of a
// fragment read fall in 8 distinct bank groups.  At the end the waves'
// accumulators are summed in LDS and the block writes its tile: int32
// partials of its K split, or the outputs with the epilogue of the wgrad
// (dW[co, :] = fl(float(acc[co, :]) * fl(step_G step_X 2^-g_co))).
// ---------------------------------------------------------------------------
constexpr int kCwA = 1024, kCwX = 1280, kCwTiles = 16;
constexpr int kCwHalo = kCwX - kCwA - 64;   // largest (RB - 1) Wp a chunk's X rows cover

template <int FM, int KWC, int RBC>   // KWC / RBC: compile-time KW / tap rows, 0 = runtime (KW <= 16, RB <= 2)
struct CwCfg {
    // two waves per SIMD; the runtime-window variant (128 accumulator
    // registers) keeps one
    static constexpr int WAVES = KWC ? 8 : 4;
    static constexpr int KWM = KWC ? KWC : 16;
    static constexpr int RBM = RBC ? RBC : 2;
    static constexpr int NX = KWM == 1 ? 0 : (KWM <= 5 ? 1 : 4);   // words read after each X chunk
    static constexpr int kAbytes = 16 * FM * kCwA;
    static constexpr int kStage = kAbytes + 16 * kCwX;
    static constexpr int STAGES = FM == 1 && KWC ? 4 : 3;   // LDS ring depth (chunks)
    static constexpr int kSmem = STAGES * kStage;
    // DMA instructions per chunk: LA per wave for A; the NXI of the X rows
    // go to waves i % T::WAVES, LXM at most per wave
    static constexpr int LA = 16 * FM / WAVES, NXI = 16 * kCwX / 1024;
    static constexpr int LXM = (NXI + WAVES - 1) / WAVES;
    static_assert(LA * WAVES == 16 * FM && NXI * 1024 == 16 * kCwX, "whole DMA instructions");
    static_assert(2 * (LA + LXM) <= 63, "vmcnt range");
};

__device__ __forceinline__ int cw_phys(int q, int r) { return (q & ~7) | ((q ^ r) & 7); }

// s_waitcnt lgkmcnt(0) leaving vmcnt and expcnt unconstrained (gfx9 encoding)
__device__ __forceinline__ void wait_lgkm0() { __builtin_amdgcn_s_waitcnt(0xF | (0x7 << 4) | (0x3 << 14)); }

template <int FM, int KWC, int RBC>
__global__ __launch_bounds__((64 * CwCfg<FM, KWC, RBC>::WAVES)) void k_conv_wgrad(ConvWgradArgs p, ConvWgradPlan pl) {
#if defined(__HIP_DEVICE_COMPILE__)
    using T = CwCfg<FM, KWC, RBC>;
    __shared__ __attribute__((aligned(1024))) int8_t smem[T::kSmem];
    using MF = Mfma<16>;
    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    // (split, tile) items split-major, XCD x (blocks L = x mod 8) taking the
    // contiguous run after those of XCDs 0 .. x-1, as in k_gemm_pipe: the
    // tiles of a K split share its L2 whatever the number of splits
    const int64_t nt = pl.tiles, total = nt * pl.splits, L = blockIdx.x;
    const int64_t xcd = L & 7, jj = L >> 3;
    int64_t start = 0;
    for (int64_t y = 0; y < xcd; ++y) start += (total - y + 7) >> 3;
    const int64_t item = start + jj, split = item / nt, bt = item - split * nt;
    const int tg = (int)(bt % pl.tap_groups);
    const int64_t rest = bt / pl.tap_groups;
    const int64_t ci0 = (rest % pl.tiles_ci) * 16, co0 = (rest / pl.tiles_ci) * (16 * FM);
    const int KW = KWC ? KWC : p.KW;
    const int r0 = tg * pl.rb;
    const int nr = RBC ? RBC : min(pl.rb, p.KH - r0);
    const int64_t c_beg = split * pl.per;
    const int nch = (int)(min(pl.chunks, c_beg + pl.per) - c_beg);

    constexpr int kRsrcFlags = 0x00020000;   // raw byte buffer, gfx9 data format
    auto rsrc = [&](const int8_t* base, int64_t bytes) {
        return __builtin_amdgcn_make_buffer_rsrc(const_cast<int8_t*>(base), (short)0,
                                                 (int)min(bytes, (int64_t)0x7FFFFFFF), kRsrcFlags);
    };
    const __amdgpu_buffer_rsrc_t rA = rsrc(p.A, p.C_out * p.lda), rX = rsrc(p.X, p.C_in * p.ldx);
    // DMA: A instruction j of this wave fills LDS row w LA + j (1 KB); X
    // instruction j fills bytes [1 KB i, 1 KB (i + 1)) of the X rows, i = w LX + j.
    // Rows past C_out / C_in read the last row (never stored).
    uint32_t offA[T::LA], offX[T::LXM];
#pragma unroll
    for (int j = 0; j < T::LA; ++j) {
        const int row = w * T::LA + j;
        const int64_t g = min(co0 + row, p.C_out - 1);
        offA[j] = (uint32_t)(g * p.lda + 16 * cw_phys(lane, row & 15));
    }
    const int nxw = (T::NXI - w + T::WAVES - 1) / T::WAVES;   // X instructions of this wave
#pragma unroll
    for (int j = 0; j < T::LXM; ++j) {
        const int i = min(w + T::WAVES * j, T::NXI - 1);
        const int b = i * 1024 + 16 * lane, xr = b / kCwX, pc = (b - xr * kCwX) / 16;
        const int64_t g = min(ci0 + xr, p.C_in - 1);
        offX[j] = (uint32_t)(g * p.ldx + (int64_t)r0 * p.Wp + 16 * cw_phys(pc, xr & 15));
    }
    auto issue = [&](int c) {
        int8_t* st = smem + (c % T::STAGES) * T::kStage;
        const int k0 = (int)((c_beg + c) * kCwTiles * 64);
#pragma unroll
        for (int j = 0; j < T::LA; ++j)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rA, (lds_void_t*)(st + (w * T::LA + j) * kCwA), 16, offA[j], k0,
                                                     0, 0);
#pragma unroll
        for (int j = 0; j < T::LXM; ++j)
            if (j < nxw)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(rX, (lds_void_t*)(st + T::kAbytes + (w + T::WAVES * j) * 1024),
                                                         16, offX[j], k0, 0, 0);
    };
    // this wave's loads of chunk c are complete once only those of the
    // STAGES - 2 chunks issued after it remain
    auto wait_chunk = [&](int later) {   // chunks issued after chunk c (0 .. STAGES - 2)
        if (later <= 0) wait_vm<0>();
        else if (later == 1) {
            if (nxw == T::LXM) wait_vm<T::LA + T::LXM>();
            else wait_vm<T::LA + T::LXM - 1>();
        } else {
            if (nxw == T::LXM) wait_vm<2 * (T::LA + T::LXM)>();
            else wait_vm<2 * (T::LA + T::LXM - 1)>();
        }
    };

    // fragment reads: lane (row lr, 16-byte K chunk lc) of K tile 4 u + w reads
    // logical chunk 16 u + q0 of its row; cw_phys(16 u + q0) = 16 u + cw_phys(q0)
    const int lr = lane & 15, lc = lane >> 4;
    const int aoff = lr * kCwA + 16 * cw_phys(4 * w + lc, lr);
    int xo0[T::RBM], xo1[T::RBM];
#pragma unroll
    for (int rr = 0; rr < T::RBM; ++rr) {
        const int q0 = 4 * w + lc + rr * (int)(p.Wp / 16);
        xo0[rr] = T::kAbytes + lr * kCwX + 16 * cw_phys(q0, lr);
        xo1[rr] = T::kAbytes + lr * kCwX + 16 * cw_phys(q0 + 1, lr);
    }

    v4i acc[FM][T::RBM][T::KWM];
#pragma unroll
    for (int f = 0; f < FM; ++f)
#pragma unroll
        for (int rr = 0; rr < T::RBM; ++rr)
#pragma unroll
            for (int s = 0; s < T::KWM; ++s) acc[f][rr][s] = v4i{0, 0, 0, 0};

    // One chunk: the wave's K tiles w + T::WAVES u.  FULL: every tile lies
    // below K; else tiles past the end (last chunk) add nothing (A cleared).
    constexpr int NU = kCwTiles / T::WAVES;
    struct Frags {
        v4i a[FM];
        v4i x[T::RBM];
        uint32_t nx[T::RBM][T::NX ? T::NX : 1];
    };
    auto load = [&](Frags& F, const int8_t* st, int u) {
#pragma unroll
        for (int f = 0; f < FM; ++f) F.a[f] = *reinterpret_cast<const v4i*>(st + aoff + f * 16 * kCwA + 64 * T::WAVES * u);
#pragma unroll
        for (int rr = 0; rr < T::RBM; ++rr) {
            if (!RBC && rr >= nr) continue;
            F.x[rr] = *reinterpret_cast<const v4i*>(st + xo0[rr] + 64 * T::WAVES * u);
            if constexpr (T::NX == 1) {
                F.nx[rr][0] = *reinterpret_cast<const uint32_t*>(st + xo1[rr] + 64 * T::WAVES * u);
            } else if constexpr (T::NX == 4) {
                const v4i y = *reinterpret_cast<const v4i*>(st + xo1[rr] + 64 * T::WAVES * u);
                F.nx[rr][0] = (uint32_t)y.x; F.nx[rr][1] = (uint32_t)y.y;
                F.nx[rr][2] = (uint32_t)y.z; F.nx[rr][3] = (uint32_t)y.w;
            }
        }
    };
    auto process = [&](Frags& F, bool valid) {
        if (!valid)
#pragma unroll
            for (int f = 0; f < FM; ++f) F.a[f] = v4i{0, 0, 0, 0};
#pragma unroll
        for (int rr = 0; rr < T::RBM; ++rr) {
            if (!RBC && rr >= nr) continue;
            uint32_t wd[8] = {(uint32_t)F.x[rr].x, (uint32_t)F.x[rr].y, (uint32_t)F.x[rr].z, (uint32_t)F.x[rr].w,
                              0u, 0u, 0u, 0u};
#pragma unroll
            for (int i = 0; i < T::NX; ++i) wd[4 + i] = F.nx[rr][i];
#pragma unroll
            for (int s = 0; s < T::KWM; ++s) {
                if (!KWC && s >= KW) continue;
                const int d = s >> 2, sh = s & 3;
                v4i b;
                if (sh == 0) {
                    b = v4i{(int)wd[d], (int)wd[d + 1], (int)wd[d + 2], (int)wd[d + 3]};
                } else {
                    b = v4i{(int)__builtin_amdgcn_alignbyte(wd[d + 1], wd[d], sh),
                            (int)__builtin_amdgcn_alignbyte(wd[d + 2], wd[d + 1], sh),
                            (int)__builtin_amdgcn_alignbyte(wd[d + 3], wd[d + 2], sh),
                            (int)__builtin_amdgcn_alignbyte(wd[d + 4], wd[d + 3], sh)};
                }
#pragma unroll
                for (int f = 0; f < FM; ++f) acc[f][rr][s] = MF::run(b, F.a[f], acc[f][rr][s]);
            }
        }
    };
    auto compute = [&](const int8_t* st, int64_t kt0, auto FULL) {
#pragma unroll
        for (int u = 0; u < NU; ++u) {
            Frags F;
            load(F, st, u);
            process(F, decltype(FULL)::value || kt0 + T::WAVES * u + w < p.ktiles);
        }
    };

    // ring of STAGES chunks: chunk c + STAGES - 1 is issued once every wave
    // has passed the barrier that follows its reads of chunk c - 1 (same stage)
    for (int k = 0; k < T::STAGES - 1; ++k)
        if (k < nch) issue(k);
    for (int c = 0; c < nch; ++c) {
        wait_chunk(min(T::STAGES - 2, nch - 1 - c));
        wait_lgkm0();
        __builtin_amdgcn_s_barrier();
        if (c + T::STAGES - 1 < nch) issue(c + T::STAGES - 1);
        const int64_t kt0 = (c_beg + c) * kCwTiles;
        if (kt0 + kCwTiles <= p.ktiles) compute(smem + (c % T::STAGES) * T::kStage, kt0, std::true_type());
        else compute(smem + (c % T::STAGES) * T::kStage, kt0, std::false_type());
    }

    // Sum the waves' accumulators through LDS, a pass of up to TP tiles
    // (f, rr, s) at a time: each wave stores its 16 x 16 tiles as they sit
    // in its lanes (lane l: output channel l % 16, input channels
    // 4 (l / 16) .. + 3), one 1 KB row per tile; then item (tile, lane) of
    // the pass adds the WAVES rows and writes the 4 outputs.
    constexpr int NT = FM * T::RBM * T::KWM;
    constexpr int TP = NT < T::kSmem / (T::WAVES * 1024) ? NT : T::kSmem / (T::WAVES * 1024);
    static_assert(TP >= 1, "one tile per pass fits the ring");
    const int64_t Ng = (int64_t)p.KH * KW * p.C_in;
    const bool split_k = pl.splits > 1;
    float base = 0.0f;
    if (!split_k && p.out) base = __fmul_rn(p.gs->step, p.os->step);
    const bool vec4 = (p.C_in & 3) == 0;
    wait_lgkm0();
    __syncthreads();
#pragma unroll
    for (int t0 = 0; t0 < NT; t0 += TP) {
#pragma unroll
        for (int tl = t0; tl < min(NT, t0 + TP); ++tl) {
            const int f = tl / (T::RBM * T::KWM), rs = tl % (T::RBM * T::KWM), rr = rs / T::KWM, s = rs % T::KWM;
            if ((!RBC && rr >= nr) || (!KWC && s >= KW)) continue;
            *reinterpret_cast<v4i*>(smem + ((w * TP + (tl - t0)) * 64 + lane) * 16) = acc[f][rr][s];
        }
        __syncthreads();
        const int nt = min(NT, t0 + TP) - t0;
        for (int item = tid; item < nt * 64; item += 64 * T::WAVES) {
            const int tl = t0 + item / 64, l = item % 64;
            const int f = tl / (T::RBM * T::KWM), rs = tl % (T::RBM * T::KWM), rr = rs / T::KWM, s = rs % T::KWM;
            if (rr >= nr || s >= KW) continue;
            const int64_t co = co0 + f * 16 + (l & 15), ci = ci0 + 4 * (l >> 4);
            if (co >= p.C_out || ci >= p.C_in) continue;
            v4i sum = v4i{0, 0, 0, 0};
#pragma unroll
            for (int ww = 0; ww < T::WAVES; ++ww)
                sum += *reinterpret_cast<const v4i*>(smem + ((ww * TP + (tl - t0)) * 64 + l) * 16);
            const int nv = (int)min((int64_t)4, p.C_in - ci);
            const int64_t j = ((int64_t)(r0 + rr) * KW + s) * p.C_in + ci;
            const int vv[4] = {sum.x, sum.y, sum.z, sum.w};
            if (split_k) {
                int32_t* dst = p.part + ((int64_t)split * p.C_out + co) * Ng + j;
                if (vec4) *reinterpret_cast<v4i*>(dst) = sum;
                else
                    for (int e = 0; e < nv; ++e) dst[e] = vv[e];
                continue;
            }
            if (p.acc)
                for (int e = 0; e < nv; ++e) p.acc[co * p.ld_acc + j + e] = vv[e];
            if (p.out) {
                const float sc = __fmul_rn(base, pow2f(-(int)p.group[co]));
                for (int e = 0; e < nv; ++e) store_f1(p.out + co * p.ld_out + j + e, __fmul_rn((float)vv[e], sc), true);
            }
        }
        __syncthreads();
    }
#endif
}

ConvWgradPlan conv_wgrad_plan(int64_t K, int64_t C_out, int64_t C_in, int KH, int KW, int64_t Wp) {
    ConvWgradPlan pl;
    pl.fm = C_out > 16 ? 2 : 1;
    const bool three = KH == 3 && KW == 3 && 2 * Wp <= kCwHalo;
    if (three) {
        pl.kwc = 3;
        pl.rbc = 3;
        pl.rb = 3;
    } else {
        pl.fm = 1;   // runtime window: one fragment of output channels, at most 2 tap rows
        pl.rb = (int)std::max<int64_t>(1, std::min<int64_t>({(int64_t)KH, 2, 1 + kCwHalo / Wp}));
    }
    pl.tap_groups = (KH + pl.rb - 1) / pl.rb;
    pl.tiles_ci = (C_in + 15) / 16;
    pl.tiles = (C_out + 16 * pl.fm - 1) / (16 * pl.fm) * pl.tiles_ci * pl.tap_groups;
    const int64_t ktiles = (K + 63) / 64;
    pl.chunks = (ktiles + kCwTiles - 1) / kCwTiles;
    // about one block per CU; each split holds whole chunks and none is empty
    int64_t splits = std::max<int64_t>(1, (256 + pl.tiles / 2) / pl.tiles);
    splits = std::max<int64_t>(1, std::min(splits, pl.chunks));
    const int64_t per = std::max<int64_t>(1, (pl.chunks + splits - 1) / splits);
    pl.per = (int)per;
    pl.splits = (int)std::max<int64_t>(1, (pl.chunks + per - 1) / per);
    return pl;
}

hipError_t launch_conv_wgrad(const ConvWgradArgs& a, const ConvWgradPlan& pl, hipStream_t s) {
    if (a.C_out <= 0 || a.C_in <= 0 || pl.chunks <= 0) return hipSuccess;
    if (a.lda % 16 || a.ldx % 16 || a.Wp <= 0 || a.Wp % 16 || a.KH < 1 || a.KW < 1 || a.KW > 16 ||
        (int64_t)(pl.rb - 1) * a.Wp > kCwHalo || (pl.kwc && (pl.kwc != a.KW || pl.rbc != a.KH)) ||
        (!pl.kwc && (pl.fm != 1 || pl.rb > 2)))
        return hipErrorInvalidValue;
    if (pl.splits > 1 ? !a.part : (!a.acc && !a.out)) return hipErrorInvalidValue;
    // every byte offset (row, chunk, row shift, halo) fits the 31-bit buffer range
    const int64_t lim = (int64_t)1 << 31;
    if (a.C_out * a.lda >= lim || a.C_in * a.ldx >= lim ||
        a.C_in * a.ldx + pl.chunks * kCwTiles * 64 + (int64_t)a.KH * a.Wp + kCwX >= lim ||
        a.C_out * a.lda + pl.chunks * kCwTiles * 64 + kCwA >= lim)
        return hipErrorInvalidValue;
    const dim3 grid((unsigned)(pl.tiles * pl.splits));
    if (pl.kwc == 3 && pl.fm == 2)
        hipLaunchKernelGGL((k_conv_wgrad<2, 3, 3>), grid, dim3(64 * CwCfg<2, 3, 3>::WAVES), 0, s, a, pl);
    else if (pl.kwc == 3)
        hipLaunchKernelGGL((k_conv_wgrad<1, 3, 3>), grid, dim3(64 * CwCfg<1, 3, 3>::WAVES), 0, s, a, pl);
    else
        hipLaunchKernelGGL((k_conv_wgrad<1, 0, 0>), grid, dim3(64 * CwCfg<1, 0, 0>::WAVES), 0, s, a, pl);
    return hipGetLastError();
}

// B operand of the conv dgrad: bc[ci, t * 64 + e] for K tile t = f * taps + tau
// is column f * 64 + e of the fold's flat sequence (appended columns [0, H),
// main columns, appended columns [H, D)) for weight column (tau, ci): the W^T
// code of that column's channel, 0 for padding and for channels >= C_out.
__global__ void k_conv_gather_w(const int8_t* __restrict__ wq_t, int64_t ld_w, int64_t C_out, int64_t C_in, int taps,
                                const int32_t* __restrict__ layout, int8_t* __restrict__ bc, int64_t ld_bc) {
    const int64_t H = layout[kLayH], D = layout[kLayD], base = layout[kLayBase];
    const int32_t* ext = layout + kLayoutHeader;
    const int64_t ncols = (int64_t)taps * (base + D);
    for (int64_t ci = blockIdx.y; ci < C_in; ci += gridDim.y)
        for (int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; j < ncols; j += (int64_t)gridDim.x * blockDim.x) {
            const int64_t t = j / 64, f = t / taps, tau = t - f * taps;
            const int64_t k = f * 64 + j % 64;
            int64_t ch;
            if (k < H) ch = ext[k];
            else if (k < H + base) ch = k - H < C_out ? k - H : -1;
            else ch = ext[k - base];
            bc[ci * ld_bc + j] = ch >= 0 ? wq_t[(tau * C_in + ci) * ld_w + ch] : (int8_t)0;
        }
}

hipError_t launch_conv_gather_w(const int8_t* wq_t, int64_t ld_w, int64_t C_out, int64_t C_in, int taps,
                                const int32_t* layout, int8_t* bc, int64_t ld_bc, hipStream_t s) {
    if (C_in <= 0 || C_out <= 0) return hipSuccess;
    const dim3 grid((unsigned)std::min<int64_t>((ld_bc + 255) / 256, 64), (unsigned)std::min<int64_t>(C_in, 1024));
    hipLaunchKernelGGL(k_conv_gather_w, grid, dim3(256), 0, s, wq_t, ld_w, C_out, C_in, taps, layout, bc, ld_bc);
    return hipGetLastError();
}

// Conv dgrad: a.K is the main width of the fold (a multiple of 64), a.A /
// a.extA the main and appended columns of q_fold ([a_rows, lda]), a.B / a.ldb
// the W^T codes.  Same-size convolutions with one K chunk and a narrow output
// stream (k_conv_stream, weights straight from W^T); the others gather the
// weights into bc in the implicit GEMM's K order and take the window kernel
// (same size, small window) or the per-tap pipelined kernel.
hipError_t launch_conv_dgrad(const GemmArgs& a0, int8_t* bc, int64_t ld_bc, hipStream_t s, int64_t* range_rows) {
    if (a0.Mg <= 0 || a0.Ng <= 0) return hipSuccess;
    if (a0.ranges && (!a0.out || !range_rows)) return hipErrorInvalidValue;
    auto al16 = [](const void* q) { return (reinterpret_cast<uintptr_t>(q) & 15) == 0; };
    auto fits = [](int64_t rows, int64_t ld) { return rows * ld < ((int64_t)1 << 31); };
    if (a0.taps < 1 || a0.K % 64 != 0 || a0.lda % 16 != 0 || a0.ldb % 16 != 0 || !al16(a0.A) || !al16(a0.B) ||
        !fits(a0.a_rows, a0.lda) || !fits((int64_t)a0.taps * a0.Ng, a0.ldb) || a0.Mg > 0x7FFFFFFF)
        return hipErrorInvalidValue;
    if (a0.extA && (a0.ld_extA != a0.lda || !al16(a0.extA))) return hipErrorInvalidValue;
    const bool same = a0.cv_Ho == a0.cv_H && a0.cv_Wo == a0.cv_W;
    auto small_out = [](const void* q, int64_t rows, int64_t ld) {
        return !q || (((reinterpret_cast<uintptr_t>(q) & 15) == 0) && ld % 4 == 0 && rows * ld * 4 < ((int64_t)1 << 31));
    };
    if (same && !a0.extA && a0.K == 64 && a0.taps <= kHaloMaxTaps && (int64_t)a0.cv_PH * a0.cv_W + a0.cv_PW <= 64 &&
        a0.Ng <= 64 && a0.Ng % 4 == 0 && small_out(a0.out, a0.Mg, a0.ld_out) && small_out(a0.acc, a0.Mg, a0.ld_acc)) {
        // whole 128-row steps per block, at most kStreamBlocks blocks
        const int64_t rows = round_up((a0.Mg + kStreamBlocks - 1) / kStreamBlocks, 128);
        const dim3 grid((unsigned)((a0.Mg + rows - 1) / rows));
        const bool fullk = a0.K_used >= 64;   // every code column of the chunk is a channel
        if (a0.ranges) {
            // channel maxima per block: one slab of `rows` rows each
            *range_rows = rows;
            if (a0.acc && fullk) hipLaunchKernelGGL((k_conv_stream<true, true, true>), grid, dim3(256), 0, s, a0, rows);
            else if (a0.acc) hipLaunchKernelGGL((k_conv_stream<true, false, true>), grid, dim3(256), 0, s, a0, rows);
            else if (fullk) hipLaunchKernelGGL((k_conv_stream<false, true, true>), grid, dim3(256), 0, s, a0, rows);
            else hipLaunchKernelGGL((k_conv_stream<false, false, true>), grid, dim3(256), 0, s, a0, rows);
            return hipGetLastError();
        }
        if (a0.acc && fullk) hipLaunchKernelGGL((k_conv_stream<true, true>), grid, dim3(256), 0, s, a0, rows);
        else if (a0.acc) hipLaunchKernelGGL((k_conv_stream<true, false>), grid, dim3(256), 0, s, a0, rows);
        else if (fullk) hipLaunchKernelGGL((k_conv_stream<false, true>), grid, dim3(256), 0, s, a0, rows);
        else hipLaunchKernelGGL((k_conv_stream<false, false>), grid, dim3(256), 0, s, a0, rows);
        return hipGetLastError();
    }
    if (a0.ranges) {
        // the other conv kernels store dX, then one pass takes 32-row slab maxima
        if ((a0.Mg + 31) / 32 > 65535) return hipErrorInvalidValue;
        GemmArgs b = a0;
        b.ranges = nullptr;
        const hipError_t e = launch_conv_dgrad(b, bc, ld_bc, s, nullptr);
        if (e != hipSuccess) return e;
        *range_rows = 32;
        return launch_slab_colmax(a0.out, a0.Mg, a0.Ng, a0.ld_out, a0.ranges, s);
    }
    // weights in the K order of the implicit GEMM
    hipError_t e = launch_conv_gather_w(a0.B, a0.ldb, a0.K_used, a0.Ng, a0.taps, a0.layout, bc, ld_bc, s);
    if (e != hipSuccess) return e;
    GemmArgs a = a0;
    a.B = bc;
    a.ldb = ld_bc;
    if (!fits(a.Ng, a.ldb)) return hipErrorInvalidValue;
    const int64_t kps = a.K;
    if (same && a.taps <= kHaloMaxTaps && 2 * ((int64_t)a.cv_PH * a.cv_W + a.cv_PW) <= kHaloExtra) {
        const dim3 grid((unsigned)((a.Mg + kHaloBM - 1) / kHaloBM), (unsigned)((a.Ng + 63) / 64));
        if (grid.y > 65535) return hipErrorInvalidValue;
        if (a.extA) hipLaunchKernelGGL(k_conv_halo<true>, grid, dim3(64 * kHaloWaves), 0, s, a);
        else hipLaunchKernelGGL(k_conv_halo<false>, grid, dim3(64 * kHaloWaves), 0, s, a);
        return hipGetLastError();
    }
    if (a.Ng <= 64)
        return a.extA ? launch_pipe<PipeNarrow, true, true>(a, 1, kps, s) : launch_pipe<PipeNarrow, false, true>(a, 1, kps, s);
    return a.extA ? launch_pipe<PipeSmall, true, true>(a, 1, kps, s) : launch_pipe<PipeSmall, false, true>(a, 1, kps, s);
}

// ---------------------------------------------------------------------------
// GEMM-based implementation of ShiftQuant's loss propagation (Sec. 3.2), the
// comparison for ShiftMM: extract one pair of smaller matrices per group
// (memory rearrangement), multiply each pair with the GEMM, then shift the
// products by N_G - 1 - g and sum them.
// ---------------------------------------------------------------------------
int64_t grouped_width(int64_t C_out, int num_groups) { return round_up(C_out + 63 * (int64_t)num_groups, 64); }

// Group plan (one block): plan[2 g] = first rearranged column of group g
// (64-aligned), plan[2 g + 1] = its padded width; perm[j] (from plan[16]) =
// the channel at rearranged column j in ascending order within its group,
// -1 for padding; then, from plan[16 + wmax], the q_fold column of that
// channel's code and its fold shift t as (t << 24) | column (-1 for padding).
constexpr int kPlanThreads = 1024;
__global__ __launch_bounds__(kPlanThreads) void k_group_plan(const uint8_t* __restrict__ group, int64_t C, int ng,
                                                             const int32_t* __restrict__ desc, int64_t base_col,
                                                             int32_t* __restrict__ plan, int64_t wmax) {
    __shared__ int cnt[kMaxRegions], off[kMaxRegions], run[kMaxRegions];
    __shared__ int wcnt[kPlanThreads / 64][kMaxRegions];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    int32_t* perm = plan + 16;
    int32_t* acol = perm + wmax;
    if (tid < kMaxRegions) { cnt[tid] = 0; run[tid] = 0; }
    __syncthreads();
    int local[kMaxRegions] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int64_t c = tid; c < C; c += kPlanThreads) {
        const int g = group[c];
#pragma unroll
        for (int q = 0; q < kMaxRegions; ++q) local[q] += g == q;
    }
#pragma unroll
    for (int q = 0; q < kMaxRegions; ++q) {
        int v = local[q];
        for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
        if (lane == 0 && v) atomicAdd(&cnt[q], v);
    }
    __syncthreads();
    if (tid == 0) {
        int o = 0;
        for (int q = 0; q < ng; ++q) {
            off[q] = o;
            const int w = (cnt[q] + 63) / 64 * 64;
            plan[2 * q] = o;
            plan[2 * q + 1] = w;
            o += w;
        }
    }
    __syncthreads();
    for (int64_t j = tid; j < wmax; j += kPlanThreads) perm[j] = acol[j] = -1;
    __syncthreads();
    // ranks: rounds of kPlanThreads channels, wave ballots plus per-wave counts
    const uint64_t below = (1ull << lane) - 1ull;
    for (int64_t c0 = 0; c0 < C; c0 += kPlanThreads) {
        const int64_t c = c0 + tid;
        const int g = c < C ? (int)group[c] : -1;
        int rank = 0;
        for (int q = 0; q < ng; ++q) {
            const uint64_t m = __ballot(g == q);
            if (g == q) rank = __popcll(m & below);
            if (lane == 0) wcnt[wave][q] = __popcll(m);
        }
        __syncthreads();
        if (g >= 0) {
            int before = run[g];
            for (int w = 0; w < wave; ++w) before += wcnt[w][g];
            const int j = off[g] + before + rank;
            const int d = desc[c], t = d & 15, pos = (d >> 4) - 1;
            perm[j] = (int32_t)c;
            acol[j] = (t << 24) | (int32_t)(pos < 0 ? c : base_col + pos);
        }
        __syncthreads();
        if (tid < ng) {
            int tot = 0;
            for (int w = 0; w < kPlanThreads / 64; ++w) tot += wcnt[w][tid];
            run[tid] += tot;
        }
        __syncthreads();
    }
}

hipError_t launch_group_plan(const uint8_t* group, int64_t C, int num_groups, const int32_t* desc, int64_t base_col,
                             int32_t* plan, int64_t wmax, hipStream_t s) {
    hipLaunchKernelGGL(k_group_plan, dim3(1), dim3(kPlanThreads), 0, s, group, C, num_groups, desc, base_col, plan,
                       wmax);
    return hipGetLastError();
}

// dst[r, j] = src[r, col_j] >> t_j with col[j] = (t << 24) | column (-1:
// padding, 0), four output bytes per thread and 4 rows per block row.
__global__ __launch_bounds__(256) void k_gather_cols(const int8_t* __restrict__ src, int64_t ld_src, int64_t rows,
                                                     const int32_t* __restrict__ col, int64_t wmax,
                                                     int8_t* __restrict__ dst, int64_t ld_dst) {
    const int64_t j = ((int64_t)blockIdx.x * 64 + (threadIdx.x & 63)) * 4;
    if (j >= wmax) return;
    int sc[4], sh[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const int v = col[j + e];
        sc[e] = v < 0 ? -1 : (v & 0xFFFFFF);
        sh[e] = v < 0 ? 0 : (v >> 24);
    }
    for (int64_t r = (int64_t)blockIdx.y * 4 + (threadIdx.x >> 6); r < rows; r += (int64_t)gridDim.y * 4) {
        const int8_t* row = src + r * ld_src;
        uint32_t w = 0u;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int8_t v = sc[e] >= 0 ? (int8_t)(row[sc[e]] >> sh[e]) : (int8_t)0;
            w |= (uint32_t)(uint8_t)v << (8 * e);
        }
        *reinterpret_cast<uint32_t*>(dst + r * ld_dst + j) = w;
    }
}

hipError_t launch_gather_cols(const int8_t* src, int64_t ld_src, int64_t rows, const int32_t* col, int64_t wmax,
                              int8_t* dst, int64_t ld_dst, hipStream_t s) {
    if (rows <= 0 || wmax <= 0) return hipSuccess;
    if (wmax % 4 != 0 || ld_dst % 4 != 0) return hipErrorInvalidValue;
    const dim3 grid((unsigned)((wmax / 4 + 63) / 64), (unsigned)std::min<int64_t>((rows + 3) / 4, 16384));
    hipLaunchKernelGGL(k_gather_cols, grid, dim3(256), 0, s, src, ld_src, rows, col, wmax, dst, ld_dst);
    return hipGetLastError();
}

// acc = sum_g part[g] << (N_G - 1 - g); out = fl(float(acc) * alpha); four
// consecutive outputs per thread when N is a multiple of 4
__global__ void k_group_combine(const int32_t* __restrict__ part, int ng, int64_t M, int64_t N,
                                int32_t* __restrict__ acc, int64_t ld_acc, float* __restrict__ out, int64_t ld_out,
                                const sq_scale* __restrict__ gs, const sq_scale* __restrict__ os) {
    const float alpha = out ? __fmul_rn(__fmul_rn(gs->step, os->step), pow2f(-(ng - 1))) : 0.0f;
    const int64_t total = M * N;
    const int V = (N % 4 == 0) ? 4 : 1;
    for (int64_t i = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * V; i < total;
         i += (int64_t)gridDim.x * blockDim.x * V) {
        int32_t v[4] = {0, 0, 0, 0};
        for (int g = 0; g < ng; ++g) {
            if (V == 4) {
                const int4 q = *reinterpret_cast<const int4*>(part + g * total + i);
                const int s = ng - 1 - g;
                v[0] += (int32_t)((uint32_t)q.x << s); v[1] += (int32_t)((uint32_t)q.y << s);
                v[2] += (int32_t)((uint32_t)q.z << s); v[3] += (int32_t)((uint32_t)q.w << s);
            } else {
                v[0] += (int32_t)((uint32_t)part[g * total + i] << (ng - 1 - g));
            }
        }
        for (int e = 0; e < V; ++e) {
            const int64_t m = (i + e) / N, n = (i + e) - m * N;
            if (acc) acc[m * ld_acc + n] = v[e];
            if (out) out[m * ld_out + n] = __fmul_rn((float)v[e], alpha);
        }
    }
}

hipError_t launch_group_combine(const int32_t* part, int num_groups, int64_t M, int64_t N, int32_t* acc,
                                int64_t ld_acc, float* out, int64_t ld_out, const sq_scale* gs, const sq_scale* os,
                                hipStream_t s) {
    if (M <= 0 || N <= 0) return hipSuccess;
    const unsigned blocks = (unsigned)std::min<int64_t>((M * N + 255) / 256, 8192);
    hipLaunchKernelGGL(k_group_combine, dim3(blocks), dim3(256), 0, s, part, num_groups, M, N, acc, ld_acc, out, ld_out,
                       gs, os);
    return hipGetLastError();
}

hipError_t launch_gather_ext(const int8_t* wq_t, int64_t ld_w, int64_t C_in, const int32_t* layout,
                             int8_t* wext, int64_t ld_ext, int64_t ext_max, hipStream_t s, bool tiled) {
    if (C_in <= 0 || ext_max <= 0) return hipSuccess;
    if (tiled && (ld_w % 64 || ld_ext % 64)) return hipErrorInvalidValue;
    const unsigned blocks = (unsigned)std::min<int64_t>(C_in, 4096);
    hipLaunchKernelGGL(k_gather_ext, dim3(blocks), dim3(64), 0, s, wq_t, ld_w, C_in, layout, wext, ld_ext,
                       (int)tiled);
    return hipGetLastError();
}

hipError_t launch_splitk_reduce(const int32_t* ws, int splits, const GemmArgs& a, hipStream_t s) {
    if (a.Mg <= 0 || a.Ng <= 0) return hipSuccess;
    int lanes = 1;
    while (lanes < 16 && 4 * (2 * lanes) <= splits) lanes *= 2;
    const int items = kRedThreads / lanes;
    const int64_t groups = (a.Mg * a.Ng + 3) / 4;
    const int64_t blocks = (groups + items - 1) / items;
    if (blocks > 0x7FFFFFFF) return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_splitk_reduce, dim3((unsigned)blocks), dim3(kRedThreads), 0, s, ws, splits, lanes, a.Mg,
                       a.Ng, a.acc, a.ld_acc, a.out, a.ld_out, a.epi_mode, a.group, a.gs, a.os, a.num_groups);
    return hipGetLastError();
}

hipError_t launch_dequant(const int32_t* acc, int64_t rows, int64_t cols, int64_t ld_acc, int kind,
                          const uint8_t* group, const sq_scale* gs, const sq_scale* os, int num_groups,
                          float* out, int64_t ld_out, hipStream_t s) {
    if (rows <= 0 || cols <= 0) return hipSuccess;
    const unsigned blocks = (unsigned)std::min<int64_t>(rows, 8192);
    hipLaunchKernelGGL(k_dequant, dim3(blocks), dim3(256), 0, s, acc, rows, cols, ld_acc, kind, group, gs, os,
                       num_groups, out, ld_out);
    return hipGetLastError();
}

}  // namespace sq
