// Integer GEMMs of the ShiftQuant backward pass for gfx950.
//
// One kernel serves both products as C[i, j] = sum_k A[i, k] * B[j, k] with
// both operands K-contiguous int8:
//   dgrad: A = shift-folded gradient codes [M, C_out(+appended)],
//          B = W^T codes [C_in, C_out]              -> dX [M, C_in]
//   wgrad: A = transposed gradient codes [C_out, M],
//          B = X^T codes [C_in, M]                   -> dW [C_out, C_in]
// int32 accumulation on the matrix cores (v_mfma_i32_32x32x32_i8, 32x32
// outputs, K = 32 per instruction), 128x128 block tiles of four 64x64 wave
// tiles, K tiles of 64 bytes double-buffered in LDS.  The dequantization of
// Eq. "dq_mm_f" is fused into the epilogue.
//
// ShiftMM (Sec. 3.2) shifts every product by the shift of its inner index
// before accumulation.  The shifts that fit int8 are folded into the
// gradient codes by the quantizer; channels that need more are appended as
// extra K regions that this kernel visits first, doubling the accumulator at
// the start of each region (Horner's rule), so the result equals
// sum_c code * w << (N_G - 1 - g_c) exactly.
#include <algorithm>

#include "sq_internal.h"

namespace sq {

namespace {

constexpr int BM = 128, BN = 128, BK = 64;
constexpr int LS = BK + 16;   // LDS row stride in bytes: conflict-free 16-byte reads
constexpr int kThreads = 256;

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

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

__global__ __launch_bounds__(kThreads, 2) void k_gemm_i8(GemmArgs p, int tiles_n, int64_t k_per_split) {
    __shared__ __attribute__((aligned(16))) int8_t sA[2][BM * LS];
    __shared__ __attribute__((aligned(16))) int8_t sB[2][BN * LS];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int64_t tile = blockIdx.x;
    const int64_t m0 = (tile / tiles_n) * BM, n0 = (tile % tiles_n) * BN;

    // K tiles: appended regions first (dgrad fold), then this split's slice
    // of the main segment.
    int n_ext = 0, E = 0;
    const int32_t* rstart = nullptr;
    if (p.extA) {
        E = p.layout[0];
        n_ext = p.layout[1] / BK;
        rstart = p.layout + 4;
    }
    const int64_t kbeg = (int64_t)blockIdx.y * k_per_split;
    const int64_t kend = min(p.K, kbeg + k_per_split);
    const int n_main = kend > kbeg ? (int)((kend - kbeg + BK - 1) / BK) : 0;
    const int n_tiles = n_ext + n_main;

    v16i acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0;

    uint4 ra[2], rb[2];

    auto load = [&](int t) {
        const int8_t *Ab, *Bb;
        int64_t la, lb, k0, klim;
        if (t < n_ext) {
            Ab = p.extA; la = p.ld_extA; Bb = p.extB; lb = p.ld_extB;
            k0 = (int64_t)t * BK; klim = (int64_t)n_ext * BK;
        } else {
            Ab = p.A; la = p.lda; Bb = p.B; lb = p.ldb;
            k0 = kbeg + (int64_t)(t - n_ext) * BK; klim = kend;
        }
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int id = tid + i * kThreads;
            const int row = id >> 2, c16 = (id & 3) * 16;
            const int64_t kk = k0 + c16;
            uint4 va = make_uint4(0u, 0u, 0u, 0u), vb = make_uint4(0u, 0u, 0u, 0u);
            if (kk < klim) {
                const int64_t gm = m0 + row, gn = n0 + row;
                if (gm < p.Mg) va = *reinterpret_cast<const uint4*>(Ab + gm * la + kk);
                if (gn < p.Ng) vb = *reinterpret_cast<const uint4*>(Bb + gn * lb + kk);
                if (kk + 16 > klim) {
                    va = mask_tail(va, (int)(klim - kk));
                    vb = mask_tail(vb, (int)(klim - kk));
                }
            }
            ra[i] = va;
            rb[i] = vb;
        }
    };
    auto store = [&](int buf) {
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int id = tid + i * kThreads;
            const int row = id >> 2, c16 = (id & 3) * 16;
            *reinterpret_cast<uint4*>(&sA[buf][row * LS + c16]) = ra[i];
            *reinterpret_cast<uint4*>(&sB[buf][row * LS + c16]) = rb[i];
        }
    };
    auto compute = [&](int buf) {
#pragma unroll
        for (int ks = 0; ks < BK / 32; ++ks) {
            v4i a[2], b[2];
            const int kb = ks * 32 + (lane >> 5) * 16;
#pragma unroll
            for (int wi = 0; wi < 2; ++wi)
                a[wi] = *reinterpret_cast<const v4i*>(&sA[buf][(wm * 64 + wi * 32 + (lane & 31)) * LS + kb]);
#pragma unroll
            for (int wj = 0; wj < 2; ++wj)
                b[wj] = *reinterpret_cast<const v4i*>(&sB[buf][(wn * 64 + wj * 32 + (lane & 31)) * LS + kb]);
            // The B tile feeds the matrix-core A operand, so each lane's
            // results run along the output row (4 consecutive columns per
            // register quartet).
#pragma unroll
            for (int wi = 0; wi < 2; ++wi)
#pragma unroll
                for (int wj = 0; wj < 2; ++wj)
                    acc[wi][wj] = __builtin_amdgcn_mfma_i32_32x32x32_i8(b[wj], a[wi], acc[wi][wj], 0, 0, 0);
        }
    };

    if (n_tiles > 0) {
        load(0);
        store(0);
        __syncthreads();
        int next_region = 0;
        for (int t = 0; t < n_tiles; ++t) {
            if (t + 1 < n_tiles) load(t + 1);
            if (next_region < E && t < n_ext && (int64_t)t * BK == rstart[next_region]) {
                // Horner step: the accumulated regions weigh twice the next one
#pragma unroll
                for (int i = 0; i < 2; ++i)
#pragma unroll
                    for (int j = 0; j < 2; ++j) acc[i][j] = acc[i][j] + acc[i][j];
                ++next_region;
            }
            compute(t & 1);
            if (t + 1 < n_tiles) store((t + 1) & 1);
            __syncthreads();
        }
    }

    // ---- epilogue ----
    float base = 0.0f, alpha = 0.0f;
    if (p.out && !p.part) {
        const sq_scale gs = *p.gs, os = *p.os;
        base = __fmul_rn(gs.step, os.step);
        alpha = __fmul_rn(base, pow2f(-(p.num_groups - 1)));
    }
    const bool vec_acc = p.acc && ((p.ld_acc & 3) == 0) && ((reinterpret_cast<uintptr_t>(p.acc) & 15) == 0);
    const bool vec_out = p.out && ((p.ld_out & 3) == 0) && ((reinterpret_cast<uintptr_t>(p.out) & 15) == 0);
    const bool vec_part = p.part && ((p.Ng & 3) == 0) && ((reinterpret_cast<uintptr_t>(p.part) & 15) == 0);
#pragma unroll
    for (int wi = 0; wi < 2; ++wi) {
        const int64_t ii = m0 + wm * 64 + wi * 32 + (lane & 31);
        if (ii >= p.Mg) continue;
        float sc = alpha;
        if (p.out && p.epi_mode == 1) sc = __fmul_rn(base, pow2f(-(int)p.group[ii]));
#pragma unroll
        for (int wj = 0; wj < 2; ++wj) {
#pragma unroll
            for (int a4 = 0; a4 < 4; ++a4) {
                const int64_t jj = n0 + wn * 64 + wj * 32 + a4 * 8 + (lane >> 5) * 4;
                if (jj >= p.Ng) continue;
                const int v0 = acc[wi][wj][a4 * 4 + 0], v1 = acc[wi][wj][a4 * 4 + 1];
                const int v2 = acc[wi][wj][a4 * 4 + 2], v3 = acc[wi][wj][a4 * 4 + 3];
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
                    const float f0 = __fmul_rn((float)v0, sc), f1 = __fmul_rn((float)v1, sc);
                    const float f2 = __fmul_rn((float)v2, sc), f3 = __fmul_rn((float)v3, sc);
                    if (vec_out && full) {
                        *reinterpret_cast<float4*>(dst) = make_float4(f0, f1, f2, f3);
                    } else {
                        const float ff[4] = {f0, f1, f2, f3};
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            if (jj + e < p.Ng) dst[e] = ff[e];
                    }
                }
            }
        }
    }
}

// Appended B columns of the dgrad fold: wext[k, j] = W^T code of the channel
// the layout lists for appended column j (0 for padding).
__global__ void k_gather_ext(const int8_t* __restrict__ wq_t, int64_t ld_w, int64_t C_in,
                             const int32_t* __restrict__ layout, int8_t* __restrict__ wext, int64_t ld_ext) {
    const int D = layout[1];
    const int32_t* ext = layout + kLayoutHeader;
    for (int64_t k = blockIdx.x; k < C_in; k += gridDim.x)
        for (int j = threadIdx.x; j < D; j += blockDim.x) {
            const int ch = ext[j];
            wext[k * ld_ext + j] = ch >= 0 ? wq_t[k * ld_w + ch] : (int8_t)0;
        }
}

// Sum of the split-K partial tiles ws [splits, Mg, Ng] (int32 addition is
// exact and order-free), then the same epilogue as the GEMM.
__global__ void k_splitk_reduce(const int32_t* __restrict__ ws, int splits, int64_t Mg, int64_t Ng,
                                int32_t* __restrict__ acc, int64_t ld_acc, float* __restrict__ out, int64_t ld_out,
                                int epi_mode, const uint8_t* __restrict__ group, const sq_scale* __restrict__ gs,
                                const sq_scale* __restrict__ os, int num_groups) {
    const int64_t plane = Mg * Ng;
    float base = 0.0f, alpha = 0.0f;
    if (out) {
        base = __fmul_rn(gs->step, os->step);
        alpha = __fmul_rn(base, pow2f(-(num_groups - 1)));
    }
    const bool vec = ((Ng & 3) == 0);
    const int64_t n_items = vec ? plane / 4 : plane;
    for (int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; q < n_items;
         q += (int64_t)gridDim.x * blockDim.x) {
        if (vec) {
            const int64_t e = q * 4;
            int4 a[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) a[u] = make_int4(0, 0, 0, 0);
            int s = 0;
            for (; s + 4 <= splits; s += 4) {
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const int4 v = *reinterpret_cast<const int4*>(ws + (int64_t)(s + u) * plane + e);
                    a[u].x += v.x; a[u].y += v.y; a[u].z += v.z; a[u].w += v.w;
                }
            }
            for (; s < splits; ++s) {
                const int4 v = *reinterpret_cast<const int4*>(ws + (int64_t)s * plane + e);
                a[0].x += v.x; a[0].y += v.y; a[0].z += v.z; a[0].w += v.w;
            }
            const int t[4] = {a[0].x + a[1].x + a[2].x + a[3].x, a[0].y + a[1].y + a[2].y + a[3].y,
                              a[0].z + a[1].z + a[2].z + a[3].z, a[0].w + a[1].w + a[2].w + a[3].w};
            const int64_t i = e / Ng, j = e % Ng;
            if (acc) {
#pragma unroll
                for (int u = 0; u < 4; ++u) acc[i * ld_acc + j + u] = t[u];
            }
            if (out) {
                const float sc = epi_mode == 1 ? __fmul_rn(base, pow2f(-(int)group[i])) : alpha;
#pragma unroll
                for (int u = 0; u < 4; ++u) out[i * ld_out + j + u] = __fmul_rn((float)t[u], sc);
            }
        } else {
            int t = 0;
            for (int s = 0; s < splits; ++s) t += ws[(int64_t)s * plane + q];
            const int64_t i = q / Ng, j = q % Ng;
            if (acc) acc[i * ld_acc + j] = t;
            if (out) {
                const float sc = epi_mode == 1 ? __fmul_rn(base, pow2f(-(int)group[i])) : alpha;
                out[i * ld_out + j] = __fmul_rn((float)t, sc);
            }
        }
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
        for (int64_t c = threadIdx.x; c < cols; c += blockDim.x)
            out[r * ld_out + c] = __fmul_rn((float)acc[r * ld_acc + c], sc);
    }
}

}  // namespace

int wgrad_splits(int64_t M, int64_t C_out, int64_t C_in) {
    const int64_t tiles = ((C_out + BM - 1) / BM) * ((C_in + BN - 1) / BN);
    const int64_t ktiles = (M + BK - 1) / BK;
    int64_t splits = (512 + tiles - 1) / tiles;
    splits = min(splits, std::max<int64_t>(1, ktiles / 8));
    splits = std::max<int64_t>(1, std::min<int64_t>(splits, 65535));
    // no empty splits
    const int64_t per = (ktiles + splits - 1) / splits;
    return (int)((ktiles + per - 1) / per);
}

hipError_t launch_gemm(const GemmArgs& a, hipStream_t s) {
    if (a.Mg <= 0 || a.Ng <= 0) return hipSuccess;
    const int64_t tiles_m = (a.Mg + BM - 1) / BM, tiles_n = (a.Ng + BN - 1) / BN;
    if (tiles_m * tiles_n > 0x7FFFFFFF) return hipErrorInvalidValue;
    const int64_t ktiles = (a.K + BK - 1) / BK;
    int splits = std::max(1, a.splits);
    const int64_t per = splits > 1 ? (ktiles + splits - 1) / splits : std::max<int64_t>(ktiles, 1);
    const int64_t k_per_split = per * BK;
    if (splits > 1) splits = (int)((ktiles + per - 1) / per);
    if (splits != std::max(1, a.splits)) return hipErrorInvalidValue;   // wgrad_splits() avoids this
    dim3 grid((unsigned)(tiles_m * tiles_n), (unsigned)splits);
    hipLaunchKernelGGL(k_gemm_i8, grid, dim3(kThreads), 0, s, a, (int)tiles_n, k_per_split);
    return hipGetLastError();
}

hipError_t launch_gather_ext(const int8_t* wq_t, int64_t ld_w, int64_t C_in, const int32_t* layout,
                             int8_t* wext, int64_t ld_ext, int64_t ext_max, hipStream_t s) {
    if (C_in <= 0 || ext_max <= 0) return hipSuccess;
    const unsigned blocks = (unsigned)std::min<int64_t>(C_in, 4096);
    hipLaunchKernelGGL(k_gather_ext, dim3(blocks), dim3(64), 0, s, wq_t, ld_w, C_in, layout, wext, ld_ext);
    return hipGetLastError();
}

hipError_t launch_splitk_reduce(const int32_t* ws, int splits, const GemmArgs& a, hipStream_t s) {
    if (a.Mg <= 0 || a.Ng <= 0) return hipSuccess;
    const int64_t items = (a.Ng & 3) == 0 ? a.Mg * a.Ng / 4 : a.Mg * a.Ng;
    const unsigned blocks = (unsigned)std::min<int64_t>((items + 255) / 256, 2048);
    hipLaunchKernelGGL(k_splitk_reduce, dim3(blocks), dim3(256), 0, s, ws, splits, a.Mg, a.Ng, a.acc, a.ld_acc,
                       a.out, a.ld_out, a.epi_mode, a.group, a.gs, a.os, a.num_groups);
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
