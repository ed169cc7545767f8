// extern "C" entry points of libshiftquant: synchronous argument checks,
// workspace carving and stream-ordered kernel launches.  The semantics of
// every call are documented in include/shiftquant.h.
#include <algorithm>
#include <cstdint>
#include <cstring>
#include <mutex>
#include <string>

#include "sq_internal.h"

#define SQ_TRY(expr)                      \
    do {                                  \
        const sq_status st__ = (expr);    \
        if (st__ != SQ_OK) return st__;   \
    } while (0)

namespace sq {

QuantCfg make_cfg(const sq_quant_params& p) {
    QuantCfg c;
    c.bits = p.bits;
    c.Q = (1 << (p.bits - 1)) - 1;
    c.num_groups = p.num_groups;
    int T = 0;
    while (c.Q * (1 << (T + 1)) <= 127) ++T;
    c.T = T;
    c.round_mode = p.round_mode;
    c.seed = p.seed;
    c.offset = p.offset;
    return c;
}

int64_t fold_ext_max(int64_t C, const QuantCfg& c) {
    if (c.num_groups - 1 <= c.T) return 0;   // one window holds every shift
    return round_up(C, kFoldPad) + (int64_t)kFoldPad * (c.num_groups - 1);
}

}  // namespace sq

namespace {

using namespace sq;

thread_local std::string g_last_error;

constexpr int64_t kMaxRows = (int64_t)1 << 31;      // rows of any operand
constexpr int64_t kMaxChannels = (int64_t)1 << 20;  // C_out, C_in, cols

sq_status fail(sq_status s, const std::string& msg) {
    g_last_error = msg;
    return s;
}

sq_status hip_status(hipError_t e, const char* what) {
    if (e == hipSuccess) return SQ_OK;
    return fail(SQ_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

sq_status check_params(const sq_quant_params* p) {
    if (!p) return fail(SQ_ERR_INVALID_ARGUMENT, "params is NULL");
    if (p->bits < 2 || p->bits > 8) return fail(SQ_ERR_INVALID_ARGUMENT, "bits must be in [2, 8]");
    if (p->num_groups < 1 || p->num_groups > 8)
        return fail(SQ_ERR_INVALID_ARGUMENT, "num_groups must be in [1, 8]");
    if (p->round_mode != SQ_ROUND_NEAREST_EVEN && p->round_mode != SQ_ROUND_STOCHASTIC)
        return fail(SQ_ERR_INVALID_ARGUMENT, "round_mode must be SQ_ROUND_NEAREST_EVEN or SQ_ROUND_STOCHASTIC");
    if (p->layout != SQ_LAYOUT_ROWS && p->layout != SQ_LAYOUT_TILED)
        return fail(SQ_ERR_INVALID_ARGUMENT, "layout must be SQ_LAYOUT_ROWS or SQ_LAYOUT_TILED");
    return SQ_OK;
}

bool tiled_of(const sq_quant_params* p) { return p->layout == SQ_LAYOUT_TILED; }

// entry points that take row-major code matrices only
sq_status rows_only(const sq_quant_params* p, const char* fn) {
    if (p->layout != SQ_LAYOUT_ROWS)
        return fail(SQ_ERR_UNSUPPORTED, std::string(fn) + " takes row-major codes only (SQ_LAYOUT_ROWS)");
    return SQ_OK;
}

// int8 code matrix [rows, ld] with ld >= min_ld, 16-byte aligned, ld % 16 == 0
sq_status check_codes(const void* q, int64_t ld, int64_t min_ld, const char* name) {
    if (!q) return fail(SQ_ERR_INVALID_ARGUMENT, std::string(name) + " is NULL");
    if (!aligned(q, 16)) return fail(SQ_ERR_INVALID_ARGUMENT, std::string(name) + " must be 16-byte aligned");
    if (ld < min_ld || ld % 16 != 0)
        return fail(SQ_ERR_INVALID_ARGUMENT, std::string("ld of ") + name + " must be a multiple of 16 and >= " +
                                                 std::to_string(min_ld));
    return SQ_OK;
}

// the same for a code matrix in either layout; tile-major: ld a multiple of
// 64 covering min_ld rounded up to 64 (the K padding the kernels write)
sq_status check_codes_l(const void* q, int64_t ld, int64_t min_ld, bool tiled, const char* name) {
    SQ_TRY(check_codes(q, ld, tiled ? round_up(min_ld, 64) : min_ld, name));
    if (tiled && ld % 64 != 0)
        return fail(SQ_ERR_INVALID_ARGUMENT, std::string("ld of ") + name + " must be a multiple of 64 (SQ_LAYOUT_TILED)");
    return SQ_OK;
}

sq_status check_f32(const void* p, int64_t ld, int64_t min_ld, const char* name) {
    if (!p) return fail(SQ_ERR_INVALID_ARGUMENT, std::string(name) + " is NULL");
    if (!aligned(p, 4)) return fail(SQ_ERR_INVALID_ARGUMENT, std::string(name) + " must be 4-byte aligned");
    if (ld < min_ld) return fail(SQ_ERR_INVALID_ARGUMENT, std::string("ld of ") + name + " is smaller than its row");
    return SQ_OK;
}

sq_status check_dims(int64_t rows, int64_t cols, const char* what) {
    if (rows < 0 || cols < 0 || rows >= kMaxRows || cols >= kMaxChannels)
        return fail(SQ_ERR_INVALID_ARGUMENT, std::string("dimensions of ") + what + " out of range");
    return SQ_OK;
}

// quantizer scratch: slab maxima [slabs, C] followed by the channel ranges [C]
size_t quant_ws_bytes(int64_t M, int64_t C) { return (size_t)round_up(std::max<int64_t>(colmax_workspace_words(M, C), 1) * 4, 256); }


// Scratch of sq_quantize_grad_noalloc: a fixed device array instead of a
// caller-provided workspace, for callers that cannot allocate.  Each GPU the
// library runs on holds its own copy until the process ends; host code uses
// the address hipGetSymbolAddress reports for the current device, never the
// array's name.  Every call on one GPU shares it.
constexpr size_t kNoAllocScratchBytes = (size_t)1 << 20;
static __device__ __align__(256) uint8_t scratch[kNoAllocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The device address of this GPU's scratch, looked up once per device (with
// that device current) and kept.
sq_status noalloc_scratch(void** out) {
    int dev = -1;
    SQ_TRY(hip_status(hipGetDevice(&dev), "hipGetDevice"));
    if (dev < 0 || dev >= kMaxDevices) return fail(SQ_ERR_UNSUPPORTED, "device index beyond the scratch table");
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* ptr = nullptr;
        SQ_TRY(hip_status(hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)), "hipGetSymbolAddress(scratch)"));
        if (!ptr || !aligned(ptr, 256)) return fail(SQ_ERR_HIP, "scratch symbol has no usable device address");
        g_scratch_ptr[dev] = ptr;
    }
    *out = g_scratch_ptr[dev];
    return SQ_OK;
}

// argument checks of the gradient quantizer shared by both entry points
// (everything but the workspace), made before any HIP call
sq_status check_quantize_grad(const float* dY, int64_t M, int64_t C_out, int64_t ld_dY, const sq_quant_params* p,
                              const int8_t* q_fold, int64_t ld_fold, const int8_t* q_t, int64_t ld_t,
                              const uint8_t* group, const sq_scale* scale, const int32_t* layout) {
    SQ_TRY(check_params(p));
    SQ_TRY(check_dims(M, C_out, "dY"));
    if (M > 0 && C_out > 0) SQ_TRY(check_f32(dY, ld_dY, C_out, "dY"));
    if (!scale || !aligned(scale, 4)) return fail(SQ_ERR_INVALID_ARGUMENT, "scale is NULL or misaligned");
    if (!layout || !aligned(layout, 4)) return fail(SQ_ERR_INVALID_ARGUMENT, "layout is NULL or misaligned");
    if (C_out > 0 && !group) return fail(SQ_ERR_INVALID_ARGUMENT, "group is NULL");
    size_t lay_bytes = 0;
    int64_t min_ld_fold = 0;
    SQ_TRY(sq_grad_layout_size(C_out, p, &lay_bytes, &min_ld_fold));
    if (q_fold && M > 0) SQ_TRY(check_codes_l(q_fold, ld_fold, min_ld_fold, tiled_of(p), "q_fold"));
    if (q_t && C_out > 0) SQ_TRY(check_codes_l(q_t, ld_t, M > 0 ? M : 1, tiled_of(p), "q_t"));
    return SQ_OK;
}

// the gradient quantizer's launches, arguments already checked
sq_status quantize_grad_impl(const float* dY, int64_t M, int64_t C_out, int64_t ld_dY, const sq_quant_params* p,
                             int8_t* q_fold, int64_t ld_fold, int8_t* q_t, int64_t ld_t, uint8_t* group,
                             sq_scale* scale, int32_t* layout, void* workspace, size_t workspace_bytes,
                             void* stream) {
    if (!workspace || !aligned(workspace, 16)) return fail(SQ_ERR_INVALID_ARGUMENT, "workspace is NULL or misaligned");
    if (workspace_bytes < quant_ws_bytes(M, C_out)) return fail(SQ_ERR_WORKSPACE_TOO_SMALL, "workspace too small");

    const QuantCfg cfg = make_cfg(*p);
    hipStream_t s = static_cast<hipStream_t>(stream);
    uint32_t* partial = static_cast<uint32_t*>(workspace);
    const int64_t ext_max = fold_ext_max(C_out, cfg);
    SQ_TRY(hip_status(launch_colmax_finalize_grad(dY, M, C_out, ld_dY, cfg, partial, group, scale, layout, ext_max, s),
                      "abs-max and finalize"));
    SQ_TRY(hip_status(launch_quantize(dY, M, C_out, ld_dY, group, scale, cfg, q_fold, ld_fold, q_t, ld_t,
                                      layout + kLayoutHeader + ext_max, s, PadGrid(), tiled_of(p)),
                      "quantize"));
    return SQ_OK;
}

}  // namespace

using namespace sq;

extern "C" {

const char* sq_status_string(sq_status s) {
    switch (s) {
        case SQ_OK: return "SQ_OK";
        case SQ_ERR_INVALID_ARGUMENT: return "SQ_ERR_INVALID_ARGUMENT";
        case SQ_ERR_OVERFLOW_RISK: return "SQ_ERR_OVERFLOW_RISK";
        case SQ_ERR_UNSUPPORTED: return "SQ_ERR_UNSUPPORTED";
        case SQ_ERR_WORKSPACE_TOO_SMALL: return "SQ_ERR_WORKSPACE_TOO_SMALL";
        case SQ_ERR_HIP: return "SQ_ERR_HIP";
    }
    return "SQ_ERR_UNKNOWN";
}

const char* sq_last_error(void) { return g_last_error.c_str(); }
const char* sq_last_error_string(void) { return g_last_error.c_str(); }

sq_status sq_grad_layout_size(int64_t C_out, const sq_quant_params* p, size_t* layout_bytes, int64_t* min_ld_fold) {
    SQ_TRY(check_params(p));
    SQ_TRY(check_dims(0, C_out, "gradient"));
    if (!layout_bytes || !min_ld_fold) return fail(SQ_ERR_INVALID_ARGUMENT, "output pointer is NULL");
    const QuantCfg cfg = make_cfg(*p);
    const int64_t ext = fold_ext_max(C_out, cfg);
    *layout_bytes = (size_t)fold_layout_words(C_out, cfg) * sizeof(int32_t);
    *min_ld_fold = ext > 0 ? fold_ext_base(C_out) + ext : round_up(C_out > 0 ? C_out : 1, 16);
    return SQ_OK;
}

sq_status sq_quantize_grad_workspace_size(int64_t M, int64_t C_out, const sq_quant_params* p, size_t* bytes) {
    SQ_TRY(check_params(p));
    SQ_TRY(check_dims(M, C_out, "gradient"));
    if (!bytes) return fail(SQ_ERR_INVALID_ARGUMENT, "bytes is NULL");
    *bytes = quant_ws_bytes(M, C_out);
    return SQ_OK;
}

sq_status sq_quantize_tensor_workspace_size(int64_t rows, int64_t cols, size_t* bytes) {
    SQ_TRY(check_dims(rows, cols, "tensor"));
    if (!bytes) return fail(SQ_ERR_INVALID_ARGUMENT, "bytes is NULL");
    *bytes = quant_ws_bytes(rows, cols);
    return SQ_OK;
}

sq_status sq_gemm_dgrad_workspace_size(int64_t M, int64_t C_out, int64_t C_in, const sq_quant_params* p,
                                       size_t* bytes) {
    SQ_TRY(check_params(p));
    SQ_TRY(check_dims(M, C_out, "gradient"));
    SQ_TRY(check_dims(C_in, C_in, "weight"));
    if (!bytes) return fail(SQ_ERR_INVALID_ARGUMENT, "bytes is NULL");
    const QuantCfg cfg = make_cfg(*p);
    // gathered W^T columns of the appended windows [C_in, ext_max] (whole
    // 16-row groups when tile-major)
    const int64_t rows = tiled_of(p) ? round_up(C_in, 16) : C_in;
    *bytes = (size_t)round_up(rows * fold_ext_max(C_out, cfg), 256);
    return SQ_OK;
}

sq_status sq_gemm_wgrad_workspace_size(int64_t M, int64_t C_out, int64_t C_in, const sq_quant_params* p,
                                       size_t* bytes) {
    SQ_TRY(check_params(p));
    SQ_TRY(check_dims(M, C_out, "gradient"));
    SQ_TRY(check_dims(C_in, C_in, "activation"));
    if (!bytes) return fail(SQ_ERR_INVALID_ARGUMENT, "bytes is NULL");
    const int splits = (M > 0 && C_out > 0 && C_in > 0) ? wgrad_splits(M, C_out, C_in) : 1;
    *bytes = splits > 1 ? (size_t)round_up((int64_t)splits * C_out * C_in * 4, 256) : 0;
    return SQ_OK;
}

sq_status sq_quantize_grad(const float* dY, int64_t M, int64_t C_out, int64_t ld_dY, const sq_quant_params* p,
                           int8_t* q_fold, int64_t ld_fold, int8_t* q_t, int64_t ld_t, uint8_t* group,
                           sq_scale* scale, int32_t* layout, void* workspace, size_t workspace_bytes,
                           void* stream) {
    SQ_TRY(check_quantize_grad(dY, M, C_out, ld_dY, p, q_fold, ld_fold, q_t, ld_t, group, scale, layout));
    return quantize_grad_impl(dY, M, C_out, ld_dY, p, q_fold, ld_fold, q_t, ld_t, group, scale, layout, workspace,
                              workspace_bytes, stream);
}

sq_status sq_quantize_grad_noalloc(const float* dY, int64_t M, int64_t C_out, int64_t ld_dY,
                                   const sq_quant_params* p, int8_t* q_fold, int64_t ld_fold, int8_t* q_t,
                                   int64_t ld_t, uint8_t* group, sq_scale* scale, int32_t* layout, void* stream) {
    SQ_TRY(check_quantize_grad(dY, M, C_out, ld_dY, p, q_fold, ld_fold, q_t, ld_t, group, scale, layout));
    const size_t need = quant_ws_bytes(M, C_out);
    if (need > kNoAllocScratchBytes)
        return fail(SQ_ERR_WORKSPACE_TOO_SMALL,
                    "sq_quantize_grad_noalloc: this gradient needs " + std::to_string(need) +
                        " bytes of scratch, above the library's fixed " + std::to_string(kNoAllocScratchBytes) +
                        "; call sq_quantize_grad with a workspace instead");
    void* ws = nullptr;
    SQ_TRY(noalloc_scratch(&ws));
    return quantize_grad_impl(dY, M, C_out, ld_dY, p, q_fold, ld_fold, q_t, ld_t, group, scale, layout, ws,
                              kNoAllocScratchBytes, stream);
}

sq_status sq_quantize_tensor(const float* T, int64_t rows, int64_t cols, int64_t ld, int32_t bits, int32_t transpose,
                             int8_t* q, int64_t ld_q, sq_scale* scale, void* workspace, size_t workspace_bytes,
                             void* stream) {
    SQ_TRY(check_dims(rows, cols, "tensor"));
    if (bits < 2 || bits > 8) return fail(SQ_ERR_INVALID_ARGUMENT, "bits must be in [2, 8]");
    if (transpose < 0 || transpose > 2) return fail(SQ_ERR_INVALID_ARGUMENT, "transpose must be 0, 1 or 2");
    if (rows > 0 && cols > 0) {
        SQ_TRY(check_f32(T, ld, cols, "T"));
        SQ_TRY(check_codes_l(q, ld_q, transpose ? rows : cols, transpose == 2, "q"));
    }
    if (!scale || !aligned(scale, 4)) return fail(SQ_ERR_INVALID_ARGUMENT, "scale is NULL or misaligned");
    if (!workspace || !aligned(workspace, 16)) return fail(SQ_ERR_INVALID_ARGUMENT, "workspace is NULL or misaligned");
    if (workspace_bytes < quant_ws_bytes(rows, cols)) return fail(SQ_ERR_WORKSPACE_TOO_SMALL, "workspace too small");

    sq_quant_params p{};
    p.bits = bits;
    p.num_groups = 1;
    p.round_mode = SQ_ROUND_NEAREST_EVEN;
    const QuantCfg cfg = make_cfg(p);
    hipStream_t s = static_cast<hipStream_t>(stream);
    uint32_t* partial = static_cast<uint32_t*>(workspace);
    int64_t slabs = 0;
    SQ_TRY(hip_status(launch_colmax(T, rows, cols, ld, partial, &slabs, s), "colmax"));
    SQ_TRY(hip_status(launch_finalize_tensor(partial, slabs, cols, cfg.Q, partial + slabs * cols, scale, s),
                      "finalize"));
    SQ_TRY(hip_status(launch_quantize(T, rows, cols, ld, nullptr, scale, cfg, transpose ? nullptr : q, ld_q,
                                      transpose ? q : nullptr, ld_q, nullptr, s, PadGrid(), transpose == 2),
                      "quantize"));
    return SQ_OK;
}

namespace {
sq_status gemm_dgrad_impl(const int8_t* q_fold, int64_t ld_fold, const int32_t* layout, const uint8_t* group,
                          const sq_scale* gscale, const int8_t* wq_t, int64_t ld_w, const sq_scale* wscale, int64_t M,
                          int64_t C_out, int64_t C_in, const sq_quant_params* p, int32_t* acc, int64_t ld_acc,
                          float* dX, int64_t ld_dX, uint32_t* ranges, void* workspace, size_t workspace_bytes,
                          void* stream) {
    SQ_TRY(check_params(p));
    SQ_TRY(check_dims(M, C_out, "gradient codes"));
    SQ_TRY(check_dims(C_in, C_in, "weight codes"));
    if (!acc && !dX) return fail(SQ_ERR_INVALID_ARGUMENT, "acc and dX are both NULL");
    if (!layout || !gscale || !wscale) return fail(SQ_ERR_INVALID_ARGUMENT, "layout or a scale is NULL");
    const QuantCfg cfg = make_cfg(*p);
    // worst case |acc| = C_out * Q * 2^(N_G-1) * 128 must stay below 2^31
    const double bound = (double)C_out * cfg.Q * (double)(1 << (cfg.num_groups - 1)) * 128.0;
    if (bound >= 2147483648.0)
        return fail(SQ_ERR_OVERFLOW_RISK, "C_out * Q * 2^(N_G-1) * 128 reaches 2^31: the int32 accumulator could overflow");
    if (M == 0 || C_in == 0) return SQ_OK;
    size_t lay_bytes = 0;
    int64_t min_ld_fold = 0;
    SQ_TRY(sq_grad_layout_size(C_out, p, &lay_bytes, &min_ld_fold));
    const bool tiled = tiled_of(p);
    SQ_TRY(check_codes_l(q_fold, ld_fold, min_ld_fold, tiled, "q_fold"));
    SQ_TRY(check_codes_l(wq_t, ld_w, C_out > 0 ? C_out : 1, tiled, "wq_t"));
    if (acc) SQ_TRY(check_f32(acc, ld_acc, C_in, "acc"));
    if (dX) SQ_TRY(check_f32(dX, ld_dX, C_in, "dX"));
    const int64_t ext_max = fold_ext_max(C_out, cfg);
    size_t need = 0;
    SQ_TRY(sq_gemm_dgrad_workspace_size(M, C_out, C_in, p, &need));
    if (need > 0) {
        if (!workspace || !aligned(workspace, 16)) return fail(SQ_ERR_INVALID_ARGUMENT, "workspace is NULL or misaligned");
        if (workspace_bytes < need) return fail(SQ_ERR_WORKSPACE_TOO_SMALL, "workspace too small");
    }
    hipStream_t s = static_cast<hipStream_t>(stream);

    GemmArgs a{};
    a.Mg = M; a.Ng = C_in;
    a.A = q_fold; a.lda = ld_fold;
    a.B = wq_t; a.ldb = ld_w;
    // tile-major: K runs over the zero-padded main columns [0, roundup(C_out, 64))
    a.K = tiled ? round_up(C_out, 64) : C_out;
    a.tiled = tiled;
    a.layout = layout;
    if (ext_max > 0) {
        int8_t* wext = static_cast<int8_t*>(workspace);
        SQ_TRY(hip_status(launch_gather_ext(wq_t, ld_w, C_in, layout, wext, ext_max, ext_max, s, tiled), "gather"));
        a.extA = tiled ? q_fold : q_fold + fold_ext_base(C_out); a.ld_extA = ld_fold;
        a.ext_koff = tiled ? fold_ext_base(C_out) : 0;
        a.extB = wext; a.ld_extB = ext_max;
    }
    if (tiled && !gemm_pipe_ok(a)) return fail(SQ_ERR_UNSUPPORTED, "tile-major operands past 31-bit offsets");
    a.splits = 1;
    a.acc = acc; a.ld_acc = ld_acc;
    a.out = dX; a.ld_out = ld_dX;
    a.epi_mode = 0;
    a.gs = gscale; a.os = wscale; a.group = group; a.num_groups = cfg.num_groups;
    if (ranges && !gemm_pipe_ok(a)) {
        // the register-staged kernel (C_out not a multiple of 64, or operands
        // past 31-bit offsets) stores dX, then one pass takes its slab maxima
        if ((M + 31) / 32 > 65535) return fail(SQ_ERR_UNSUPPORTED, "dX ranges support at most 2^21 rows here");
        SQ_TRY(hip_status(launch_gemm(a, s), "gemm_dgrad"));
        return hip_status(launch_slab_colmax(dX, M, C_in, ld_dX, ranges, s), "dX ranges");
    }
    a.ranges = ranges;
    return hip_status(launch_gemm(a, s), "gemm_dgrad");
}
}  // namespace

sq_status sq_gemm_dgrad(const int8_t* q_fold, int64_t ld_fold, const int32_t* layout, const uint8_t* group,
                        const sq_scale* gscale, const int8_t* wq_t, int64_t ld_w, const sq_scale* wscale, int64_t M,
                        int64_t C_out, int64_t C_in, const sq_quant_params* p, int32_t* acc, int64_t ld_acc,
                        float* dX, int64_t ld_dX, void* workspace, size_t workspace_bytes, void* stream) {
    return gemm_dgrad_impl(q_fold, ld_fold, layout, group, gscale, wq_t, ld_w, wscale, M, C_out, C_in, p, acc, ld_acc,
                           dX, ld_dX, nullptr, workspace, workspace_bytes, stream);
}

sq_status sq_gemm_dgrad_range_slabs(int64_t M, int64_t* slabs) {
    if (!slabs) return fail(SQ_ERR_INVALID_ARGUMENT, "slabs is NULL");
    if (M < 0 || M >= kMaxRows) return fail(SQ_ERR_INVALID_ARGUMENT, "M out of range");
    *slabs = (M + 31) / 32;
    return SQ_OK;
}

sq_status sq_gemm_dgrad_ranged(const int8_t* q_fold, int64_t ld_fold, const int32_t* layout, const uint8_t* group,
                               const sq_scale* gscale, const int8_t* wq_t, int64_t ld_w, const sq_scale* wscale,
                               int64_t M, int64_t C_out, int64_t C_in, const sq_quant_params* p, int32_t* acc,
                               int64_t ld_acc, float* dX, int64_t ld_dX, uint32_t* dX_ranges, void* workspace,
                               size_t workspace_bytes, void* stream) {
    if (!dX) return fail(SQ_ERR_INVALID_ARGUMENT, "dX is NULL (the ranges are taken of dX)");
    if (!dX_ranges || !aligned(dX_ranges, 4)) return fail(SQ_ERR_INVALID_ARGUMENT, "dX_ranges is NULL or misaligned");
    return gemm_dgrad_impl(q_fold, ld_fold, layout, group, gscale, wq_t, ld_w, wscale, M, C_out, C_in, p, acc, ld_acc,
                           dX, ld_dX, dX_ranges, workspace, workspace_bytes, stream);
}

sq_status sq_quantize_channels_workspace_size(int64_t rows, int64_t cols, int32_t axis, size_t* bytes) {
    SQ_TRY(check_dims(rows, cols, "tensor"));
    if (axis != 0 && axis != 1) return fail(SQ_ERR_INVALID_ARGUMENT, "axis must be 0 (rows) or 1 (columns)");
    if (!bytes) return fail(SQ_ERR_INVALID_ARGUMENT, "bytes is NULL");
    *bytes = axis == 1 ? quant_ws_bytes(rows, cols) : 0;
    return SQ_OK;
}

sq_status sq_quantize_channels(const float* T, int64_t rows, int64_t cols, int64_t ld, int32_t bits, int32_t axis,
                               int32_t transpose, int8_t* q, int64_t ld_q, sq_scale* scales, void* workspace,
                               size_t workspace_bytes, void* stream) {
    SQ_TRY(check_dims(rows, cols, "tensor"));
    if (bits < 2 || bits > 8) return fail(SQ_ERR_INVALID_ARGUMENT, "bits must be in [2, 8]");
    if (axis != 0 && axis != 1) return fail(SQ_ERR_INVALID_ARGUMENT, "axis must be 0 (rows) or 1 (columns)");
    if (transpose != 0 && transpose != 1) return fail(SQ_ERR_INVALID_ARGUMENT, "transpose must be 0 or 1");
    if (rows == 0 || cols == 0) return SQ_OK;
    SQ_TRY(check_f32(T, ld, cols, "T"));
    SQ_TRY(check_codes(q, ld_q, transpose ? rows : cols, "q"));
    if (!scales || !aligned(scales, 4)) return fail(SQ_ERR_INVALID_ARGUMENT, "scales is NULL or misaligned");
    size_t need = 0;
    SQ_TRY(sq_quantize_channels_workspace_size(rows, cols, axis, &need));
    if (need > 0) {
        if (!workspace || !aligned(workspace, 16)) return fail(SQ_ERR_INVALID_ARGUMENT, "workspace is NULL or misaligned");
        if (workspace_bytes < need) return fail(SQ_ERR_WORKSPACE_TOO_SMALL, "workspace too small");
    }
    return hip_status(launch_quantize_channels(T, rows, cols, ld, bits, axis, transpose, q, ld_q, scales,
                                               static_cast<uint32_t*>(workspace), static_cast<hipStream_t>(stream)),
                      "quantize_channels");
}

sq_status sq_gemm_forward(const int8_t* xq_fold, int64_t ld_fold, const int32_t* layout, const uint8_t* group,
                          const sq_scale* xscale, const int8_t* wq, int64_t ld_w, const sq_scale* wscales, int64_t M,
                          int64_t C_in, int64_t C_out, const sq_quant_params* p, int32_t* acc, int64_t ld_acc,
                          float* Y, int64_t ld_Y, void* workspace, size_t workspace_bytes, void* stream) {
    SQ_TRY(check_params(p));
    SQ_TRY(rows_only(p, "sq_gemm_forward"));
    SQ_TRY(check_dims(M, C_in, "activation codes"));
    SQ_TRY(check_dims(C_out, C_out, "weight codes"));
    if (!acc && !Y) return fail(SQ_ERR_INVALID_ARGUMENT, "acc and Y are both NULL");
    if (!layout || !xscale || !wscales) return fail(SQ_ERR_INVALID_ARGUMENT, "layout or a scale is NULL");
    const QuantCfg cfg = make_cfg(*p);
    const double bound = (double)C_in * cfg.Q * (double)(1 << (cfg.num_groups - 1)) * 128.0;
    if (bound >= 2147483648.0)
        return fail(SQ_ERR_OVERFLOW_RISK, "C_in * Q * 2^(N_G-1) * 128 reaches 2^31: the int32 accumulator could overflow");
    if (M == 0 || C_out == 0) return SQ_OK;
    size_t lay_bytes = 0;
    int64_t min_ld_fold = 0;
    SQ_TRY(sq_grad_layout_size(C_in, p, &lay_bytes, &min_ld_fold));
    SQ_TRY(check_codes(xq_fold, ld_fold, min_ld_fold, "xq_fold"));
    SQ_TRY(check_codes(wq, ld_w, C_in > 0 ? C_in : 1, "wq"));
    if (acc) SQ_TRY(check_f32(acc, ld_acc, C_out, "acc"));
    if (Y) SQ_TRY(check_f32(Y, ld_Y, C_out, "Y"));
    const int64_t ext_max = fold_ext_max(C_in, cfg);
    size_t need = 0;
    SQ_TRY(sq_gemm_dgrad_workspace_size(M, C_in, C_out, p, &need));
    if (need > 0) {
        if (!workspace || !aligned(workspace, 16)) return fail(SQ_ERR_INVALID_ARGUMENT, "workspace is NULL or misaligned");
        if (workspace_bytes < need) return fail(SQ_ERR_WORKSPACE_TOO_SMALL, "workspace too small");
    }
    hipStream_t s = static_cast<hipStream_t>(stream);
    GemmArgs a{};
    a.Mg = M; a.Ng = C_out;
    a.A = xq_fold; a.lda = ld_fold;
    a.B = wq; a.ldb = ld_w;
    a.K = C_in;
    a.layout = layout;
    if (ext_max > 0) {
        int8_t* wext = static_cast<int8_t*>(workspace);
        SQ_TRY(hip_status(launch_gather_ext(wq, ld_w, C_out, layout, wext, ext_max, ext_max, s), "gather"));
        a.extA = xq_fold + fold_ext_base(C_in); a.ld_extA = ld_fold;
        a.extB = wext; a.ld_extB = ext_max;
    }
    a.splits = 1;
    a.acc = acc; a.ld_acc = ld_acc;
    a.out = Y; a.ld_out = ld_Y;
    a.epi_mode = 2;
    a.gs = xscale; a.os = wscales; a.group = group; a.num_groups = cfg.num_groups;
    return hip_status(launch_gemm(a, s), "gemm_forward");
}

static int64_t grouped_ws_parts(int64_t M, int64_t C_out, int64_t C_in, const QuantCfg& cfg, int64_t* off_a,
                                 int64_t* off_b, int64_t* off_p) {
    const int64_t wmax = grouped_width(C_out, cfg.num_groups);
    *off_a = round_up(4 * (16 + 2 * wmax), 256);
    *off_b = *off_a + round_up(M * wmax, 256);
    *off_p = *off_b + round_up(C_in * wmax, 256);
    return *off_p + round_up((int64_t)cfg.num_groups * M * C_in * 4, 256);
}

sq_status sq_gemm_dgrad_grouped_workspace_size(int64_t M, int64_t C_out, int64_t C_in, const sq_quant_params* p,
                                               size_t* bytes) {
    SQ_TRY(check_params(p));
    SQ_TRY(check_dims(M, C_out, "gradient"));
    SQ_TRY(check_dims(C_in, C_in, "weight"));
    if (!bytes) return fail(SQ_ERR_INVALID_ARGUMENT, "bytes is NULL");
    int64_t a, b, c;
    *bytes = (size_t)grouped_ws_parts(M, C_out, C_in, make_cfg(*p), &a, &b, &c);
    return SQ_OK;
}

sq_status sq_gemm_dgrad_grouped(const int8_t* q_fold, int64_t ld_fold, const int32_t* layout, const uint8_t* group,
                                const sq_scale* gscale, const int8_t* wq_t, int64_t ld_w, const sq_scale* wscale,
                                int64_t M, int64_t C_out, int64_t C_in, const sq_quant_params* p, int32_t* acc,
                                int64_t ld_acc, float* dX, int64_t ld_dX, void* workspace, size_t workspace_bytes,
                                void* stream) {
    SQ_TRY(check_params(p));
    SQ_TRY(rows_only(p, "sq_gemm_dgrad_grouped"));
    SQ_TRY(check_dims(M, C_out, "gradient codes"));
    SQ_TRY(check_dims(C_in, C_in, "weight codes"));
    if (!acc && !dX) return fail(SQ_ERR_INVALID_ARGUMENT, "acc and dX are both NULL");
    if (!layout || !gscale || !wscale) return fail(SQ_ERR_INVALID_ARGUMENT, "layout or a scale is NULL");
    const QuantCfg cfg = make_cfg(*p);
    const double bound = (double)C_out * cfg.Q * (double)(1 << (cfg.num_groups - 1)) * 128.0;
    if (bound >= 2147483648.0)
        return fail(SQ_ERR_OVERFLOW_RISK, "C_out * Q * 2^(N_G-1) * 128 reaches 2^31: the int32 accumulator could overflow");
    if (M == 0 || C_in == 0) return SQ_OK;
    size_t lay_bytes = 0;
    int64_t min_ld_fold = 0;
    SQ_TRY(sq_grad_layout_size(C_out, p, &lay_bytes, &min_ld_fold));
    const bool tiled = tiled_of(p);
    SQ_TRY(check_codes_l(q_fold, ld_fold, min_ld_fold, tiled, "q_fold"));
    SQ_TRY(check_codes_l(wq_t, ld_w, C_out > 0 ? C_out : 1, tiled, "wq_t"));
    if (acc) SQ_TRY(check_f32(acc, ld_acc, C_in, "acc"));
    if (dX) SQ_TRY(check_f32(dX, ld_dX, C_in, "dX"));
    int64_t off_a, off_b, off_p;
    const int64_t need = grouped_ws_parts(M, C_out, C_in, cfg, &off_a, &off_b, &off_p);
    if (!workspace || !aligned(workspace, 256)) return fail(SQ_ERR_INVALID_ARGUMENT, "workspace is NULL or not 256-byte aligned");
    if (workspace_bytes < (size_t)need) return fail(SQ_ERR_WORKSPACE_TOO_SMALL, "workspace too small");
    if (M * grouped_width(C_out, cfg.num_groups) >= ((int64_t)1 << 31) ||
        C_in * grouped_width(C_out, cfg.num_groups) >= ((int64_t)1 << 31))
        return fail(SQ_ERR_UNSUPPORTED, "grouped dgrad: a rearranged operand spans 2^31 bytes or more");
    hipStream_t s = static_cast<hipStream_t>(stream);
    int8_t* ws = static_cast<int8_t*>(workspace);
    int32_t* plan = reinterpret_cast<int32_t*>(ws);
    int8_t* A_r = ws + off_a;
    int8_t* B_r = ws + off_b;
    int32_t* part = reinterpret_cast<int32_t*>(ws + off_p);
    const int64_t wmax = grouped_width(C_out, cfg.num_groups);
    const int32_t* desc = layout + kLayoutHeader + fold_ext_max(C_out, cfg);
    // 1. memory rearrangement: the channels of each group side by side
    SQ_TRY(hip_status(launch_group_plan(group, C_out, cfg.num_groups, desc, fold_ext_base(C_out), plan, wmax, s),
                      "group_plan"));
    // codes: q_fold column and fold shift per rearranged column; weights: the channel itself
    SQ_TRY(hip_status(launch_gather_cols(q_fold, ld_fold, M, plan + 16 + wmax, wmax, A_r, wmax, s), "rearrange codes"));
    SQ_TRY(hip_status(launch_gather_cols(wq_t, ld_w, C_in, plan + 16, wmax, B_r, wmax, s), "rearrange weights"));
    // 2. one GEMM per group over its columns
    for (int g = 0; g < cfg.num_groups; ++g) {
        GemmArgs a{};
        a.Mg = M; a.Ng = C_in;
        a.A = A_r; a.lda = wmax;
        a.B = B_r; a.ldb = wmax;
        a.K = wmax;
        a.kseg = plan + 2 * g;
        a.splits = 1;
        a.acc = part + (int64_t)g * M * C_in; a.ld_acc = C_in;
        a.gs = gscale; a.os = wscale; a.group = group; a.num_groups = cfg.num_groups;
        SQ_TRY(hip_status(launch_gemm(a, s), "group gemm"));
    }
    // 3. shift and sum
    return hip_status(launch_group_combine(part, cfg.num_groups, M, C_in, acc, ld_acc, dX, ld_dX, gscale, wscale, s),
                      "group_combine");
}

static sq_status check_conv(int64_t N, int64_t H, int64_t W, int64_t C_out, int64_t C_in, int32_t KH, int32_t KW,
                            int32_t PH, int32_t PW) {
    if (N < 0 || H < 1 || W < 1 || C_out < 0 || C_in < 0)
        return fail(SQ_ERR_INVALID_ARGUMENT, "conv: need N >= 0, H, W >= 1, C_out, C_in >= 0");
    if (KH < 1 || KW < 1 || KH > 15 || KW > 15 || PH < 0 || PW < 0 || PH >= KH || PW >= KW)
        return fail(SQ_ERR_INVALID_ARGUMENT, "conv: need 1 <= KH, KW <= 15 and 0 <= PH < KH, 0 <= PW < KW");
    if (H + 2 * (int64_t)PH - KH + 1 < 1 || W + 2 * (int64_t)PW - KW + 1 < 1)
        return fail(SQ_ERR_INVALID_ARGUMENT, "conv: the window is larger than the padded input");
    if (N * H * W > 0x7FFFFFFF) return fail(SQ_ERR_UNSUPPORTED, "conv: more than 2^31 - 1 input pixels");
    return SQ_OK;
}

sq_status sq_conv_dgrad_workspace_size(int64_t C_out, int64_t C_in, int32_t KH, int32_t KW, const sq_quant_params* p,
                                       size_t* bytes) {
    SQ_TRY(check_params(p));
    SQ_TRY(check_dims(C_out, C_in, "conv weight"));
    if (KH < 1 || KW < 1 || KH > 15 || KW > 15) return fail(SQ_ERR_INVALID_ARGUMENT, "conv: need 1 <= KH, KW <= 15");
    if (!bytes) return fail(SQ_ERR_INVALID_ARGUMENT, "bytes is NULL");
    const QuantCfg cfg = make_cfg(*p);
    *bytes = (size_t)round_up(C_in * conv_bc_ld(C_out, (int64_t)KH * KW, fold_ext_max(C_out, cfg)), 256);
    return SQ_OK;
}

static sq_status conv_dgrad_impl(const int8_t* q_fold, int64_t ld_fold, const int32_t* layout, const uint8_t* group,
                                 const sq_scale* gscale, const int8_t* wq_t, int64_t ld_w, const sq_scale* wscale,
                                 int64_t N, int64_t H, int64_t W, int64_t C_out, int64_t C_in, int32_t KH, int32_t KW,
                                 int32_t PH, int32_t PW, const sq_quant_params* p, int32_t* acc, int64_t ld_acc,
                                 float* dX, int64_t ld_dX, uint32_t* ranges, int64_t* range_rows, void* workspace,
                                 size_t workspace_bytes, void* stream) {
    SQ_TRY(check_params(p));
    SQ_TRY(rows_only(p, "sq_conv_dgrad"));
    SQ_TRY(check_conv(N, H, W, C_out, C_in, KH, KW, PH, PW));
    if (!acc && !dX) return fail(SQ_ERR_INVALID_ARGUMENT, "acc and dX are both NULL");
    if (!layout || !gscale || !wscale) return fail(SQ_ERR_INVALID_ARGUMENT, "layout or a scale is NULL");
    const QuantCfg cfg = make_cfg(*p);
    const int64_t taps = (int64_t)KH * KW;
    // worst case |acc| = KH * KW * C_out * Q * 2^(N_G-1) * 128 must stay below 2^31
    const double bound = (double)taps * C_out * cfg.Q * (double)(1 << (cfg.num_groups - 1)) * 128.0;
    if (bound >= 2147483648.0)
        return fail(SQ_ERR_OVERFLOW_RISK,
                    "KH * KW * C_out * Q * 2^(N_G-1) * 128 reaches 2^31: the int32 accumulator could overflow");
    const int64_t pixels = N * H * W;
    const int64_t Ho = H + 2 * (int64_t)PH - KH + 1, Wo = W + 2 * (int64_t)PW - KW + 1;
    if (pixels == 0 || C_in == 0) return SQ_OK;
    size_t lay_bytes = 0;
    int64_t min_ld_fold = 0;
    SQ_TRY(sq_grad_layout_size(C_out, p, &lay_bytes, &min_ld_fold));
    const bool tiled = tiled_of(p);
    SQ_TRY(check_codes_l(q_fold, ld_fold, min_ld_fold, tiled, "q_fold"));
    SQ_TRY(check_codes_l(wq_t, ld_w, C_out > 0 ? C_out : 1, tiled, "wq_t"));
    if (acc) SQ_TRY(check_f32(acc, ld_acc, C_in, "acc"));
    if (dX) SQ_TRY(check_f32(dX, ld_dX, C_in, "dX"));
    const int64_t ext_max = fold_ext_max(C_out, cfg);
    size_t need = 0;
    SQ_TRY(sq_conv_dgrad_workspace_size(C_out, C_in, KH, KW, p, &need));
    if (!workspace || !aligned(workspace, 16)) return fail(SQ_ERR_INVALID_ARGUMENT, "workspace is NULL or misaligned");
    if (workspace_bytes < need) return fail(SQ_ERR_WORKSPACE_TOO_SMALL, "workspace too small");
    if (N * Ho * Wo * ld_fold >= ((int64_t)1 << 31))
        return fail(SQ_ERR_UNSUPPORTED, "conv: q_fold spans 2^31 bytes or more");
    hipStream_t s = static_cast<hipStream_t>(stream);

    int8_t* bc = static_cast<int8_t*>(workspace);
    const int64_t ld_bc = conv_bc_ld(C_out, taps, ext_max);
    GemmArgs a{};
    a.Mg = pixels; a.Ng = C_in;
    a.A = q_fold; a.lda = ld_fold;
    a.B = wq_t; a.ldb = ld_w;
    a.K_used = C_out;
    a.K = fold_ext_base(C_out);
    a.layout = layout;
    if (ext_max > 0) { a.extA = q_fold + fold_ext_base(C_out); a.ld_extA = ld_fold; }
    a.splits = 1;
    a.acc = acc; a.ld_acc = ld_acc;
    a.out = dX; a.ld_out = ld_dX;
    a.epi_mode = 0;
    a.gs = gscale; a.os = wscale; a.group = group; a.num_groups = cfg.num_groups;
    a.taps = (int)taps; a.cv_KW = KW; a.cv_PH = PH; a.cv_PW = PW;
    a.cv_H = H; a.cv_W = W; a.cv_Ho = Ho; a.cv_Wo = Wo; a.a_rows = N * Ho * Wo;
    a.ranges = ranges;
    return hip_status(launch_conv_dgrad(a, bc, ld_bc, s, range_rows), "conv_dgrad");
}

sq_status sq_conv_dgrad(const int8_t* q_fold, int64_t ld_fold, const int32_t* layout, const uint8_t* group,
                        const sq_scale* gscale, const int8_t* wq_t, int64_t ld_w, const sq_scale* wscale, int64_t N,
                        int64_t H, int64_t W, int64_t C_out, int64_t C_in, int32_t KH, int32_t KW, int32_t PH,
                        int32_t PW, const sq_quant_params* p, int32_t* acc, int64_t ld_acc, float* dX,
                        int64_t ld_dX, void* workspace, size_t workspace_bytes, void* stream) {
    return conv_dgrad_impl(q_fold, ld_fold, layout, group, gscale, wq_t, ld_w, wscale, N, H, W, C_out, C_in, KH, KW,
                           PH, PW, p, acc, ld_acc, dX, ld_dX, nullptr, nullptr, workspace, workspace_bytes, stream);
}

sq_status sq_conv_dgrad_ranged(const int8_t* q_fold, int64_t ld_fold, const int32_t* layout, const uint8_t* group,
                               const sq_scale* gscale, const int8_t* wq_t, int64_t ld_w, const sq_scale* wscale,
                               int64_t N, int64_t H, int64_t W, int64_t C_out, int64_t C_in, int32_t KH, int32_t KW,
                               int32_t PH, int32_t PW, const sq_quant_params* p, int32_t* acc, int64_t ld_acc,
                               float* dX, int64_t ld_dX, uint32_t* dX_ranges, int64_t* range_slabs,
                               int64_t* range_rows, void* workspace, size_t workspace_bytes, void* stream) {
    if (!dX) return fail(SQ_ERR_INVALID_ARGUMENT, "dX is NULL (the ranges are those of dX)");
    if (!range_slabs || !range_rows) return fail(SQ_ERR_INVALID_ARGUMENT, "range_slabs or range_rows is NULL");
    if (!dX_ranges || !aligned(dX_ranges, 4)) return fail(SQ_ERR_INVALID_ARGUMENT, "dX_ranges is NULL or misaligned");
    const int64_t pixels = N * H * W;
    if (pixels > 0 && (pixels + 31) / 32 > 65535)
        return fail(SQ_ERR_UNSUPPORTED, "dX ranges support at most 2^21 input pixels here");
    *range_slabs = 0;
    *range_rows = 0;
    int64_t rows = 0;
    SQ_TRY(conv_dgrad_impl(q_fold, ld_fold, layout, group, gscale, wq_t, ld_w, wscale, N, H, W, C_out, C_in, KH, KW,
                           PH, PW, p, acc, ld_acc, dX, ld_dX, dX_ranges, &rows, workspace, workspace_bytes, stream));
    *range_rows = rows;
    *range_slabs = rows > 0 ? (pixels + rows - 1) / rows : 0;
    return SQ_OK;
}

sq_status sq_gemm_wgrad(const int8_t* q_t, int64_t ld_t, const uint8_t* group, const sq_scale* gscale,
                        const int8_t* xq_t, int64_t ld_x, const sq_scale* xscale, int64_t M, int64_t C_out,
                        int64_t C_in, const sq_quant_params* p, int32_t* acc, int64_t ld_acc, float* dW,
                        int64_t ld_dW, void* workspace, size_t workspace_bytes, void* stream) {
    SQ_TRY(check_params(p));
    SQ_TRY(check_dims(M, C_out, "gradient codes"));
    SQ_TRY(check_dims(C_in, C_in, "activation codes"));
    if (!acc && !dW) return fail(SQ_ERR_INVALID_ARGUMENT, "acc and dW are both NULL");
    if (!gscale || !xscale) return fail(SQ_ERR_INVALID_ARGUMENT, "a scale is NULL");
    const QuantCfg cfg = make_cfg(*p);
    const double bound = (double)M * cfg.Q * 128.0;
    if (bound >= 2147483648.0)
        return fail(SQ_ERR_OVERFLOW_RISK, "M * Q * 128 reaches 2^31: the int32 accumulator could overflow");
    if (C_out == 0 || C_in == 0) return SQ_OK;
    if (!group) return fail(SQ_ERR_INVALID_ARGUMENT, "group is NULL");
    const bool tiled = tiled_of(p);
    if (M > 0) {
        SQ_TRY(check_codes_l(q_t, ld_t, M, tiled, "q_t"));
        SQ_TRY(check_codes_l(xq_t, ld_x, M, tiled, "xq_t"));
    }
    if (acc) SQ_TRY(check_f32(acc, ld_acc, C_in, "acc"));
    if (dW) SQ_TRY(check_f32(dW, ld_dW, C_in, "dW"));
    size_t need = 0;
    SQ_TRY(sq_gemm_wgrad_workspace_size(M, C_out, C_in, p, &need));
    const int splits = (M > 0) ? wgrad_splits(M, C_out, C_in) : 1;
    hipStream_t s = static_cast<hipStream_t>(stream);

    GemmArgs a{};
    a.Mg = C_out; a.Ng = C_in;
    a.A = q_t; a.lda = ld_t;
    a.B = xq_t; a.ldb = ld_x;
    // tile-major: K runs over the zero-padded token columns [0, roundup(M, 64))
    a.K = tiled ? round_up(M, 64) : M;
    a.tiled = tiled;
    if (tiled && M > 0 && !gemm_pipe_ok(a)) return fail(SQ_ERR_UNSUPPORTED, "tile-major operands past 31-bit offsets");
    a.gs = gscale; a.os = xscale; a.group = group; a.num_groups = cfg.num_groups;
    a.epi_mode = 1;
    if (splits <= 1) {
        a.splits = 1;
        a.acc = acc; a.ld_acc = ld_acc;
        a.out = dW; a.ld_out = ld_dW;
        return hip_status(launch_gemm(a, s), "gemm_wgrad");
    }
    if (!workspace || !aligned(workspace, 16)) return fail(SQ_ERR_INVALID_ARGUMENT, "workspace is NULL or misaligned");
    if (workspace_bytes < need) return fail(SQ_ERR_WORKSPACE_TOO_SMALL, "workspace too small");
    int32_t* ws = static_cast<int32_t*>(workspace);
    GemmArgs g = a;
    g.splits = splits;
    g.part = ws;
    SQ_TRY(hip_status(launch_gemm(g, s), "gemm_wgrad"));
    a.acc = acc; a.ld_acc = ld_acc;
    a.out = dW; a.ld_out = ld_dW;
    return hip_status(launch_splitk_reduce(ws, splits, a, s), "splitk_reduce");
}

// ---------------------------------------------------------------------------
// Implicit-im2col conv wgrad
// ---------------------------------------------------------------------------
namespace {

struct ConvGrid {
    int64_t Ho, Wo, Hp, Wp, K, ld_q, rows_x, ld_x;
};

// padded pixel grid: Hp = H + 2 PH rows, Wp = roundup(W + 2 PW, 16) columns
// per image; K = roundup(N Hp Wp, 64); the input grid extends (KH - 1) Wp + 64
// zero columns past K for the shifts of the taps
ConvGrid conv_grid(int64_t N, int64_t H, int64_t W, int64_t C_in, int KH, int KW, int PH, int PW) {
    (void)KW;
    ConvGrid g{};
    g.Ho = H + 2 * (int64_t)PH - KH + 1;
    g.Wo = W + 2 * (int64_t)PW - KW + 1;
    g.Hp = H + 2 * (int64_t)PH;
    g.Wp = round_up(W + 2 * (int64_t)PW, 16);
    g.K = round_up(std::max<int64_t>(N * g.Hp * g.Wp, 1), 64);
    g.ld_q = g.K;
    g.rows_x = C_in;
    g.ld_x = g.K + (int64_t)(KH - 1) * g.Wp + 64;
    return g;
}

sq_status check_conv_geom(int64_t N, int64_t H, int64_t W, int64_t C_out, int64_t C_in, int32_t KH, int32_t KW,
                          int32_t PH, int32_t PW) {
    if (N < 1 || H < 1 || W < 1 || C_out < 0 || C_in < 0 || KH < 1 || KW < 1 || PH < 0 || PW < 0 || KH > 16 ||
        KW > 16 || PH >= KH || PW >= KW)
        return fail(SQ_ERR_INVALID_ARGUMENT, "conv geometry out of range");
    if (H + 2 * (int64_t)PH - KH + 1 < 1 || W + 2 * (int64_t)PW - KW + 1 < 1)
        return fail(SQ_ERR_INVALID_ARGUMENT, "the window is larger than the padded input");
    const ConvGrid g = conv_grid(N, H, W, C_in, KH, KW, PH, PW);
    if (g.rows_x * g.ld_x >= ((int64_t)1 << 31) || std::max<int64_t>(C_out, 1) * g.ld_q >= ((int64_t)1 << 31))
        return fail(SQ_ERR_UNSUPPORTED, "the padded code grids exceed 2^31 bytes");
    return SQ_OK;
}

}  // namespace

sq_status sq_conv_wgrad_layout(int64_t N, int64_t H, int64_t W, int64_t C_in, int32_t KH, int32_t KW, int32_t PH,
                               int32_t PW, int64_t* x_rows, int64_t* x_ld, int64_t* q_ld) {
    if (!x_rows || !x_ld || !q_ld) return fail(SQ_ERR_INVALID_ARGUMENT, "an output pointer is NULL");
    SQ_TRY(check_conv_geom(N, H, W, 1, C_in, KH, KW, PH, PW));
    const ConvGrid g = conv_grid(N, H, W, C_in, KH, KW, PH, PW);
    *x_rows = g.rows_x;
    *x_ld = g.ld_x;
    *q_ld = g.ld_q;
    return SQ_OK;
}

sq_status sq_conv_pack_input(const int8_t* xq_t, int64_t ld_xq, int64_t N, int64_t H, int64_t W, int64_t C_in,
                             int32_t KH, int32_t KW, int32_t PH, int32_t PW, int8_t* xs, int64_t ld_xs,
                             void* stream) {
    SQ_TRY(check_conv_geom(N, H, W, 1, C_in, KH, KW, PH, PW));
    const ConvGrid g = conv_grid(N, H, W, C_in, KH, KW, PH, PW);
    if (C_in == 0) return SQ_OK;
    SQ_TRY(check_codes(xq_t, ld_xq, N * H * W, "xq_t"));
    SQ_TRY(check_codes(xs, ld_xs, g.ld_x, "xs"));
    return hip_status(launch_grid_pack(xq_t, ld_xq, C_in, N, H, W, PH, PW, g.Hp, g.Wp, xs, ld_xs,
                                       static_cast<hipStream_t>(stream)),
                      "conv pack input");
}

sq_status sq_conv_pack_grad(const int8_t* q_t, int64_t ld_t, int64_t N, int64_t H, int64_t W, int64_t C_out,
                            int32_t KH, int32_t KW, int32_t PH, int32_t PW, int8_t* q_tp, int64_t ld_tp,
                            void* stream) {
    SQ_TRY(check_conv_geom(N, H, W, C_out, 1, KH, KW, PH, PW));
    const ConvGrid g = conv_grid(N, H, W, 1, KH, KW, PH, PW);
    if (C_out == 0) return SQ_OK;
    SQ_TRY(check_codes(q_t, ld_t, N * g.Ho * g.Wo, "q_t"));
    SQ_TRY(check_codes(q_tp, ld_tp, g.ld_q, "q_tp"));
    return hip_status(launch_grid_pack(q_t, ld_t, C_out, N, g.Ho, g.Wo, 0, 0, g.Hp, g.Wp, q_tp, ld_tp,
                                       static_cast<hipStream_t>(stream)),
                      "conv pack gradient");
}

sq_status sq_quantize_input_conv(const float* X, int64_t N, int64_t H, int64_t W, int64_t C_in, int64_t ld_X,
                                 int32_t KH, int32_t KW, int32_t PH, int32_t PW, int32_t bits, int8_t* xq,
                                 int64_t ld_xq, int8_t* xs, int64_t ld_xs, sq_scale* scale, void* workspace,
                                 size_t workspace_bytes, void* stream) {
    SQ_TRY(check_conv_geom(N, H, W, 1, C_in, KH, KW, PH, PW));
    if (bits < 2 || bits > 8) return fail(SQ_ERR_INVALID_ARGUMENT, "bits must be in [2, 8]");
    const ConvGrid g = conv_grid(N, H, W, C_in, KH, KW, PH, PW);
    const int64_t M = N * H * W;
    SQ_TRY(check_dims(M, C_in, "X"));
    if (g.Hp * g.Wp >= ((int64_t)1 << 32) || M >= ((int64_t)1 << 32))
        return fail(SQ_ERR_UNSUPPORTED, "the padded grid exceeds 2^32 pixels");
    if (C_in > 0) {
        SQ_TRY(check_f32(X, ld_X, C_in, "X"));
        SQ_TRY(check_codes(xs, ld_xs, g.ld_x, "xs"));
        if (xq) SQ_TRY(check_codes(xq, ld_xq, C_in, "xq"));
    }
    if (!scale || !aligned(scale, 4)) return fail(SQ_ERR_INVALID_ARGUMENT, "scale is NULL or misaligned");
    if (!workspace || !aligned(workspace, 16)) return fail(SQ_ERR_INVALID_ARGUMENT, "workspace is NULL or misaligned");
    if (workspace_bytes < quant_ws_bytes(M, C_in)) return fail(SQ_ERR_WORKSPACE_TOO_SMALL, "workspace too small");

    sq_quant_params p{};
    p.bits = bits;
    p.num_groups = 1;
    p.round_mode = SQ_ROUND_NEAREST_EVEN;
    const QuantCfg cfg = make_cfg(p);
    hipStream_t s = static_cast<hipStream_t>(stream);
    uint32_t* partial = static_cast<uint32_t*>(workspace);
    int64_t slabs = 0;
    SQ_TRY(hip_status(launch_colmax(X, M, C_in, ld_X, partial, &slabs, s), "colmax"));
    SQ_TRY(hip_status(launch_finalize_tensor(partial, slabs, C_in, cfg.Q, partial + slabs * C_in, scale, s),
                      "finalize"));
    // input pixel (n, ih, iw) at grid column n Hp Wp + (ih + PH) Wp + iw + PW
    PadGrid pg;
    pg.Wo = (uint32_t)W;
    pg.HoWo = (uint32_t)(H * W);
    pg.Wp = (uint32_t)g.Wp;
    pg.HpWp = (uint32_t)(g.Hp * g.Wp);
    pg.off = (uint32_t)(PH * g.Wp + PW);
    SQ_TRY(hip_status(launch_quantize(X, M, C_in, ld_X, nullptr, scale, cfg, xq, ld_xq, xs, ld_xs, nullptr, s, pg),
                      "quantize"));
    return SQ_OK;
}

// ranges == nullptr: the quantizer's own abs-max pass; else the channel
// ranges as partial maxima [range_slabs, C_out] from the producer of dY
static sq_status quantize_grad_conv_impl(const float* dY, int64_t N, int64_t H, int64_t W, int64_t C_out,
                                         int64_t ld_dY, int32_t KH, int32_t KW, int32_t PH, int32_t PW,
                                         const sq_quant_params* p, const uint32_t* ranges, int64_t range_slabs,
                                         int8_t* q_fold, int64_t ld_fold, int8_t* q_tp, int64_t ld_tp,
                                         uint8_t* group, sq_scale* scale, int32_t* layout, void* workspace,
                                         size_t workspace_bytes, void* stream) {
    SQ_TRY(check_params(p));
    SQ_TRY(rows_only(p, "sq_quantize_grad_conv"));
    SQ_TRY(check_conv_geom(N, H, W, C_out, 1, KH, KW, PH, PW));
    const ConvGrid g = conv_grid(N, H, W, 1, KH, KW, PH, PW);
    const int64_t M = N * g.Ho * g.Wo;
    SQ_TRY(check_dims(M, C_out, "dY"));
    if (g.Hp * g.Wp >= ((int64_t)1 << 32) || M >= ((int64_t)1 << 32))
        return fail(SQ_ERR_UNSUPPORTED, "the padded grid exceeds 2^32 pixels");
    if (C_out > 0) SQ_TRY(check_f32(dY, ld_dY, C_out, "dY"));
    if (!scale || !aligned(scale, 4)) return fail(SQ_ERR_INVALID_ARGUMENT, "scale is NULL or misaligned");
    if (!layout || !aligned(layout, 4)) return fail(SQ_ERR_INVALID_ARGUMENT, "layout is NULL or misaligned");
    if (C_out > 0 && !group) return fail(SQ_ERR_INVALID_ARGUMENT, "group is NULL");
    size_t lay_bytes = 0;
    int64_t min_ld_fold = 0;
    SQ_TRY(sq_grad_layout_size(C_out, p, &lay_bytes, &min_ld_fold));
    if (q_fold) SQ_TRY(check_codes(q_fold, ld_fold, min_ld_fold, "q_fold"));
    if (C_out > 0) SQ_TRY(check_codes(q_tp, ld_tp, g.ld_q, "q_tp"));
    if (ranges && C_out > 0 && (!aligned(ranges, 4) || range_slabs < 1 || range_slabs >= kMaxRows))
        return fail(SQ_ERR_INVALID_ARGUMENT, "ranges misaligned or range_slabs < 1");
    if (!workspace || !aligned(workspace, 16)) return fail(SQ_ERR_INVALID_ARGUMENT, "workspace is NULL or misaligned");
    if (workspace_bytes < quant_ws_bytes(M, C_out)) return fail(SQ_ERR_WORKSPACE_TOO_SMALL, "workspace too small");

    const QuantCfg cfg = make_cfg(*p);
    hipStream_t s = static_cast<hipStream_t>(stream);
    uint32_t* partial = static_cast<uint32_t*>(workspace);
    const int64_t ext_max = fold_ext_max(C_out, cfg);
    if (ranges) {
        if (C_out > 0)
            SQ_TRY(hip_status(launch_finalize_grad(ranges, range_slabs, C_out, cfg, partial, group, scale, layout,
                                                   ext_max, s),
                              "finalize"));
    } else {
        SQ_TRY(hip_status(launch_colmax_finalize_grad(dY, M, C_out, ld_dY, cfg, partial, group, scale, layout,
                                                      ext_max, s),
                          "abs-max and finalize"));
    }
    PadGrid pg;
    pg.Wo = (uint32_t)g.Wo;
    pg.HoWo = (uint32_t)(g.Ho * g.Wo);
    pg.Wp = (uint32_t)g.Wp;
    pg.HpWp = (uint32_t)(g.Hp * g.Wp);
    SQ_TRY(hip_status(launch_quantize(dY, M, C_out, ld_dY, group, scale, cfg, q_fold, ld_fold, q_tp, ld_tp,
                                      layout + kLayoutHeader + ext_max, s, pg),
                      "quantize"));
    return SQ_OK;
}

sq_status sq_quantize_grad_conv(const float* dY, int64_t N, int64_t H, int64_t W, int64_t C_out, int64_t ld_dY,
                                int32_t KH, int32_t KW, int32_t PH, int32_t PW, const sq_quant_params* p,
                                int8_t* q_fold, int64_t ld_fold, int8_t* q_tp, int64_t ld_tp, uint8_t* group,
                                sq_scale* scale, int32_t* layout, void* workspace, size_t workspace_bytes,
                                void* stream) {
    return quantize_grad_conv_impl(dY, N, H, W, C_out, ld_dY, KH, KW, PH, PW, p, nullptr, 0, q_fold, ld_fold, q_tp,
                                   ld_tp, group, scale, layout, workspace, workspace_bytes, stream);
}

sq_status sq_quantize_grad_conv_from_ranges(const float* dY, int64_t N, int64_t H, int64_t W, int64_t C_out,
                                            int64_t ld_dY, int32_t KH, int32_t KW, int32_t PH, int32_t PW,
                                            const sq_quant_params* p, const uint32_t* ranges, int64_t range_slabs,
                                            int8_t* q_fold, int64_t ld_fold, int8_t* q_tp, int64_t ld_tp,
                                            uint8_t* group, sq_scale* scale, int32_t* layout, void* workspace,
                                            size_t workspace_bytes, void* stream) {
    if (C_out > 0 && !ranges) return fail(SQ_ERR_INVALID_ARGUMENT, "ranges is NULL");
    return quantize_grad_conv_impl(dY, N, H, W, C_out, ld_dY, KH, KW, PH, PW, p, ranges, range_slabs, q_fold, ld_fold,
                                   q_tp, ld_tp, group, scale, layout, workspace, workspace_bytes, stream);
}

namespace {
// 1 x 1 windows: the plain product of the two grids (no shifts), split as the
// linear wgrad; otherwise the single-copy window kernel
int conv_wgrad_splits_1x1(const ConvGrid& g, int64_t C_out, int64_t C_in) { return wgrad_splits(g.K, C_out, C_in); }
}  // namespace

sq_status sq_conv_wgrad_workspace_size(int64_t N, int64_t H, int64_t W, int64_t C_out, int64_t C_in, int32_t KH,
                                       int32_t KW, int32_t PH, int32_t PW, const sq_quant_params* p, size_t* bytes) {
    if (!bytes) return fail(SQ_ERR_INVALID_ARGUMENT, "bytes is NULL");
    SQ_TRY(check_params(p));
    SQ_TRY(check_conv_geom(N, H, W, C_out, C_in, KH, KW, PH, PW));
    const ConvGrid g = conv_grid(N, H, W, C_in, KH, KW, PH, PW);
    const int64_t Ng = (int64_t)KH * KW * C_in;
    int splits = 1;
    if (C_out > 0 && C_in > 0)
        splits = (KH == 1 && KW == 1) ? conv_wgrad_splits_1x1(g, C_out, C_in)
                                      : conv_wgrad_plan(g.K, C_out, C_in, KH, KW, g.Wp).splits;
    *bytes = splits > 1 ? (size_t)splits * C_out * Ng * 4 : 0;
    return SQ_OK;
}

sq_status sq_conv_wgrad(const int8_t* q_tp, int64_t ld_tp, const uint8_t* group, const sq_scale* gscale,
                        const int8_t* xs, int64_t ld_xs, const sq_scale* xscale, int64_t N, int64_t H, int64_t W,
                        int64_t C_out, int64_t C_in, int32_t KH, int32_t KW, int32_t PH, int32_t PW,
                        const sq_quant_params* p, int32_t* acc, int64_t ld_acc, float* dW, int64_t ld_dW,
                        void* workspace, size_t workspace_bytes, void* stream) {
    SQ_TRY(check_params(p));
    SQ_TRY(rows_only(p, "sq_conv_wgrad"));
    SQ_TRY(check_conv_geom(N, H, W, C_out, C_in, KH, KW, PH, PW));
    if (!acc && !dW) return fail(SQ_ERR_INVALID_ARGUMENT, "acc and dW are both NULL");
    if (!gscale || !xscale) return fail(SQ_ERR_INVALID_ARGUMENT, "a scale is NULL");
    const QuantCfg cfg = make_cfg(*p);
    const ConvGrid g = conv_grid(N, H, W, C_in, KH, KW, PH, PW);
    const int64_t M = N * g.Ho * g.Wo, Ng = (int64_t)KH * KW * C_in;
    if ((double)M * cfg.Q * 128.0 >= 2147483648.0)
        return fail(SQ_ERR_OVERFLOW_RISK, "N Ho Wo * Q * 128 reaches 2^31: the int32 accumulator could overflow");
    if (C_out == 0 || C_in == 0) return SQ_OK;
    if (!group) return fail(SQ_ERR_INVALID_ARGUMENT, "group is NULL");
    SQ_TRY(check_codes(q_tp, ld_tp, g.ld_q, "q_tp"));
    SQ_TRY(check_codes(xs, ld_xs, g.ld_x, "xs"));
    if ((int64_t)C_out * ld_tp >= ((int64_t)1 << 31) || (int64_t)C_in * ld_xs >= ((int64_t)1 << 31))
        return fail(SQ_ERR_UNSUPPORTED, "a padded code grid exceeds 2^31 bytes");
    if (acc) SQ_TRY(check_f32(acc, ld_acc, Ng, "acc"));
    if (dW) SQ_TRY(check_f32(dW, ld_dW, Ng, "dW"));
    size_t need = 0;
    SQ_TRY(sq_conv_wgrad_workspace_size(N, H, W, C_out, C_in, KH, KW, PH, PW, p, &need));
    if (need > 0) {
        if (!workspace || !aligned(workspace, 16))
            return fail(SQ_ERR_INVALID_ARGUMENT, "workspace is NULL or misaligned");
        if (workspace_bytes < need) return fail(SQ_ERR_WORKSPACE_TOO_SMALL, "workspace too small");
    }
    hipStream_t s = static_cast<hipStream_t>(stream);
    int32_t* part = static_cast<int32_t*>(workspace);
    // the epilogue of the wgrad (one scale per output channel)
    GemmArgs a{};
    a.Mg = C_out; a.Ng = Ng;
    a.A = q_tp; a.lda = ld_tp;
    a.B = xs; a.ldb = ld_xs;
    a.K = g.K;
    a.gs = gscale; a.os = xscale; a.group = group; a.num_groups = cfg.num_groups;
    a.epi_mode = 1;
    a.acc = acc; a.ld_acc = ld_acc;
    a.out = dW; a.ld_out = ld_dW;
    int splits = 1;
    if (KH == 1 && KW == 1) {
        splits = conv_wgrad_splits_1x1(g, C_out, C_in);
        GemmArgs gp = a;
        gp.splits = splits;
        if (splits > 1) {
            gp.part = part;
            gp.acc = nullptr;
            gp.out = nullptr;
        }
        SQ_TRY(hip_status(launch_gemm(gp, s), "conv wgrad"));
    } else {
        const ConvWgradPlan pl = conv_wgrad_plan(g.K, C_out, C_in, KH, KW, g.Wp);
        splits = pl.splits;
        ConvWgradArgs c{};
        c.A = q_tp; c.lda = ld_tp;
        c.X = xs; c.ldx = ld_xs;
        c.C_out = C_out; c.C_in = C_in; c.Wp = g.Wp; c.ktiles = g.K / 64;
        c.KH = KH; c.KW = KW;
        c.part = splits > 1 ? part : nullptr;
        c.acc = acc; c.ld_acc = ld_acc;
        c.out = dW; c.ld_out = ld_dW;
        c.group = group; c.gs = gscale; c.os = xscale;
        SQ_TRY(hip_status(launch_conv_wgrad(c, pl, s), "conv wgrad"));
    }
    if (splits <= 1) return SQ_OK;
    return hip_status(launch_splitk_reduce(part, splits, a, s), "splitk_reduce");
}

sq_status sq_quantize_grad_from_ranges(const float* dY, int64_t M, int64_t C_out, int64_t ld_dY,
                                       const sq_quant_params* p, const uint32_t* ranges, int64_t range_slabs,
                                       int8_t* q_fold, int64_t ld_fold, int8_t* q_t, int64_t ld_t, uint8_t* group,
                                       sq_scale* scale, int32_t* layout, void* workspace, size_t workspace_bytes,
                                       void* stream) {
    SQ_TRY(check_params(p));
    SQ_TRY(check_dims(M, C_out, "dY"));
    if (M > 0 && C_out > 0) SQ_TRY(check_f32(dY, ld_dY, C_out, "dY"));
    if (C_out > 0 && (!ranges || !aligned(ranges, 4)))
        return fail(SQ_ERR_INVALID_ARGUMENT, "ranges is NULL or misaligned");
    if (C_out > 0 && (range_slabs < 1 || range_slabs >= kMaxRows))
        return fail(SQ_ERR_INVALID_ARGUMENT, "range_slabs must be >= 1");
    if (!scale || !aligned(scale, 4)) return fail(SQ_ERR_INVALID_ARGUMENT, "scale is NULL or misaligned");
    if (!layout || !aligned(layout, 4)) return fail(SQ_ERR_INVALID_ARGUMENT, "layout is NULL or misaligned");
    if (C_out > 0 && !group) return fail(SQ_ERR_INVALID_ARGUMENT, "group is NULL");
    size_t lay_bytes = 0;
    int64_t min_ld_fold = 0;
    SQ_TRY(sq_grad_layout_size(C_out, p, &lay_bytes, &min_ld_fold));
    if (q_fold && M > 0) SQ_TRY(check_codes_l(q_fold, ld_fold, min_ld_fold, tiled_of(p), "q_fold"));
    if (q_t && C_out > 0) SQ_TRY(check_codes_l(q_t, ld_t, M > 0 ? M : 1, tiled_of(p), "q_t"));
    if (!workspace || !aligned(workspace, 16)) return fail(SQ_ERR_INVALID_ARGUMENT, "workspace is NULL or misaligned");
    if (workspace_bytes < quant_ws_bytes(M, C_out)) return fail(SQ_ERR_WORKSPACE_TOO_SMALL, "workspace too small");

    const QuantCfg cfg = make_cfg(*p);
    hipStream_t s = static_cast<hipStream_t>(stream);
    uint32_t* rbits = static_cast<uint32_t*>(workspace);
    const int64_t ext_max = fold_ext_max(C_out, cfg);
    if (C_out > 0)
        SQ_TRY(hip_status(launch_finalize_grad(ranges, range_slabs, C_out, cfg, rbits, group, scale, layout, ext_max, s),
                          "finalize"));
    SQ_TRY(hip_status(launch_quantize(dY, M, C_out, ld_dY, group, scale, cfg, q_fold, ld_fold, q_t, ld_t,
                                      layout + kLayoutHeader + ext_max, s, PadGrid(), tiled_of(p)),
                      "quantize"));
    return SQ_OK;
}

// ---------------------------------------------------------------------------
// L1BNQ
// ---------------------------------------------------------------------------
static_assert(sizeof(sq_l1bn_channel) == 32, "sq_l1bn_channel layout");
static_assert(sizeof(sq_l1bn_layer) == 56, "sq_l1bn_layer layout");

namespace {

constexpr int64_t kBnMaxRows = (int64_t)1 << 24;

sq_status check_bn_dims(int64_t M, int64_t C) {
    if (M < 1 || C < 0 || C >= kMaxChannels) return fail(SQ_ERR_INVALID_ARGUMENT, "L1BNQ needs M >= 1 and C >= 0");
    if (M > kBnMaxRows) return fail(SQ_ERR_UNSUPPORTED, "L1BNQ supports at most 2^24 rows");
    return SQ_OK;
}

size_t bn_fwd_ws_bytes(int64_t M, int64_t C) {
    return (size_t)round_up(std::max<int64_t>(l1bn_part_words(M, C), 1) * 4, 256);
}

// backward scratch: quantizer scratch | fold layout | gradient codes [M, ldc]
// | column-sum partials | per-channel constants [C, 4]
struct BnBwdWs {
    size_t quant, layout, codes, part, coef, total;
    int64_t ldc;
};

BnBwdWs bn_bwd_ws(int64_t M, int64_t C, const QuantCfg& cfg) {
    BnBwdWs w{};
    w.ldc = round_up(std::max<int64_t>(C, 1), 16);
    w.quant = 0;
    w.layout = w.quant + quant_ws_bytes(M, C);
    // groups and scales only: the finalize runs without a fold plan (one
    // window, descriptors for C channels)
    w.codes = w.layout + (size_t)round_up((kLayoutHeader + C) * 4, 256);
    w.part = w.codes + (size_t)round_up(M * w.ldc, 256);
    w.coef = w.part + (size_t)round_up(std::max<int64_t>(l1bn_part_words(M, C), 1) * 4, 256);
    w.total = w.coef + (size_t)round_up(std::max<int64_t>(C, 1) * 16, 256);
    return w;
}

}  // namespace

sq_status sq_l1bn_range_slabs(int64_t M, int64_t C, int64_t* slabs) {
    if (!slabs) return fail(SQ_ERR_INVALID_ARGUMENT, "slabs is NULL");
    SQ_TRY(check_bn_dims(M, C));
    *slabs = l1bn_range_slabs(M, C);
    return SQ_OK;
}

sq_status sq_l1bn_forward_workspace_size(int64_t M, int64_t C, size_t* bytes) {
    if (!bytes) return fail(SQ_ERR_INVALID_ARGUMENT, "bytes is NULL");
    SQ_TRY(check_bn_dims(M, C));
    *bytes = bn_fwd_ws_bytes(M, C);
    return SQ_OK;
}

sq_status sq_l1bn_backward_workspace_size(int64_t M, int64_t C, const sq_quant_params* p, size_t* bytes) {
    if (!bytes) return fail(SQ_ERR_INVALID_ARGUMENT, "bytes is NULL");
    SQ_TRY(check_params(p));
    SQ_TRY(check_bn_dims(M, C));
    *bytes = bn_bwd_ws(M, C, make_cfg(*p)).total;
    return SQ_OK;
}

sq_status sq_l1bn_forward(const int8_t* xq, int64_t M, int64_t C, int64_t ld_x, const sq_scale* xscale,
                          const float* gamma, const float* beta, float* y, int64_t ld_y, sq_l1bn_channel* chan,
                          sq_l1bn_layer* layer, void* workspace, size_t workspace_bytes, void* stream) {
    SQ_TRY(check_bn_dims(M, C));
    if (!xscale || !aligned(xscale, 4)) return fail(SQ_ERR_INVALID_ARGUMENT, "xscale is NULL or misaligned");
    if (!layer || !aligned(layer, 8)) return fail(SQ_ERR_INVALID_ARGUMENT, "layer is NULL or misaligned");
    if (C > 0) {
        SQ_TRY(check_codes(xq, ld_x, C, "xq"));
        SQ_TRY(check_f32(y, ld_y, C, "y"));
        if (!gamma || !beta || !aligned(gamma, 4) || !aligned(beta, 4))
            return fail(SQ_ERR_INVALID_ARGUMENT, "gamma / beta NULL or misaligned");
        if (!chan || !aligned(chan, 8)) return fail(SQ_ERR_INVALID_ARGUMENT, "chan is NULL or misaligned");
    }
    if (!workspace || !aligned(workspace, 16)) return fail(SQ_ERR_INVALID_ARGUMENT, "workspace is NULL or misaligned");
    if (workspace_bytes < bn_fwd_ws_bytes(M, C)) return fail(SQ_ERR_WORKSPACE_TOO_SMALL, "workspace too small");
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (C == 0) return SQ_OK;
    return hip_status(launch_l1bn_forward(xq, M, C, ld_x, xscale, gamma, beta, y, ld_y, chan, layer,
                                          static_cast<int32_t*>(workspace), s),
                      "l1bn forward");
}

sq_status sq_l1bn_backward(const float* dy, int64_t M, int64_t C, int64_t ld_dy, const sq_quant_params* p,
                           const int8_t* xq, int64_t ld_x, const sq_l1bn_channel* chan, const sq_l1bn_layer* layer,
                           float* dx, int64_t ld_dx, float* dgamma, float* dbeta, uint8_t* group, sq_scale* gscale,
                           uint32_t* dx_ranges, void* workspace, size_t workspace_bytes, void* stream) {
    SQ_TRY(check_params(p));
    SQ_TRY(rows_only(p, "sq_l1bn_backward"));
    SQ_TRY(check_bn_dims(M, C));
    if (!layer || !aligned(layer, 8)) return fail(SQ_ERR_INVALID_ARGUMENT, "layer is NULL or misaligned");
    if (!gscale || !aligned(gscale, 4)) return fail(SQ_ERR_INVALID_ARGUMENT, "gscale is NULL or misaligned");
    if (C > 0) {
        SQ_TRY(check_f32(dy, ld_dy, C, "dy"));
        SQ_TRY(check_codes(xq, ld_x, C, "xq"));
        SQ_TRY(check_f32(dx, ld_dx, C, "dx"));
        if (!dgamma || !dbeta || !aligned(dgamma, 4) || !aligned(dbeta, 4))
            return fail(SQ_ERR_INVALID_ARGUMENT, "dgamma / dbeta NULL or misaligned");
        if (!chan || !aligned(chan, 8)) return fail(SQ_ERR_INVALID_ARGUMENT, "chan is NULL or misaligned");
        if (!group) return fail(SQ_ERR_INVALID_ARGUMENT, "group is NULL");
        if (dx_ranges && !aligned(dx_ranges, 4)) return fail(SQ_ERR_INVALID_ARGUMENT, "dx_ranges is misaligned");
    }
    if (!workspace || !aligned(workspace, 256))
        return fail(SQ_ERR_INVALID_ARGUMENT, "workspace is NULL or not 256-byte aligned");
    const QuantCfg cfg = make_cfg(*p);
    const BnBwdWs w = bn_bwd_ws(M, C, cfg);
    if (workspace_bytes < w.total) return fail(SQ_ERR_WORKSPACE_TOO_SMALL, "workspace too small");
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (C == 0) return SQ_OK;
    char* base = static_cast<char*>(workspace);
    uint32_t* partial = reinterpret_cast<uint32_t*>(base + w.quant);
    int32_t* lay = reinterpret_cast<int32_t*>(base + w.layout);
    int8_t* codes = reinterpret_cast<int8_t*>(base + w.codes);
    int64_t slabs = 0;
    SQ_TRY(hip_status(launch_colmax(dy, M, C, ld_dy, partial, &slabs, s), "colmax"));
    // the groups and the scale do not depend on the fold (only the dgrad
    // operand does), so the finalize skips the fold plan: ext_max = 0
    SQ_TRY(hip_status(launch_finalize_grad(partial, slabs, C, cfg, partial + slabs * C, group, gscale, lay, 0, s),
                      "finalize"));
    // canonical codes (no fold descriptor: every channel in its own column, unshifted)
    SQ_TRY(hip_status(launch_quantize(dy, M, C, ld_dy, group, gscale, cfg, codes, w.ldc, nullptr, 0, nullptr, s),
                      "quantize"));
    return hip_status(launch_l1bn_backward(codes, w.ldc, xq, ld_x, M, C, chan, layer, group, gscale, dx, ld_dx, dgamma,
                                           dbeta, dx_ranges, reinterpret_cast<int32_t*>(base + w.part),
                                           reinterpret_cast<float*>(base + w.coef), s),
                      "l1bn backward");
}

sq_status sq_dequant(const int32_t* acc, int64_t rows, int64_t cols, int64_t ld_acc, int32_t kind,
                     const uint8_t* group, const sq_scale* gscale, const sq_scale* oscale, int32_t num_groups,
                     float* out, int64_t ld_out, void* stream) {
    SQ_TRY(check_dims(rows, cols, "accumulator"));
    if (kind < 0 || kind > 2) return fail(SQ_ERR_INVALID_ARGUMENT, "kind must be 0 (dgrad), 1 (wgrad) or 2 (per-column)");
    if (num_groups < 1 || num_groups > 8) return fail(SQ_ERR_INVALID_ARGUMENT, "num_groups must be in [1, 8]");
    if (!gscale || !oscale) return fail(SQ_ERR_INVALID_ARGUMENT, "a scale is NULL");
    if (rows == 0 || cols == 0) return SQ_OK;
    SQ_TRY(check_f32(acc, ld_acc, cols, "acc"));
    SQ_TRY(check_f32(out, ld_out, cols, "out"));
    if (kind == 1 && !group) return fail(SQ_ERR_INVALID_ARGUMENT, "group is NULL");
    return hip_status(launch_dequant(acc, rows, cols, ld_acc, kind, group, gscale, oscale, num_groups, out, ld_out,
                                     static_cast<hipStream_t>(stream)),
                      "dequant");
}

}  // extern "C"
