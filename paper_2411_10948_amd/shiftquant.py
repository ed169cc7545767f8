"""ctypes binding of libshiftquant (include/shiftquant.h).

The functions named ``sq_*`` mirror the C entry points one to one and only
marshal arguments: torch tensors supply device pointers, leading dimensions
and the current HIP stream; every step of the path runs in the library's HIP
kernels.  There is no fallback: if the library is not built this module
fails to import.

The convenience layer below them (``quantize_grad``, ``quantize_tensor``,
``gemm_dgrad``, ``gemm_wgrad``, ``BackwardPlan``) allocates outputs and
workspaces with torch and calls the ``sq_*`` functions.
"""
from __future__ import annotations

import ctypes as ct
import dataclasses
import os
from typing import Optional, Tuple

# torch is imported before the library is loaded: torch ships the HIP runtime
# (soname libamdhip64.so.7), and loading it first makes libshiftquant bind to
# that same runtime, so torch's streams and allocations are valid in it.
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libshiftquant.so")

SQ_OK = 0
STATUS_NAMES = {0: "SQ_OK", 1: "SQ_ERR_INVALID_ARGUMENT", 2: "SQ_ERR_OVERFLOW_RISK",
                3: "SQ_ERR_UNSUPPORTED", 4: "SQ_ERR_WORKSPACE_TOO_SMALL", 5: "SQ_ERR_HIP"}
LAYOUT_ROWS = 0
LAYOUT_TILED = 1
ROUND_NEAREST_EVEN = 0
ROUND_STOCHASTIC = 1
FLAG_NONFINITE = 1
FLAG_ZERO = 2

# Every symbol include/shiftquant.h declares.
EXPORTS = (
    "sq_grad_layout_size", "sq_quantize_grad_workspace_size", "sq_quantize_tensor_workspace_size",
    "sq_gemm_dgrad_workspace_size", "sq_gemm_wgrad_workspace_size", "sq_conv_dgrad_workspace_size",
    "sq_gemm_dgrad_grouped_workspace_size", "sq_quantize_channels_workspace_size",
    "sq_quantize_grad", "sq_quantize_tensor", "sq_gemm_dgrad", "sq_gemm_wgrad", "sq_conv_dgrad", "sq_dequant",
    "sq_gemm_dgrad_grouped", "sq_quantize_channels", "sq_gemm_forward",
    "sq_quantize_grad_from_ranges", "sq_l1bn_range_slabs", "sq_l1bn_forward_workspace_size",
    "sq_l1bn_backward_workspace_size", "sq_l1bn_forward", "sq_l1bn_backward",
    "sq_conv_wgrad_layout", "sq_conv_pack_input", "sq_conv_pack_grad", "sq_quantize_input_conv",
    "sq_quantize_grad_conv",
    "sq_conv_wgrad_workspace_size", "sq_conv_wgrad", "sq_gemm_dgrad_range_slabs", "sq_gemm_dgrad_ranged",
    "sq_quantize_grad_noalloc", "sq_conv_dgrad_ranged", "sq_quantize_grad_conv_from_ranges",
    "sq_status_string", "sq_last_error", "sq_last_error_string",
)


class ShiftQuantError(RuntimeError):
    def __init__(self, fn: str, status: int, message: str):
        self.status = status
        super().__init__(f"{fn}: {STATUS_NAMES.get(status, status)}: {message}")


class Params(ct.Structure):
    """sq_quant_params"""
    _fields_ = [("bits", ct.c_int32), ("num_groups", ct.c_int32), ("round_mode", ct.c_int32),
                ("layout", ct.c_int32), ("seed", ct.c_uint64), ("offset", ct.c_uint64)]

    @classmethod
    def make(cls, bits: int, num_groups: int = 4, round_mode: int = ROUND_NEAREST_EVEN,
             seed: int = 0, offset: int = 0, layout: int = 0) -> "Params":
        return cls(bits, num_groups, round_mode, layout, seed, offset)

    @property
    def tiled(self) -> bool:
        return self.layout == LAYOUT_TILED


def code_matrix(rows: int, cols: int, tiled: bool, device) -> torch.Tensor:
    """A zero-filled int8 code matrix [rows, ld] for the given layout: ld a
    multiple of 16 (row-major) or of 64 covering the K padding (tile-major,
    storage for whole 16-row groups).  Returned as the first `rows` rows of
    the allocation, so stride(0) is ld."""
    if tiled:
        ld = round_up(max(cols, 1), 64)
        return torch.zeros((round_up(max(rows, 1), 16), ld), dtype=torch.int8, device=device)[:rows]
    return torch.zeros((max(rows, 1), round_up(max(cols, 1), 16)), dtype=torch.int8, device=device)[:rows]


def untile(t: torch.Tensor) -> torch.Tensor:
    """Row-major copy [rows, ld] of a tile-major code matrix made by
    code_matrix(..., tiled=True)."""
    rows, ld = t.shape[0], t.stride(0)
    r16 = round_up(max(rows, 1), 16)
    full = t.as_strided((r16 // 16, ld // 64, 16, 64), (16 * ld, 1024, 64, 1))
    return full.permute(0, 2, 1, 3).reshape(r16, ld)[:rows]


_P = ct.c_void_p
_I64 = ct.c_int64
_SZ = ct.c_size_t
_lib = None


def load() -> ct.CDLL:
    """Load libshiftquant.so (built in-tree by paper_2411_10948_amd.build)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2411_10948_amd.build`")
    L = ct.CDLL(LIB_PATH)
    pp = ct.POINTER(Params)
    sig = {
        "sq_grad_layout_size": [_I64, pp, ct.POINTER(_SZ), ct.POINTER(_I64)],
        "sq_quantize_grad_workspace_size": [_I64, _I64, pp, ct.POINTER(_SZ)],
        "sq_quantize_tensor_workspace_size": [_I64, _I64, ct.POINTER(_SZ)],
        "sq_gemm_dgrad_workspace_size": [_I64, _I64, _I64, pp, ct.POINTER(_SZ)],
        "sq_gemm_wgrad_workspace_size": [_I64, _I64, _I64, pp, ct.POINTER(_SZ)],
        "sq_quantize_grad": [_P, _I64, _I64, _I64, pp, _P, _I64, _P, _I64, _P, _P, _P, _P, _SZ, _P],
        "sq_quantize_grad_noalloc": [_P, _I64, _I64, _I64, pp, _P, _I64, _P, _I64, _P, _P, _P, _P],
        "sq_quantize_tensor": [_P, _I64, _I64, _I64, ct.c_int32, ct.c_int32, _P, _I64, _P, _P, _SZ, _P],
        "sq_gemm_dgrad": [_P, _I64, _P, _P, _P, _P, _I64, _P, _I64, _I64, _I64, pp, _P, _I64, _P, _I64,
                          _P, _SZ, _P],
        "sq_gemm_wgrad": [_P, _I64, _P, _P, _P, _I64, _P, _I64, _I64, _I64, pp, _P, _I64, _P, _I64, _P,
                          _SZ, _P],
        "sq_dequant": [_P, _I64, _I64, _I64, ct.c_int32, _P, _P, _P, ct.c_int32, _P, _I64, _P],
        "sq_conv_dgrad_workspace_size": [_I64, _I64, ct.c_int32, ct.c_int32, pp, ct.POINTER(_SZ)],
        "sq_gemm_dgrad_grouped_workspace_size": [_I64, _I64, _I64, pp, ct.POINTER(_SZ)],
        "sq_quantize_channels_workspace_size": [_I64, _I64, ct.c_int32, ct.POINTER(_SZ)],
        "sq_quantize_channels": [_P, _I64, _I64, _I64, ct.c_int32, ct.c_int32, ct.c_int32, _P, _I64, _P, _P, _SZ,
                                 _P],
        "sq_gemm_forward": [_P, _I64, _P, _P, _P, _P, _I64, _P, _I64, _I64, _I64, pp, _P, _I64, _P, _I64, _P,
                            _SZ, _P],
        "sq_gemm_dgrad_grouped": [_P, _I64, _P, _P, _P, _P, _I64, _P, _I64, _I64, _I64, pp, _P, _I64, _P, _I64,
                                  _P, _SZ, _P],
        "sq_conv_dgrad": [_P, _I64, _P, _P, _P, _P, _I64, _P, _I64, _I64, _I64, _I64, _I64, ct.c_int32,
                          ct.c_int32, ct.c_int32, ct.c_int32, pp, _P, _I64, _P, _I64, _P, _SZ, _P],
        "sq_quantize_grad_from_ranges": [_P, _I64, _I64, _I64, pp, _P, _I64, _P, _I64, _P, _I64, _P, _P, _P, _P,
                                         _SZ, _P],
        "sq_l1bn_range_slabs": [_I64, _I64, ct.POINTER(_I64)],
        "sq_gemm_dgrad_range_slabs": [_I64, ct.POINTER(_I64)],
        "sq_conv_dgrad_ranged": [_P, _I64, _P, _P, _P, _P, _I64, _P, _I64, _I64, _I64, _I64, _I64, ct.c_int32,
                                 ct.c_int32, ct.c_int32, ct.c_int32, pp, _P, _I64, _P, _I64, _P,
                                 ct.POINTER(_I64), ct.POINTER(_I64), _P, _SZ, _P],
        "sq_quantize_grad_conv_from_ranges": [_P, _I64, _I64, _I64, _I64, _I64, ct.c_int32, ct.c_int32, ct.c_int32,
                                              ct.c_int32, pp, _P, _I64, _P, _I64, _P, _I64, _P, _P, _P, _P, _SZ,
                                              _P],
        "sq_gemm_dgrad_ranged": [_P, _I64, _P, _P, _P, _P, _I64, _P, _I64, _I64, _I64, pp, _P, _I64, _P, _I64, _P,
                                 _P, _SZ, _P],
        "sq_conv_wgrad_layout": [_I64, _I64, _I64, _I64, ct.c_int32, ct.c_int32, ct.c_int32, ct.c_int32,
                                 ct.POINTER(_I64), ct.POINTER(_I64), ct.POINTER(_I64)],
        "sq_conv_pack_grad": [_P, _I64, _I64, _I64, _I64, _I64, ct.c_int32, ct.c_int32, ct.c_int32, ct.c_int32,
                              _P, _I64, _P],
        "sq_quantize_grad_conv": [_P, _I64, _I64, _I64, _I64, _I64, ct.c_int32, ct.c_int32, ct.c_int32,
                                  ct.c_int32, pp, _P, _I64, _P, _I64, _P, _P, _P, _P, _SZ, _P],
        "sq_conv_pack_input": [_P, _I64, _I64, _I64, _I64, _I64, ct.c_int32, ct.c_int32, ct.c_int32, ct.c_int32,
                               _P, _I64, _P],
        "sq_quantize_input_conv": [_P, _I64, _I64, _I64, _I64, _I64, ct.c_int32, ct.c_int32, ct.c_int32, ct.c_int32,
                                   ct.c_int32, _P, _I64, _P, _I64, _P, _P, _SZ, _P],
        "sq_conv_wgrad_workspace_size": [_I64, _I64, _I64, _I64, _I64, ct.c_int32, ct.c_int32, ct.c_int32,
                                         ct.c_int32, pp, ct.POINTER(_SZ)],
        "sq_conv_wgrad": [_P, _I64, _P, _P, _P, _I64, _P, _I64, _I64, _I64, _I64, _I64, ct.c_int32, ct.c_int32,
                          ct.c_int32, ct.c_int32, pp, _P, _I64, _P, _I64, _P, _SZ, _P],
        "sq_l1bn_forward_workspace_size": [_I64, _I64, ct.POINTER(_SZ)],
        "sq_l1bn_backward_workspace_size": [_I64, _I64, pp, ct.POINTER(_SZ)],
        "sq_l1bn_forward": [_P, _I64, _I64, _I64, _P, _P, _P, _P, _I64, _P, _P, _P, _SZ, _P],
        "sq_l1bn_backward": [_P, _I64, _I64, _I64, pp, _P, _I64, _P, _P, _P, _I64, _P, _P, _P, _P, _P, _P, _SZ,
                             _P],
    }
    for name, args in sig.items():
        f = getattr(L, name)
        f.argtypes = args
        f.restype = ct.c_int
    L.sq_status_string.argtypes = [ct.c_int]
    L.sq_status_string.restype = ct.c_char_p
    L.sq_last_error.argtypes = []
    L.sq_last_error.restype = ct.c_char_p
    L.sq_last_error_string.argtypes = []
    L.sq_last_error_string.restype = ct.c_char_p
    _lib = L
    return L


def sq_status_string(status: int) -> str:
    return load().sq_status_string(status).decode()


def sq_last_error() -> str:
    return load().sq_last_error().decode()


def _check(fn: str, status: int) -> None:
    if status != SQ_OK:
        raise ShiftQuantError(fn, status, sq_last_error())


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ct.c_void_p(t.data_ptr())


def _ld(t: Optional[torch.Tensor]) -> int:
    if t is None:
        return 0
    if t.dim() != 2 or (t.shape[1] > 1 and t.stride(1) != 1):
        raise ValueError("expected a 2-D tensor with unit column stride")
    return t.stride(0)


def _stream(stream) -> ct.c_void_p:
    s = torch.cuda.current_stream() if stream is None else stream
    return ct.c_void_p(s.cuda_stream)


def _ws_ptr(ws: Optional[torch.Tensor]):
    return (None, 0) if ws is None else (ct.c_void_p(ws.data_ptr()), ws.numel() * ws.element_size())


# ---------------------------------------------------------------------------
# one-to-one wrappers of the C entry points
# ---------------------------------------------------------------------------
def sq_grad_layout_size(C_out: int, params: Params) -> Tuple[int, int]:
    nb, ld = _SZ(0), _I64(0)
    _check("sq_grad_layout_size", load().sq_grad_layout_size(C_out, ct.byref(params), ct.byref(nb), ct.byref(ld)))
    return nb.value, ld.value


def sq_quantize_grad_workspace_size(M: int, C_out: int, params: Params) -> int:
    nb = _SZ(0)
    _check("sq_quantize_grad_workspace_size",
           load().sq_quantize_grad_workspace_size(M, C_out, ct.byref(params), ct.byref(nb)))
    return nb.value


def sq_quantize_tensor_workspace_size(rows: int, cols: int) -> int:
    nb = _SZ(0)
    _check("sq_quantize_tensor_workspace_size", load().sq_quantize_tensor_workspace_size(rows, cols, ct.byref(nb)))
    return nb.value


def sq_gemm_dgrad_workspace_size(M: int, C_out: int, C_in: int, params: Params) -> int:
    nb = _SZ(0)
    _check("sq_gemm_dgrad_workspace_size",
           load().sq_gemm_dgrad_workspace_size(M, C_out, C_in, ct.byref(params), ct.byref(nb)))
    return nb.value


def sq_gemm_wgrad_workspace_size(M: int, C_out: int, C_in: int, params: Params) -> int:
    nb = _SZ(0)
    _check("sq_gemm_wgrad_workspace_size",
           load().sq_gemm_wgrad_workspace_size(M, C_out, C_in, ct.byref(params), ct.byref(nb)))
    return nb.value


def sq_conv_dgrad_workspace_size(C_out: int, C_in: int, KH: int, KW: int, params: Params) -> int:
    nb = _SZ(0)
    _check("sq_conv_dgrad_workspace_size",
           load().sq_conv_dgrad_workspace_size(C_out, C_in, KH, KW, ct.byref(params), ct.byref(nb)))
    return nb.value


def sq_gemm_dgrad_grouped_workspace_size(M: int, C_out: int, C_in: int, params: Params) -> int:
    nb = _SZ(0)
    _check("sq_gemm_dgrad_grouped_workspace_size",
           load().sq_gemm_dgrad_grouped_workspace_size(M, C_out, C_in, ct.byref(params), ct.byref(nb)))
    return nb.value


def sq_quantize_channels_workspace_size(rows: int, cols: int, axis: int) -> int:
    nb = _SZ(0)
    _check("sq_quantize_channels_workspace_size",
           load().sq_quantize_channels_workspace_size(rows, cols, axis, ct.byref(nb)))
    return nb.value


def sq_quantize_channels(T, bits, axis, transpose, q, scales, workspace, stream=None) -> None:
    rows, cols = T.shape
    ws, nws = _ws_ptr(workspace)
    _check("sq_quantize_channels", load().sq_quantize_channels(
        _ptr(T), rows, cols, _ld(T), bits, axis, int(transpose), _ptr(q), _ld(q), _ptr(scales), ws, nws,
        _stream(stream)))


def sq_gemm_forward(xq_fold, layout, group, xscale, wq, wscales, M, C_in, C_out, params, acc, Y, workspace,
                    stream=None) -> None:
    ws, nws = _ws_ptr(workspace)
    _check("sq_gemm_forward", load().sq_gemm_forward(
        _ptr(xq_fold), _ld(xq_fold), _ptr(layout), _ptr(group), _ptr(xscale), _ptr(wq), _ld(wq), _ptr(wscales),
        M, C_in, C_out, ct.byref(params), _ptr(acc), _ld(acc), _ptr(Y), _ld(Y), ws, nws, _stream(stream)))


def sq_quantize_grad(dY, params, q_fold, q_t, group, scale, layout, workspace, stream=None) -> None:
    M, C = dY.shape
    ws, nws = _ws_ptr(workspace)
    _check("sq_quantize_grad", load().sq_quantize_grad(
        _ptr(dY), M, C, _ld(dY), ct.byref(params), _ptr(q_fold), _ld(q_fold), _ptr(q_t), _ld(q_t),
        _ptr(group), _ptr(scale), _ptr(layout), ws, nws, _stream(stream)))


def sq_quantize_grad_noalloc(dY, params, q_fold, q_t, group, scale, layout, stream=None) -> None:
    M, C = dY.shape
    _check("sq_quantize_grad_noalloc", load().sq_quantize_grad_noalloc(
        _ptr(dY), M, C, _ld(dY), ct.byref(params), _ptr(q_fold), _ld(q_fold), _ptr(q_t), _ld(q_t),
        _ptr(group), _ptr(scale), _ptr(layout), _stream(stream)))


def sq_quantize_grad_from_ranges(dY, params, ranges, range_slabs, q_fold, q_t, group, scale, layout, workspace,
                                 stream=None) -> None:
    M, C = dY.shape
    ws, nws = _ws_ptr(workspace)
    _check("sq_quantize_grad_from_ranges", load().sq_quantize_grad_from_ranges(
        _ptr(dY), M, C, _ld(dY), ct.byref(params), _ptr(ranges), range_slabs, _ptr(q_fold), _ld(q_fold),
        _ptr(q_t), _ld(q_t), _ptr(group), _ptr(scale), _ptr(layout), ws, nws, _stream(stream)))


def sq_conv_wgrad_layout(N, H, W, C_in, KH, KW, PH, PW) -> Tuple[int, int, int]:
    """(x_rows, x_ld, q_ld) of the padded pixel grids of sq_conv_wgrad."""
    rows, ld, qld = _I64(0), _I64(0), _I64(0)
    _check("sq_conv_wgrad_layout", load().sq_conv_wgrad_layout(N, H, W, C_in, KH, KW, PH, PW, ct.byref(rows),
                                                               ct.byref(ld), ct.byref(qld)))
    return rows.value, ld.value, qld.value


def sq_conv_pack_grad(q_t, N, H, W, C_out, KH, KW, PH, PW, q_tp, stream=None) -> None:
    _check("sq_conv_pack_grad", load().sq_conv_pack_grad(_ptr(q_t), _ld(q_t), N, H, W, C_out, KH, KW, PH, PW,
                                                         _ptr(q_tp), _ld(q_tp), _stream(stream)))


def sq_quantize_grad_conv(dY, N, H, W, KH, KW, PH, PW, params, q_fold, q_tp, group, scale, layout, workspace,
                          stream=None) -> None:
    C = dY.shape[1]
    ws, nws = _ws_ptr(workspace)
    _check("sq_quantize_grad_conv", load().sq_quantize_grad_conv(
        _ptr(dY), N, H, W, C, _ld(dY), KH, KW, PH, PW, ct.byref(params), _ptr(q_fold), _ld(q_fold), _ptr(q_tp),
        _ld(q_tp), _ptr(group), _ptr(scale), _ptr(layout), ws, nws, _stream(stream)))


def sq_conv_pack_input(xq_t, N, H, W, C_in, KH, KW, PH, PW, xs, stream=None) -> None:
    _check("sq_conv_pack_input", load().sq_conv_pack_input(_ptr(xq_t), _ld(xq_t), N, H, W, C_in, KH, KW, PH, PW,
                                                           _ptr(xs), _ld(xs), _stream(stream)))


def sq_quantize_input_conv(X, N, H, W, KH, KW, PH, PW, bits, xq, xs, scale, workspace, stream=None) -> None:
    C = X.shape[1]
    ws, nws = _ws_ptr(workspace)
    _check("sq_quantize_input_conv", load().sq_quantize_input_conv(
        _ptr(X), N, H, W, C, _ld(X), KH, KW, PH, PW, bits, _ptr(xq), _ld(xq) if xq is not None else 0, _ptr(xs),
        _ld(xs), _ptr(scale), ws, nws, _stream(stream)))


def sq_conv_wgrad_workspace_size(N, H, W, C_out, C_in, KH, KW, PH, PW, params: Params) -> int:
    nb = _SZ(0)
    _check("sq_conv_wgrad_workspace_size", load().sq_conv_wgrad_workspace_size(
        N, H, W, C_out, C_in, KH, KW, PH, PW, ct.byref(params), ct.byref(nb)))
    return nb.value


def sq_conv_wgrad(q_t, group, gscale, xs, xscale, N, H, W, C_out, C_in, KH, KW, PH, PW, params, acc, dW, workspace,
                  stream=None) -> None:
    ws, nws = _ws_ptr(workspace)
    _check("sq_conv_wgrad", load().sq_conv_wgrad(
        _ptr(q_t), _ld(q_t), _ptr(group), _ptr(gscale), _ptr(xs), _ld(xs), _ptr(xscale), N, H, W, C_out, C_in,
        KH, KW, PH, PW, ct.byref(params), _ptr(acc), _ld(acc), _ptr(dW), _ld(dW), ws, nws, _stream(stream)))


def sq_gemm_dgrad_range_slabs(M: int) -> int:
    n = _I64(0)
    _check("sq_gemm_dgrad_range_slabs", load().sq_gemm_dgrad_range_slabs(M, ct.byref(n)))
    return n.value


def sq_gemm_dgrad_ranged(q_fold, layout, group, gscale, wq_t, wscale, M, C_out, C_in, params, acc, dX, dX_ranges,
                         workspace, stream=None) -> None:
    ws, nws = _ws_ptr(workspace)
    _check("sq_gemm_dgrad_ranged", load().sq_gemm_dgrad_ranged(
        _ptr(q_fold), _ld(q_fold), _ptr(layout), _ptr(group), _ptr(gscale), _ptr(wq_t), _ld(wq_t), _ptr(wscale), M,
        C_out, C_in, ct.byref(params), _ptr(acc), _ld(acc), _ptr(dX), _ld(dX), _ptr(dX_ranges), ws, nws,
        _stream(stream)))


def sq_l1bn_range_slabs(M: int, C: int) -> int:
    n = _I64(0)
    _check("sq_l1bn_range_slabs", load().sq_l1bn_range_slabs(M, C, ct.byref(n)))
    return n.value


def sq_l1bn_forward_workspace_size(M: int, C: int) -> int:
    nb = _SZ(0)
    _check("sq_l1bn_forward_workspace_size", load().sq_l1bn_forward_workspace_size(M, C, ct.byref(nb)))
    return nb.value


def sq_l1bn_backward_workspace_size(M: int, C: int, params: Params) -> int:
    nb = _SZ(0)
    _check("sq_l1bn_backward_workspace_size",
           load().sq_l1bn_backward_workspace_size(M, C, ct.byref(params), ct.byref(nb)))
    return nb.value


def sq_l1bn_forward(xq, xscale, gamma, beta, y, chan, layer, workspace, stream=None) -> None:
    M, C = xq.shape
    ws, nws = _ws_ptr(workspace)
    _check("sq_l1bn_forward", load().sq_l1bn_forward(
        _ptr(xq), M, C, _ld(xq), _ptr(xscale), _ptr(gamma), _ptr(beta), _ptr(y), _ld(y), _ptr(chan), _ptr(layer),
        ws, nws, _stream(stream)))


def sq_l1bn_backward(dy, params, xq, chan, layer, dx, dgamma, dbeta, group, gscale, dx_ranges, workspace,
                     stream=None) -> None:
    M, C = dy.shape
    ws, nws = _ws_ptr(workspace)
    _check("sq_l1bn_backward", load().sq_l1bn_backward(
        _ptr(dy), M, C, _ld(dy), ct.byref(params), _ptr(xq), _ld(xq), _ptr(chan), _ptr(layer), _ptr(dx), _ld(dx),
        _ptr(dgamma), _ptr(dbeta), _ptr(group), _ptr(gscale), _ptr(dx_ranges), ws, nws, _stream(stream)))


def sq_quantize_tensor(T, bits, transpose, q, scale, workspace, stream=None) -> None:
    rows, cols = T.shape
    ws, nws = _ws_ptr(workspace)
    _check("sq_quantize_tensor", load().sq_quantize_tensor(
        _ptr(T), rows, cols, _ld(T), bits, int(transpose), _ptr(q), _ld(q), _ptr(scale), ws, nws,
        _stream(stream)))


def sq_gemm_dgrad(q_fold, layout, group, gscale, wq_t, wscale, M, C_out, C_in, params, acc, dX,
                  workspace, stream=None) -> None:
    ws, nws = _ws_ptr(workspace)
    _check("sq_gemm_dgrad", load().sq_gemm_dgrad(
        _ptr(q_fold), _ld(q_fold), _ptr(layout), _ptr(group), _ptr(gscale), _ptr(wq_t), _ld(wq_t),
        _ptr(wscale), M, C_out, C_in, ct.byref(params), _ptr(acc), _ld(acc), _ptr(dX), _ld(dX),
        ws, nws, _stream(stream)))


def sq_conv_dgrad_ranged(q_fold, layout, group, gscale, wq_t, wscale, N, H, W, C_out, C_in, KH, KW, PH, PW,
                         params, acc, dX, dX_ranges, workspace, stream=None) -> Tuple[int, int]:
    """sq_conv_dgrad plus the channel ranges of dX; returns (slabs, rows per slab)."""
    ws, nws = _ws_ptr(workspace)
    slabs, rows = _I64(0), _I64(0)
    _check("sq_conv_dgrad_ranged", load().sq_conv_dgrad_ranged(
        _ptr(q_fold), _ld(q_fold), _ptr(layout), _ptr(group), _ptr(gscale), _ptr(wq_t), _ld(wq_t),
        _ptr(wscale), N, H, W, C_out, C_in, KH, KW, PH, PW, ct.byref(params), _ptr(acc), _ld(acc),
        _ptr(dX), _ld(dX), _ptr(dX_ranges), ct.byref(slabs), ct.byref(rows), ws, nws, _stream(stream)))
    return int(slabs.value), int(rows.value)


def sq_quantize_grad_conv_from_ranges(dY, N, H, W, KH, KW, PH, PW, params, ranges, range_slabs, q_fold, q_tp, group,
                                      scale, layout, workspace, stream=None) -> None:
    C = dY.shape[1]
    ws, nws = _ws_ptr(workspace)
    _check("sq_quantize_grad_conv_from_ranges", load().sq_quantize_grad_conv_from_ranges(
        _ptr(dY), N, H, W, C, _ld(dY), KH, KW, PH, PW, ct.byref(params), _ptr(ranges), range_slabs,
        _ptr(q_fold), _ld(q_fold), _ptr(q_tp), _ld(q_tp), _ptr(group), _ptr(scale), _ptr(layout), ws, nws,
        _stream(stream)))


def sq_conv_dgrad(q_fold, layout, group, gscale, wq_t, wscale, N, H, W, C_out, C_in, KH, KW, PH, PW, params,
                  acc, dX, workspace, stream=None) -> None:
    ws, nws = _ws_ptr(workspace)
    _check("sq_conv_dgrad", load().sq_conv_dgrad(
        _ptr(q_fold), _ld(q_fold), _ptr(layout), _ptr(group), _ptr(gscale), _ptr(wq_t), _ld(wq_t),
        _ptr(wscale), N, H, W, C_out, C_in, KH, KW, PH, PW, ct.byref(params), _ptr(acc), _ld(acc),
        _ptr(dX), _ld(dX), ws, nws, _stream(stream)))


def sq_gemm_dgrad_grouped(q_fold, layout, group, gscale, wq_t, wscale, M, C_out, C_in, params, acc, dX,
                          workspace, stream=None) -> None:
    ws, nws = _ws_ptr(workspace)
    _check("sq_gemm_dgrad_grouped", load().sq_gemm_dgrad_grouped(
        _ptr(q_fold), _ld(q_fold), _ptr(layout), _ptr(group), _ptr(gscale), _ptr(wq_t), _ld(wq_t),
        _ptr(wscale), M, C_out, C_in, ct.byref(params), _ptr(acc), _ld(acc), _ptr(dX), _ld(dX),
        ws, nws, _stream(stream)))


def sq_gemm_wgrad(q_t, group, gscale, xq_t, xscale, M, C_out, C_in, params, acc, dW, workspace,
                  stream=None) -> None:
    ws, nws = _ws_ptr(workspace)
    _check("sq_gemm_wgrad", load().sq_gemm_wgrad(
        _ptr(q_t), _ld(q_t), _ptr(group), _ptr(gscale), _ptr(xq_t), _ld(xq_t), _ptr(xscale),
        M, C_out, C_in, ct.byref(params), _ptr(acc), _ld(acc), _ptr(dW), _ld(dW), ws, nws,
        _stream(stream)))


def sq_dequant(acc, kind, group, gscale, oscale, num_groups, out, stream=None) -> None:
    rows, cols = acc.shape
    _check("sq_dequant", load().sq_dequant(
        _ptr(acc), rows, cols, _ld(acc), kind, _ptr(group), _ptr(gscale), _ptr(oscale), num_groups,
        _ptr(out), _ld(out), _stream(stream)))


# ---------------------------------------------------------------------------
# convenience layer (allocates with torch, then calls the wrappers above)
# ---------------------------------------------------------------------------
def round_up(x: int, m: int) -> int:
    return (x + m - 1) // m * m


def new_scale(device) -> torch.Tensor:
    """Device storage for one sq_scale (r_max, inv, step, flags)."""
    return torch.zeros(4, dtype=torch.float32, device=device)


def scale_to_host(scale: torch.Tensor) -> dict:
    s = scale.detach().cpu()
    return {"r_max": s[0].item(), "inv": s[1].item(), "step": s[2].item(),
            "flags": int(s.view(torch.int32)[3].item()),
            "bits": s.view(torch.int32).tolist()}


def _workspace(nbytes: int, device) -> Optional[torch.Tensor]:
    return torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)


@dataclasses.dataclass
class GradCodes:
    """Output of sq_quantize_grad for one gradient tensor (code matrices in the
    layout params.layout names)."""
    q_fold: torch.Tensor      # [M, ld_fold] int8, dgrad operand
    q_t: torch.Tensor         # [C_out, ld_t] int8, codes transposed (wgrad operand)
    group: torch.Tensor       # [C_out] uint8
    scale: torch.Tensor       # sq_scale
    layout: torch.Tensor      # fold descriptor (int32)
    params: Params
    M: int
    C_out: int

    def codes(self) -> torch.Tensor:
        """The codes [M, C_out] themselves (q_t transposed)."""
        qt = untile(self.q_t) if self.params.tiled else self.q_t
        return qt[:, :self.M].t()

    def fold_rows(self) -> torch.Tensor:
        """q_fold as a row-major [M, ld_fold] matrix (a copy when tile-major)."""
        return untile(self.q_fold) if self.params.tiled else self.q_fold


def quantize_grad(dY: torch.Tensor, bits: int, num_groups: int = 4, round_mode: int = ROUND_NEAREST_EVEN,
                  seed: int = 0, offset: int = 0, stream=None, tiled: bool = False) -> GradCodes:
    M, C = dY.shape
    dev = dY.device
    p = Params.make(bits, num_groups, round_mode, seed, offset, LAYOUT_TILED if tiled else LAYOUT_ROWS)
    lay_bytes, min_ld = sq_grad_layout_size(C, p)
    q_fold = code_matrix(M, min_ld, tiled, dev)
    q_t = code_matrix(C, M, tiled, dev)
    group = torch.empty(max(C, 1), dtype=torch.uint8, device=dev)[:C]
    scale = new_scale(dev)
    layout = torch.zeros(lay_bytes // 4, dtype=torch.int32, device=dev)
    ws = _workspace(sq_quantize_grad_workspace_size(M, C, p), dev)
    sq_quantize_grad(dY, p, q_fold, q_t, group, scale, layout, ws, stream)
    return GradCodes(q_fold, q_t, group, scale, layout, p, M, C)


def quantize_tensor(T: torch.Tensor, bits: int = 8, transpose: bool = True, stream=None, tiled: bool = False):
    """Per-tensor codes of T; transpose: [cols, rows] (the GEMM operand),
    tiled: that matrix tile-major (transpose = 2 of the C call)."""
    rows, cols = T.shape
    dev = T.device
    if transpose:
        q = code_matrix(cols, rows, tiled, dev)
    else:
        assert not tiled, "tile-major codes are transposed"
        q = code_matrix(rows, cols, False, dev)
    scale = new_scale(dev)
    ws = _workspace(sq_quantize_tensor_workspace_size(rows, cols), dev)
    sq_quantize_tensor(T, bits, 2 if tiled else int(transpose), q, scale, ws, stream)
    return q, scale


def quantize_channels(T: torch.Tensor, bits: int = 8, axis: int = 0, transpose: bool = False, stream=None):
    """Per-channel codes of T: one scale per row (axis 0) or column (axis 1).
    Returns (codes, scales [n, 4] float32 words = n sq_scale structs)."""
    rows, cols = T.shape
    dev = T.device
    if transpose:
        q = torch.zeros((max(cols, 1), round_up(max(rows, 1), 16)), dtype=torch.int8, device=dev)[:cols]
    else:
        q = torch.zeros((max(rows, 1), round_up(max(cols, 1), 16)), dtype=torch.int8, device=dev)[:rows]
    n = rows if axis == 0 else cols
    scales = torch.zeros((max(n, 1), 4), dtype=torch.float32, device=dev)
    ws = _workspace(sq_quantize_channels_workspace_size(rows, cols, axis), dev)
    sq_quantize_channels(T, bits, axis, transpose, q, scales, ws, stream)
    return q, scales


def gemm_forward(xcodes: GradCodes, wq: torch.Tensor, wscales: torch.Tensor, want_acc: bool = False,
                 want_out: bool = True, stream=None):
    """Y = X W^T: xcodes from quantize_grad(X), wq [C_out, C_in] per-output-channel codes."""
    M, C_in, C_out = xcodes.M, xcodes.C_out, wq.shape[0]
    dev = wq.device
    acc = torch.empty((M, C_out), dtype=torch.int32, device=dev) if want_acc else None
    Y = torch.empty((M, C_out), dtype=torch.float32, device=dev) if want_out else None
    ws = _workspace(sq_gemm_dgrad_workspace_size(M, C_in, C_out, xcodes.params), dev)
    sq_gemm_forward(xcodes.q_fold, xcodes.layout, xcodes.group, xcodes.scale, wq, wscales, M, C_in, C_out,
                    xcodes.params, acc, Y, ws, stream)
    return acc, Y


def gemm_dgrad(codes: GradCodes, wq_t: torch.Tensor, wscale: torch.Tensor, want_acc: bool = False,
               want_out: bool = True, stream=None):
    M, C_out, C_in = codes.M, codes.C_out, wq_t.shape[0]
    dev = wq_t.device
    acc = torch.empty((M, C_in), dtype=torch.int32, device=dev) if want_acc else None
    dX = torch.empty((M, C_in), dtype=torch.float32, device=dev) if want_out else None
    ws = _workspace(sq_gemm_dgrad_workspace_size(M, C_out, C_in, codes.params), dev)
    sq_gemm_dgrad(codes.q_fold, codes.layout, codes.group, codes.scale, wq_t, wscale, M, C_out, C_in,
                  codes.params, acc, dX, ws, stream)
    return acc, dX


def gemm_dgrad_grouped(codes: GradCodes, wq_t: torch.Tensor, wscale: torch.Tensor, want_acc: bool = False,
                       want_out: bool = True, stream=None):
    """The GEMM-based comparison implementation of gemm_dgrad (same results)."""
    M, C_out, C_in = codes.M, codes.C_out, wq_t.shape[0]
    dev = wq_t.device
    acc = torch.empty((M, C_in), dtype=torch.int32, device=dev) if want_acc else None
    dX = torch.empty((M, C_in), dtype=torch.float32, device=dev) if want_out else None
    ws = _workspace(sq_gemm_dgrad_grouped_workspace_size(M, C_out, C_in, codes.params), dev)
    sq_gemm_dgrad_grouped(codes.q_fold, codes.layout, codes.group, codes.scale, wq_t, wscale, M, C_out, C_in,
                          codes.params, acc, dX, ws, stream)
    return acc, dX


def conv_dgrad(codes: GradCodes, wq_t: torch.Tensor, wscale: torch.Tensor, N: int, H: int, W: int,
               KH: int, KW: int, PH: int, PW: int, want_acc: bool = False, want_out: bool = True, stream=None):
    """Input gradient [N*H*W, C_in] (NHWC) of a stride-1 convolution whose output
    gradient was quantized into `codes` ([N*Ho*Wo, C_out]); wq_t holds the W^T
    codes of W [C_out, KH*KW*C_in] (columns in (r, s, ci) order)."""
    C_out = codes.C_out
    C_in = wq_t.shape[0] // (KH * KW)
    assert wq_t.shape[0] == KH * KW * C_in
    dev = wq_t.device
    acc = torch.empty((N * H * W, C_in), dtype=torch.int32, device=dev) if want_acc else None
    dX = torch.empty((N * H * W, C_in), dtype=torch.float32, device=dev) if want_out else None
    ws = _workspace(sq_conv_dgrad_workspace_size(C_out, C_in, KH, KW, codes.params), dev)
    sq_conv_dgrad(codes.q_fold, codes.layout, codes.group, codes.scale, wq_t, wscale, N, H, W, C_out, C_in,
                  KH, KW, PH, PW, codes.params, acc, dX, ws, stream)
    return acc, dX


def gemm_wgrad(codes: GradCodes, xq_t: torch.Tensor, xscale: torch.Tensor, want_acc: bool = False,
               want_out: bool = True, stream=None):
    M, C_out, C_in = codes.M, codes.C_out, xq_t.shape[0]
    dev = xq_t.device
    acc = torch.empty((C_out, C_in), dtype=torch.int32, device=dev) if want_acc else None
    dW = torch.empty((C_out, C_in), dtype=torch.float32, device=dev) if want_out else None
    ws = _workspace(sq_gemm_wgrad_workspace_size(M, C_out, C_in, codes.params), dev)
    sq_gemm_wgrad(codes.q_t, codes.group, codes.scale, xq_t, xscale, M, C_out, C_in, codes.params,
                  acc, dW, ws, stream)
    return acc, dW


def quantize_grad_from_ranges(dY: torch.Tensor, ranges: torch.Tensor, bits: int, num_groups: int = 4,
                              round_mode: int = ROUND_NEAREST_EVEN, seed: int = 0, offset: int = 0,
                              stream=None, tiled: bool = False) -> GradCodes:
    """quantize_grad with the channel ranges given as partial maxima
    ranges [slabs, C] (uint32 bit patterns, as int32) from the producer of dY."""
    M, C = dY.shape
    dev = dY.device
    p = Params.make(bits, num_groups, round_mode, seed, offset, LAYOUT_TILED if tiled else LAYOUT_ROWS)
    lay_bytes, min_ld = sq_grad_layout_size(C, p)
    q_fold = code_matrix(M, min_ld, tiled, dev)
    q_t = code_matrix(C, M, tiled, dev)
    group = torch.empty(max(C, 1), dtype=torch.uint8, device=dev)[:C]
    scale = new_scale(dev)
    layout = torch.zeros(lay_bytes // 4, dtype=torch.int32, device=dev)
    ws = _workspace(sq_quantize_grad_workspace_size(M, C, p), dev)
    sq_quantize_grad_from_ranges(dY, p, ranges, ranges.shape[0], q_fold, q_t, group, scale, layout, ws, stream)
    return GradCodes(q_fold, q_t, group, scale, layout, p, M, C)


# sq_l1bn_channel (32 bytes) and sq_l1bn_layer (56 bytes) as int32 words
L1BN_CHANNEL_WORDS = 8
L1BN_LAYER_WORDS = 14


def l1bn_channels_to_host(chan: torch.Tensor) -> dict:
    w = chan.view(-1, L1BN_CHANNEL_WORDS).cpu()
    return {"mu": w[:, 0].numpy().copy(), "sigma": w[:, 1].numpy().copy(), "sign_sum": w[:, 2].numpy().copy(),
            "gamma_q": w[:, 3].view(torch.float32).numpy().copy(), "beta_q": w[:, 4].view(torch.float32).numpy().copy(),
            "kappa": w[:, 5].view(torch.float32).numpy().copy(),
            "dev_sum": w[:, 6:8].contiguous().view(torch.int64).reshape(-1).numpy().copy()}


def l1bn_layer_to_host(layer: torch.Tensor) -> dict:
    w = layer.cpu()
    i64 = w[0:4].view(torch.int64)
    return {"rows": int(i64[0]), "dev_max": int(i64[1]), "x_step": float(w[4:5].view(torch.float32)[0]),
            "flags": int(w[5])}


class L1BNState:
    """Forward state of an L1BNQ layer (device tensors)."""

    def __init__(self, chan, layer, xq, M, C):
        self.chan, self.layer, self.xq, self.M, self.C = chan, layer, xq, M, C


def l1bn_forward(xq: torch.Tensor, xscale: torch.Tensor, gamma: torch.Tensor, beta: torch.Tensor,
                 stream=None):
    """L1BNQ forward of 8-bit codes xq [M, C] (ld a multiple of 16):
    returns (y [M, C] fp32, L1BNState)."""
    M, C = xq.shape
    dev = xq.device
    y = torch.empty((M, C), dtype=torch.float32, device=dev)
    chan = torch.zeros(max(C, 1) * L1BN_CHANNEL_WORDS, dtype=torch.int32, device=dev)
    layer = torch.zeros(16, dtype=torch.int32, device=dev)
    ws = _workspace(sq_l1bn_forward_workspace_size(M, C), dev)
    sq_l1bn_forward(xq, xscale, gamma, beta, y, chan, layer, ws, stream)
    return y, L1BNState(chan, layer, xq, M, C)


def l1bn_backward(dy: torch.Tensor, state: L1BNState, bits: int = 8, num_groups: int = 4,
                  round_mode: int = ROUND_NEAREST_EVEN, seed: int = 0, offset: int = 0, want_ranges: bool = False,
                  stream=None) -> dict:
    """L1BNQ backward: dx, dgamma, dbeta, the gradient quantizer's group and
    scale, and (want_ranges) the partial maxima of |dx| per channel."""
    M, C = dy.shape
    dev = dy.device
    p = Params.make(bits, num_groups, round_mode, seed, offset)
    dx = torch.empty((M, C), dtype=torch.float32, device=dev)
    dgamma = torch.empty(max(C, 1), dtype=torch.float32, device=dev)[:C]
    dbeta = torch.empty(max(C, 1), dtype=torch.float32, device=dev)[:C]
    group = torch.empty(max(C, 1), dtype=torch.uint8, device=dev)[:C]
    gscale = new_scale(dev)
    ranges = None
    if want_ranges:
        ranges = torch.empty((sq_l1bn_range_slabs(M, C), max(C, 1)), dtype=torch.int32, device=dev)[:, :C]
    ws = _workspace(sq_l1bn_backward_workspace_size(M, C, p), dev)
    sq_l1bn_backward(dy, p, state.xq, state.chan, state.layer, dx, dgamma, dbeta, group, gscale, ranges, ws, stream)
    return {"dx": dx, "dgamma": dgamma, "dbeta": dbeta, "group": group, "gscale": gscale, "ranges": ranges}


def conv_pack_input(xq_t: torch.Tensor, N: int, H: int, W: int, KH: int, KW: int, PH: int, PW: int,
                    stream=None) -> torch.Tensor:
    """Input codes xq_t [C_in, >= N*H*W] packed for sq_conv_wgrad."""
    C_in = xq_t.shape[0]
    rows, ld, _ = sq_conv_wgrad_layout(N, H, W, C_in, KH, KW, PH, PW)
    xs = torch.empty((max(rows, 1), ld), dtype=torch.int8, device=xq_t.device)[:rows]
    sq_conv_pack_input(xq_t, N, H, W, C_in, KH, KW, PH, PW, xs, stream)
    return xs


def quantize_input_conv(X: torch.Tensor, N: int, H: int, W: int, KH: int, KW: int, PH: int, PW: int,
                        bits: int = 8, want_rows: bool = False, stream=None):
    """Per-tensor codes of the conv input X [N*H*W, C_in] on the padded grid of
    sq_conv_wgrad (a zero-filled buffer: the padding is never written), and,
    with want_rows, row-major as well: (xs, xq or None, scale)."""
    C_in = X.shape[1]
    dev = X.device
    rows, ld, _ = sq_conv_wgrad_layout(N, H, W, C_in, KH, KW, PH, PW)
    xs = torch.zeros((max(rows, 1), ld), dtype=torch.int8, device=dev)[:rows]
    xq = torch.empty((N * H * W, round_up(max(C_in, 1), 16)), dtype=torch.int8, device=dev)[:, :C_in] \
        if want_rows else None
    scale = new_scale(dev)
    ws = _workspace(sq_quantize_tensor_workspace_size(N * H * W, C_in), dev)
    sq_quantize_input_conv(X, N, H, W, KH, KW, PH, PW, bits, xq, xs, scale, ws, stream)
    return xs, xq, scale


def conv_pack_grad(codes: "GradCodes", N: int, H: int, W: int, KH: int, KW: int, PH: int, PW: int,
                   stream=None) -> torch.Tensor:
    """The transposed gradient codes of `codes` on the padded pixel grid."""
    _, _, qld = sq_conv_wgrad_layout(N, H, W, 1, KH, KW, PH, PW)
    q_tp = torch.empty((max(codes.C_out, 1), qld), dtype=torch.int8, device=codes.q_t.device)[:codes.C_out]
    sq_conv_pack_grad(codes.q_t, N, H, W, codes.C_out, KH, KW, PH, PW, q_tp, stream)
    return q_tp


def conv_wgrad(codes: "GradCodes", xs: torch.Tensor, xscale: torch.Tensor, N: int, H: int, W: int, C_in: int,
               KH: int, KW: int, PH: int, PW: int, want_acc: bool = False, q_tp: Optional[torch.Tensor] = None,
               stream=None):
    """Implicit-im2col conv wgrad: (dW [C_out, KH*KW*C_in] fp32, acc or None).
    q_tp: the padded gradient codes (sq_quantize_grad_conv); packed from
    codes.q_t when not given."""
    dev = codes.q_t.device
    C_out = codes.C_out
    if q_tp is None:
        q_tp = conv_pack_grad(codes, N, H, W, KH, KW, PH, PW, stream)
    Ng = KH * KW * C_in
    dW = torch.empty((max(C_out, 1), Ng), dtype=torch.float32, device=dev)[:C_out]
    acc = torch.empty((max(C_out, 1), Ng), dtype=torch.int32, device=dev)[:C_out] if want_acc else None
    ws = _workspace(sq_conv_wgrad_workspace_size(N, H, W, C_out, C_in, KH, KW, PH, PW, codes.params), dev)
    sq_conv_wgrad(q_tp, codes.group, codes.scale, xs, xscale, N, H, W, C_out, C_in, KH, KW, PH, PW,
                  codes.params, acc, dW, ws, stream)
    return dW, acc


class BackwardPlan:
    """All buffers of one backward step (quantize dY -> dgrad -> wgrad) for a
    fixed layer shape, allocated once; ``run`` enqueues the three calls and
    allocates nothing."""

    def __init__(self, M: int, C_out: int, C_in: int, params: Params, device="cuda",
                 want_acc: bool = False, grouped_dgrad: bool = False, dx_ranges: bool = False):
        self.M, self.C_out, self.C_in, self.params = M, C_out, C_in, params
        self.grouped_dgrad = grouped_dgrad
        # dx_ranges: the dgrad also writes the channel ranges of dX (for the
        # quantizer of the layer below, quantize_from_ranges)
        self.dX_ranges = (torch.empty((sq_gemm_dgrad_range_slabs(M), C_in), dtype=torch.int32,
                                      device=torch.device(device)) if dx_ranges else None)
        dev = torch.device(device)
        lay_bytes, min_ld = sq_grad_layout_size(C_out, params)
        # code matrices in the layout params.layout names (W^T and X^T codes
        # passed to dgrad / wgrad must be in the same one)
        self.q_fold = code_matrix(M, min_ld, params.tiled, dev)
        self.q_t = code_matrix(C_out, M, params.tiled, dev)
        self.group = torch.empty(C_out, dtype=torch.uint8, device=dev)
        self.scale = new_scale(dev)
        self.layout = torch.zeros(lay_bytes // 4, dtype=torch.int32, device=dev)
        self.ws_q = _workspace(sq_quantize_grad_workspace_size(M, C_out, params), dev)
        self.ws_d = _workspace((sq_gemm_dgrad_grouped_workspace_size if grouped_dgrad else
                                sq_gemm_dgrad_workspace_size)(M, C_out, C_in, params), dev)
        self.ws_w = _workspace(sq_gemm_wgrad_workspace_size(M, C_out, C_in, params), dev)
        self.dX = torch.empty((M, C_in), dtype=torch.float32, device=dev)
        self.dW = torch.empty((C_out, C_in), dtype=torch.float32, device=dev)
        self.acc_dX = torch.empty((M, C_in), dtype=torch.int32, device=dev) if want_acc else None
        self.acc_dW = torch.empty((C_out, C_in), dtype=torch.int32, device=dev) if want_acc else None

    def quantize(self, dY, stream=None):
        sq_quantize_grad(dY, self.params, self.q_fold, self.q_t, self.group, self.scale, self.layout,
                         self.ws_q, stream)

    def quantize_from_ranges(self, dY, ranges, stream=None):
        sq_quantize_grad_from_ranges(dY, self.params, ranges, ranges.shape[0], self.q_fold, self.q_t, self.group,
                                     self.scale, self.layout, self.ws_q, stream)

    def dgrad(self, wq_t, wscale, stream=None):
        if self.dX_ranges is not None:
            return sq_gemm_dgrad_ranged(self.q_fold, self.layout, self.group, self.scale, wq_t, wscale, self.M,
                                        self.C_out, self.C_in, self.params, self.acc_dX, self.dX, self.dX_ranges,
                                        self.ws_d, stream)
        fn = sq_gemm_dgrad_grouped if self.grouped_dgrad else sq_gemm_dgrad
        fn(self.q_fold, self.layout, self.group, self.scale, wq_t, wscale, self.M, self.C_out, self.C_in,
           self.params, self.acc_dX, self.dX, self.ws_d, stream)

    def wgrad(self, xq_t, xscale, stream=None):
        sq_gemm_wgrad(self.q_t, self.group, self.scale, xq_t, xscale, self.M, self.C_out, self.C_in,
                      self.params, self.acc_dW, self.dW, self.ws_w, stream)

    def run(self, dY, wq_t, wscale, xq_t, xscale, stream=None):
        self.quantize(dY, stream)
        self.dgrad(wq_t, wscale, stream)
        self.wgrad(xq_t, xscale, stream)
        return self.dX, self.dW


class ConvBackwardPlan(BackwardPlan):
    """Backward step of a stride-1 convolution lowered by im2col, with the input
    gradient taken by sq_conv_dgrad (implicit im2col and col2im: dX is
    [N*H*W, C_in_ch], NHWC) and the weight gradient by sq_conv_wgrad on the
    packed input codes (implicit_wgrad, the default: ``run`` takes the output
    of conv_pack_input as its xq_t argument, ``run_packed`` the input codes
    xq_t [C_in, >= N*H*W] of sq_quantize_tensor, which it packs onto the
    plan's grid first) or by sq_gemm_wgrad on the im2col'd activations.
    Buffers are allocated once; ``run`` and ``run_packed`` allocate nothing."""

    def __init__(self, N: int, H: int, W: int, C_out: int, C_in_ch: int, KH: int, KW: int, PH: int, PW: int,
                 params: Params, device="cuda", want_acc: bool = False, implicit_wgrad: bool = True,
                 dx_ranges: bool = False):
        Ho, Wo = H + 2 * PH - KH + 1, W + 2 * PW - KW + 1
        super().__init__(N * Ho * Wo, C_out, KH * KW * C_in_ch, params, device, want_acc)
        dev = torch.device(device)
        # dx_ranges: the dgrad also writes the channel ranges of dX (for the
        # quantizer of the layer below, quantize_from_ranges); range_slabs is
        # the number of slab rows the last dgrad wrote
        self.dX_ranges = (torch.empty((sq_gemm_dgrad_range_slabs(N * H * W), C_in_ch), dtype=torch.int32,
                                      device=dev) if dx_ranges else None)
        self.range_slabs, self.range_rows = 0, 0
        self.geom = (N, H, W, KH, KW, PH, PW)
        self.C_in_ch = C_in_ch
        self.implicit_wgrad = implicit_wgrad
        if implicit_wgrad:
            self.ws_w = _workspace(sq_conv_wgrad_workspace_size(N, H, W, C_out, C_in_ch, KH, KW, PH, PW, params), dev)
            _, _, qld = sq_conv_wgrad_layout(N, H, W, C_in_ch, KH, KW, PH, PW)
            # the quantizer never writes the padding of the grid: zero it once
            self.q_tp = torch.zeros((C_out, qld), dtype=torch.int8, device=dev)
            self.q_t = None
            # the input codes on the grid (written whole by pack_input; the
            # input quantizer writes the pixels only, so the padding is zeroed
            # once)
            xrows, xld, _ = sq_conv_wgrad_layout(N, H, W, C_in_ch, KH, KW, PH, PW)
            self.x_grid = torch.zeros((max(xrows, 1), xld), dtype=torch.int8, device=dev)[:xrows]
            self.x_scale = new_scale(dev)
            self.ws_x = _workspace(sq_quantize_tensor_workspace_size(N * H * W, C_in_ch), dev)
        self.ws_d = _workspace(sq_conv_dgrad_workspace_size(C_out, C_in_ch, KH, KW, params), dev)
        self.dX = torch.empty((N * H * W, C_in_ch), dtype=torch.float32, device=dev)
        self.acc_dX = torch.empty((N * H * W, C_in_ch), dtype=torch.int32, device=dev) if want_acc else None

    def dgrad(self, wq_t, wscale, stream=None):
        N, H, W, KH, KW, PH, PW = self.geom
        if self.dX_ranges is not None:
            self.range_slabs, self.range_rows = sq_conv_dgrad_ranged(
                self.q_fold, self.layout, self.group, self.scale, wq_t, wscale, N, H, W, self.C_out, self.C_in_ch,
                KH, KW, PH, PW, self.params, self.acc_dX, self.dX, self.dX_ranges, self.ws_d, stream)
            return
        sq_conv_dgrad(self.q_fold, self.layout, self.group, self.scale, wq_t, wscale, N, H, W, self.C_out,
                      self.C_in_ch, KH, KW, PH, PW, self.params, self.acc_dX, self.dX, self.ws_d, stream)

    def quantize(self, dY, stream=None):
        if not self.implicit_wgrad:
            return super().quantize(dY, stream)
        N, H, W, KH, KW, PH, PW = self.geom
        sq_quantize_grad_conv(dY, N, H, W, KH, KW, PH, PW, self.params, self.q_fold, self.q_tp, self.group,
                              self.scale, self.layout, self.ws_q, stream)

    def quantize_from_ranges(self, dY, ranges, stream=None, range_slabs=None):
        """Quantize dY with channel ranges from its producer (e.g. the
        dX_ranges of the layer above's ranged dgrad)."""
        slabs = ranges.shape[0] if range_slabs is None else range_slabs
        if not self.implicit_wgrad:
            return sq_quantize_grad_from_ranges(dY, self.params, ranges, slabs, self.q_fold, self.q_t, self.group,
                                                self.scale, self.layout, self.ws_q, stream)
        N, H, W, KH, KW, PH, PW = self.geom
        sq_quantize_grad_conv_from_ranges(dY, N, H, W, KH, KW, PH, PW, self.params, ranges, slabs, self.q_fold,
                                          self.q_tp, self.group, self.scale, self.layout, self.ws_q, stream)

    def pack_input(self, xq_t, stream=None):
        """The input codes xq_t [C_in, >= N*H*W] onto the plan's padded grid."""
        N, H, W, KH, KW, PH, PW = self.geom
        sq_conv_pack_input(xq_t, N, H, W, self.C_in_ch, KH, KW, PH, PW, self.x_grid, stream)

    def quantize_input(self, X, stream=None):
        """The forward pass's input quantizer: per-tensor 8-bit codes of X
        [N*H*W, C_in] straight onto the plan's grid (x_grid, x_scale), so the
        step runs without pack_input."""
        N, H, W, KH, KW, PH, PW = self.geom
        sq_quantize_input_conv(X, N, H, W, KH, KW, PH, PW, 8, None, self.x_grid, self.x_scale, self.ws_x, stream)

    def run_packed(self, dY, wq_t, wscale, xq_t, xscale, stream=None):
        """The step from unpacked input codes: pack_input, then run."""
        self.pack_input(xq_t, stream)
        return self.run(dY, wq_t, wscale, self.x_grid, xscale, stream)

    def wgrad(self, xq_t, xscale, stream=None):
        if not self.implicit_wgrad:
            return super().wgrad(xq_t, xscale, stream)
        N, H, W, KH, KW, PH, PW = self.geom
        sq_conv_wgrad(self.q_tp, self.group, self.scale, xq_t, xscale, N, H, W, self.C_out, self.C_in_ch, KH, KW,
                      PH, PW, self.params, self.acc_dW, self.dW, self.ws_w, stream)
