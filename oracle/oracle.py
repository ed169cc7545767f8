"""numpy front end of the C oracle (oracle/sq_oracle.c).  TEST INFRASTRUCTURE ONLY.

Every function here marshals numpy arrays into the plain C implementation and
back; the arithmetic lives in sq_oracle.c, whose header lists the readings of
the paper it follows.
"""
from __future__ import annotations

import ctypes as ct
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")

FLAG_NONFINITE = 1
FLAG_ZERO = 2
ROUND_NEAREST_EVEN = 0
ROUND_STOCHASTIC = 1


class _Scale(ct.Structure):
    _fields_ = [("r_max", ct.c_float), ("inv0", ct.c_float), ("d0", ct.c_float), ("flags", ct.c_uint32)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH) or (
                os.path.getmtime(_LIB_PATH) < os.path.getmtime(os.path.join(_HERE, "sq_oracle.c"))):
            from . import build as _b
            _b.build()
        _lib = _bind(ct.CDLL(_LIB_PATH))
    return _lib


def use_library(path):
    """Bind the oracle front end to another build of sq_oracle.c (used by the
    mutation tests, which compile deliberately broken copies); returns the
    previously bound library so it can be restored with restore_library()."""
    global _lib
    prev = lib()
    _lib = _bind(ct.CDLL(path))
    return prev


def restore_library(prev):
    global _lib
    _lib = prev


def _bind(L):
    P = ct.c_void_p
    i64 = ct.c_int64
    L.sqo_philox4x32_10.argtypes = [P, P, P]
    L.sqo_philox4x32_10.restype = None
    L.sqo_sr_uniform16.argtypes = [ct.c_uint64, ct.c_uint64, ct.c_uint64]
    L.sqo_sr_uniform16.restype = ct.c_uint32
    L.sqo_channel_range.argtypes = [P, i64, i64, i64, P, P]
    L.sqo_channel_range.restype = ct.c_int
    L.sqo_group_of.argtypes = [ct.c_float, ct.c_float, ct.c_int]
    L.sqo_group_of.restype = ct.c_int
    L.sqo_quantize_grad.argtypes = [P, i64, i64, i64, ct.c_int, ct.c_int, ct.c_int,
                                    ct.c_uint64, ct.c_uint64, P, P, P, P]
    L.sqo_quantize_grad.restype = ct.c_int
    L.sqo_quantize_tensor.argtypes = [P, i64, i64, i64, ct.c_int, P, P]
    L.sqo_quantize_tensor.restype = ct.c_int
    L.sqo_dgrad.argtypes = [P, i64, i64, P, ct.c_int, P, i64, P, i64, P]
    L.sqo_dgrad.restype = ct.c_int
    L.sqo_conv_dgrad.argtypes = [P, i64, i64, i64, i64, P, ct.c_int, P, i64, ct.c_int, ct.c_int, ct.c_int,
                                 ct.c_int, P, i64, P]
    L.sqo_conv_dgrad.restype = ct.c_int
    L.sqo_quantize_channels.argtypes = [P, i64, i64, i64, ct.c_int, ct.c_int, P, P]
    L.sqo_quantize_channels.restype = ct.c_int
    L.sqo_dequant_cols.argtypes = [P, i64, i64, ct.c_float, P, ct.c_int, P]
    L.sqo_dequant_cols.restype = None
    L.sqo_wgrad.argtypes = [P, i64, i64, P, i64, P, i64, P]
    L.sqo_wgrad.restype = ct.c_int
    L.sqo_dequant_dgrad.argtypes = [P, i64, ct.c_float, ct.c_float, ct.c_int, P]
    L.sqo_dequant_dgrad.restype = None
    L.sqo_dequant_wgrad.argtypes = [P, i64, i64, P, ct.c_float, ct.c_float, P]
    L.sqo_dequant_wgrad.restype = None
    L.sqo_conv_wgrad.argtypes = [P, i64, i64, i64, i64, P, i64, ct.c_int, ct.c_int, ct.c_int, ct.c_int, P]
    L.sqo_conv_wgrad.restype = ct.c_int
    L.sqo_l1bn_forward.argtypes = [P, i64, i64, ct.c_float, P, P, P, P, P, P, P, P, P, P, P]
    L.sqo_l1bn_forward.restype = ct.c_int
    L.sqo_l1bn_backward.argtypes = [P, P, ct.c_float, i64, i64, P, ct.c_float, P, P, P, P, i64, P, P, P]
    L.sqo_l1bn_backward.restype = ct.c_int
    L.sqo_set_threads.argtypes = [ct.c_int]
    L.sqo_set_threads.restype = ct.c_int
    L.sqo_max_threads.argtypes = []
    L.sqo_max_threads.restype = ct.c_int
    return L


def set_threads(n: int) -> int:
    """Threads of the oracle's OpenMP loops (1 = plain serial loops).  The
    results do not depend on it: each output is computed by one thread."""
    return int(lib().sqo_set_threads(int(n)))


def max_threads() -> int:
    """Processors OpenMP sees on this host."""
    return int(lib().sqo_max_threads())


def _p(a: np.ndarray):
    return a.ctypes.data_as(ct.c_void_p)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def _scale_dict(s: _Scale) -> dict:
    return {"r_max": np.float32(s.r_max), "inv0": np.float32(s.inv0), "d0": np.float32(s.d0),
            "flags": int(s.flags)}


def philox4x32_10(counter, key) -> np.ndarray:
    """Philox4x32-10 block function: 4 counter words, 2 key words -> 4 words."""
    c = _c(counter, np.uint32)
    k = _c(key, np.uint32)
    out = np.zeros(4, np.uint32)
    lib().sqo_philox4x32_10(_p(c), _p(k), _p(out))
    return out


def sr_uniform16(idx: int, seed: int, offset: int) -> int:
    return int(lib().sqo_sr_uniform16(idx, seed, offset))


def channel_range(x: np.ndarray):
    x = _c(x, np.float32)
    M, C = x.shape
    r = np.zeros(C, np.float32)
    nf = ct.c_int(0)
    rc = lib().sqo_channel_range(_p(x), M, C, C, _p(r), ct.byref(nf))
    assert rc == 0
    return r, bool(nf.value)


def group_of(r_c: float, r_max: float, num_groups: int) -> int:
    return int(lib().sqo_group_of(float(r_c), float(r_max), int(num_groups)))


def quantize_grad(dY: np.ndarray, bits: int, num_groups: int, round_mode: int = 0,
                  seed: int = 0, offset: int = 0):
    """ShiftQuant of dY [M, C] -> (codes int8 [M, C], group uint8 [C], scale dict, r [C])."""
    dY = _c(dY, np.float32)
    M, C = dY.shape
    q = np.zeros((M, C), np.int8)
    g = np.zeros(C, np.uint8)
    r = np.zeros(max(C, 1), np.float32)
    s = _Scale()
    rc = lib().sqo_quantize_grad(_p(dY), M, C, C, bits, num_groups, round_mode, seed, offset,
                                 _p(q), _p(g), _p(r), ct.byref(s))
    if rc:
        raise ValueError(f"sqo_quantize_grad failed ({rc})")
    return q, g, _scale_dict(s), r[:C]


def quantize_tensor(T: np.ndarray, bits: int = 8):
    """Per-tensor symmetric quantization -> (codes int8 like T, scale dict)."""
    T = _c(T, np.float32)
    rows, cols = T.shape
    q = np.zeros((rows, cols), np.int8)
    s = _Scale()
    rc = lib().sqo_quantize_tensor(_p(T), rows, cols, cols, bits, _p(q), ct.byref(s))
    if rc:
        raise ValueError(f"sqo_quantize_tensor failed ({rc})")
    return q, _scale_dict(s)


class RangeError(ValueError):
    pass


def dgrad(q: np.ndarray, g: np.ndarray, num_groups: int, wq: np.ndarray, rows=None) -> np.ndarray:
    """A[n, k] = sum_c (q[n, c] * wq[c, k]) << (N_G-1-g_c), int32 (selected rows)."""
    q = _c(q, np.int8)
    g = _c(g, np.uint8)
    wq = _c(wq, np.int8)
    M, C_out = q.shape
    C_in = wq.shape[1]
    assert wq.shape[0] == C_out and g.shape[0] == C_out
    if rows is None:
        A = np.zeros((M, C_in), np.int32)
        rc = lib().sqo_dgrad(_p(q), M, C_out, _p(g), num_groups, _p(wq), C_in, None, 0, _p(A))
    else:
        rows = _c(rows, np.int64)
        A = np.zeros((rows.shape[0], C_in), np.int32)
        rc = lib().sqo_dgrad(_p(q), M, C_out, _p(g), num_groups, _p(wq), C_in, _p(rows),
                             rows.shape[0], _p(A))
    if rc == 2:
        raise RangeError("dgrad accumulator leaves int32")
    assert rc == 0
    return A


def quantize_channels(T: np.ndarray, bits: int = 8, axis: int = 0):
    """Per-channel symmetric quantization: one scale per row (axis 0) or
    column (axis 1).  Returns (codes int8 [rows, cols], list of scale dicts)."""
    T = _c(T, np.float32)
    rows, cols = T.shape
    q = np.zeros((rows, cols), np.int8)
    n = rows if axis == 0 else cols
    sc = (_Scale * max(n, 1))()
    rc = lib().sqo_quantize_channels(_p(T), rows, cols, cols, bits, axis, _p(q), ct.cast(sc, ct.c_void_p))
    assert rc == 0
    return q, [_scale_dict(sc[i]) for i in range(n)]


def dequant_cols(A: np.ndarray, d_a, d_w: np.ndarray, num_groups: int) -> np.ndarray:
    """out[i, k] = fl(float(A[i, k]) * fl(fl(d_a * d_w[k]) * 2^-(N_G-1)))."""
    A = _c(A, np.int32)
    d_w = _c(d_w, np.float32)
    n_rows, n_cols = A.shape
    assert d_w.shape[0] == n_cols
    out = np.zeros(A.shape, np.float32)
    lib().sqo_dequant_cols(_p(A), n_rows, n_cols, float(d_a), _p(d_w), num_groups, _p(out))
    return out


def conv_dgrad(q: np.ndarray, g: np.ndarray, num_groups: int, wq: np.ndarray, N: int, H: int, W: int,
               KH: int, KW: int, PH: int, PW: int, pix=None) -> np.ndarray:
    """Input gradient of a stride-1 convolution, int32: the col2im of the
    im2col'd ShiftMM dgrad (sqo_conv_dgrad).  q [N*Ho*Wo, C_out] codes of dY
    (NHWC), wq [C_out, KH*KW*C_in] in (r, s, ci) column order; returns
    A [N*H*W, C_in] (or the listed input pixels)."""
    q = _c(q, np.int8)
    g = _c(g, np.uint8)
    wq = _c(wq, np.int8)
    C_out = q.shape[1]
    C_in = wq.shape[1] // (KH * KW)
    assert wq.shape == (C_out, KH * KW * C_in) and g.shape[0] == C_out
    Ho, Wo = H + 2 * PH - KH + 1, W + 2 * PW - KW + 1
    assert q.shape[0] == N * Ho * Wo
    if pix is None:
        A = np.zeros((N * H * W, C_in), np.int32)
        rc = lib().sqo_conv_dgrad(_p(q), N, H, W, C_out, _p(g), num_groups, _p(wq), C_in, KH, KW, PH, PW,
                                  None, 0, _p(A))
    else:
        pix = _c(pix, np.int64)
        A = np.zeros((pix.shape[0], C_in), np.int32)
        rc = lib().sqo_conv_dgrad(_p(q), N, H, W, C_out, _p(g), num_groups, _p(wq), C_in, KH, KW, PH, PW,
                                  _p(pix), pix.shape[0], _p(A))
    if rc == 2:
        raise RangeError("conv dgrad accumulator leaves int32")
    assert rc == 0, rc
    return A


def conv_wgrad(q: np.ndarray, xq: np.ndarray, N: int, H: int, W: int, KH: int, KW: int, PH: int,
               PW: int) -> np.ndarray:
    """Weight gradient of a stride-1 conv: B [C_out, KH*KW*C_in] int32 from
    gradient codes q [N*Ho*Wo, C_out] and input codes xq [N*H*W, C_in]."""
    q = _c(q, np.int8)
    xq = _c(xq, np.int8)
    C_out, C_in = q.shape[1], xq.shape[1]
    B = np.zeros((C_out, KH * KW * C_in), np.int32)
    rc = lib().sqo_conv_wgrad(_p(q), N, H, W, C_out, _p(xq), C_in, KH, KW, PH, PW, _p(B))
    if rc == 2:
        raise RangeError("conv wgrad accumulator leaves int32")
    assert rc == 0, rc
    return B


def wgrad(q: np.ndarray, xq: np.ndarray, rows=None) -> np.ndarray:
    """B[c, k] = sum_m q[m, c] * xq[m, k], int32 (selected output channels)."""
    q = _c(q, np.int8)
    xq = _c(xq, np.int8)
    M, C_out = q.shape
    C_in = xq.shape[1]
    assert xq.shape[0] == M
    if rows is None:
        B = np.zeros((C_out, C_in), np.int32)
        rc = lib().sqo_wgrad(_p(q), M, C_out, _p(xq), C_in, None, 0, _p(B))
    else:
        rows = _c(rows, np.int64)
        B = np.zeros((rows.shape[0], C_in), np.int32)
        rc = lib().sqo_wgrad(_p(q), M, C_out, _p(xq), C_in, _p(rows), rows.shape[0], _p(B))
    if rc == 2:
        raise RangeError("wgrad accumulator leaves int32")
    assert rc == 0
    return B


def dequant_dgrad(A: np.ndarray, d_grad, d_w, num_groups: int) -> np.ndarray:
    A = _c(A, np.int32)
    out = np.zeros(A.shape, np.float32)
    lib().sqo_dequant_dgrad(_p(A), A.size, float(d_grad), float(d_w), num_groups, _p(out))
    return out


def dequant_wgrad(B: np.ndarray, g_rows: np.ndarray, d_grad, d_x) -> np.ndarray:
    B = _c(B, np.int32)
    g_rows = _c(g_rows, np.uint8)
    n_rows, C_in = B.shape
    assert g_rows.shape[0] == n_rows
    out = np.zeros(B.shape, np.float32)
    lib().sqo_dequant_wgrad(_p(B), n_rows, C_in, _p(g_rows), float(d_grad), float(d_x), _p(out))
    return out


def backward(dY, W, X, bits, num_groups, round_mode=0, seed=0, offset=0,
             dgrad_rows=None, wgrad_rows=None) -> dict:
    """Whole oracle path: quantize dY, W, X; dgrad; wgrad; dequantize."""
    q, g, gs, _ = quantize_grad(dY, bits, num_groups, round_mode, seed, offset)
    wq, ws = quantize_tensor(W, 8)
    xq, xs = quantize_tensor(X, 8)
    A = dgrad(q, g, num_groups, wq, dgrad_rows)
    B = wgrad(q, xq, wgrad_rows)
    g_rows = g if wgrad_rows is None else g[np.asarray(wgrad_rows)]
    dX = dequant_dgrad(A, gs["d0"], ws["d0"], num_groups)
    dW = dequant_wgrad(B, g_rows, gs["d0"], xs["d0"])
    return {"q": q, "g": g, "gscale": gs, "wq": wq, "wscale": ws, "xq": xq, "xscale": xs,
            "A": A, "B": B, "dX": dX, "dW": dW}


def l1bn_forward(xq: np.ndarray, x_step: float, gamma: np.ndarray, beta: np.ndarray) -> dict:
    """L1BNQ forward (Sec. 4, App. C) of 8-bit codes xq [M, C] with step
    x_step: y fp32 [M, C] and the per-channel state (mu / sigma codes, sign
    and deviation sums, quantized gamma / beta, kappa) plus dev_max."""
    xq = _c(xq, np.int8)
    M, C = xq.shape
    gamma = _c(gamma, np.float32)
    beta = _c(beta, np.float32)
    assert gamma.shape == (C,) and beta.shape == (C,)
    n = max(C, 1)
    y = np.zeros((M, C), np.float32)
    mu = np.zeros(n, np.int32)
    sigma = np.zeros(n, np.int32)
    sign_sum = np.zeros(n, np.int32)
    dev_sum = np.zeros(n, np.int64)
    gq = np.zeros(n, np.float32)
    bq = np.zeros(n, np.float32)
    kappa = np.zeros(n, np.float32)
    dev_max = ct.c_int64(0)
    rc = lib().sqo_l1bn_forward(_p(xq), M, C, float(x_step), _p(gamma), _p(beta), _p(y), _p(mu), _p(sigma),
                                _p(sign_sum), _p(dev_sum), _p(gq), _p(bq), _p(kappa), ct.byref(dev_max))
    if rc:
        raise ValueError(f"sqo_l1bn_forward failed ({rc})")
    return {"y": y, "mu": mu[:C], "sigma": sigma[:C], "sign_sum": sign_sum[:C], "dev_sum": dev_sum[:C],
            "gamma_q": gq[:C], "beta_q": bq[:C], "kappa": kappa[:C], "dev_max": int(dev_max.value),
            "x_step": float(np.float32(x_step)), "M": M}


def l1bn_backward(dy: np.ndarray, fwd: dict, xq: np.ndarray, bits: int = 8, num_groups: int = 4,
                  round_mode: int = 0, seed: int = 0, offset: int = 0) -> dict:
    """L1BNQ backward: ShiftQuant of dy, then dx, dgamma, dbeta from the
    forward state `fwd` (as returned by l1bn_forward)."""
    dy = _c(dy, np.float32)
    xq = _c(xq, np.int8)
    M, C = dy.shape
    assert xq.shape == (M, C)
    qg, grp, gs, _ = quantize_grad(dy, bits, num_groups, round_mode, seed, offset)
    dx = np.zeros((M, C), np.float32)
    n = max(C, 1)
    dgamma = np.zeros(n, np.float32)
    dbeta = np.zeros(n, np.float32)
    f = {k: _c(fwd[k], np.int32) for k in ("mu", "sigma", "sign_sum")}
    gq = _c(fwd["gamma_q"], np.float32)
    rc = lib().sqo_l1bn_backward(_p(qg), _p(grp), float(gs["d0"]), M, C, _p(xq), float(fwd["x_step"]),
                                 _p(f["mu"]), _p(f["sigma"]), _p(f["sign_sum"]), _p(gq), int(fwd["dev_max"]),
                                 _p(dx), _p(dgamma), _p(dbeta))
    if rc:
        raise ValueError(f"sqo_l1bn_backward failed ({rc})")
    return {"dx": dx, "dgamma": dgamma[:C], "dbeta": dbeta[:C], "qg": qg, "group": grp, "gscale": gs}
