"""Seeded synthetic inputs for the ShiftQuant backward path.

This module draws random tensors and nothing else: it holds none of the
quantizer's or the GEMMs' arithmetic, so both the HIP path and the CPU oracle
can consume the same bytes without sharing any method code.

The five layer workloads stand in for the paper's ResNet and Transformer
training runs (Sec. 5.1, Tables "resnet" and "transformer"); no dataset or
trained weight is used.  Gradients are drawn with a heavy-tailed per-channel
scale, because the paper motivates ShiftQuant with gradients whose channel
ranges differ by orders of magnitude and carry outlier channels (Sec. 3,
Fig. "meth"; Sec. 1).

Recipe (every tensor is sampled in float64 and rounded once to float32):

* dY[m, c] = z[m, c] * sigma_c, with z ~ N(0, 1) (Student-t(3) for the MLP
  workload) and sigma_c ~ LogNormal(0, s).  A chosen set of channels (the
  count is round-half-even(frac * C_out), at least 1) has sigma multiplied by
  an outlier factor.
* X and W follow the per-workload distributions in ``WORKLOADS``.
* Generator: numpy ``PCG64(SeedSequence([seed, workload_index, tensor_id]))``
  with tensor ids 0 = sigma vector, 1 = outlier choice, 2 = dY base,
  3 = X, 4 = W.
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np

TID_SIGMA, TID_OUTLIER, TID_DY, TID_X, TID_W = 0, 1, 2, 3, 4

ROUND_NEAREST_EVEN = 0
ROUND_STOCHASTIC = 1


@dataclasses.dataclass(frozen=True)
class Workload:
    """One backward layer: dY [M, C_out], W [C_out, C_in], X [M, C_in]."""
    name: str
    index: int
    M: int
    C_out: int
    C_in: int
    bits: int
    num_groups: int
    round_mode: int
    description: str
    # dY recipe
    dy_dist: str          # "normal" or "student_t3"
    sigma_lognormal_s: float
    outlier_frac: float   # 0 disables outliers
    outlier_factor: float
    # X recipe
    x_kind: str           # "normal", "relu_normal", "conv3x3_relu"
    x_std: float
    # W recipe
    w_std: float
    # conv geometry (only for x_kind == "conv3x3_relu")
    conv_hw: int = 0
    conv_cin: int = 0
    sr_seed: int = 0
    sr_offset: int = 0

    @property
    def ops(self) -> int:
        """Integer ops of one backward step: two GEMMs of 2*M*C_out*C_in."""
        return 4 * self.M * self.C_out * self.C_in


WORKLOADS = {
    w.name: w for w in [
        Workload("linear_256", 0, 256, 256, 256, 4, 4, ROUND_NEAREST_EVEN,
                 "single linear layer backward, 4-bit gradients",
                 "normal", 1.0, 0.02, 100.0, "normal", 0.02, 0.02),
        Workload("resnet18_conv3x3", 1, 64 * 56 * 56, 64, 64 * 9, 4, 4, ROUND_NEAREST_EVEN,
                 "ResNet-18 3x3 conv 64->64 at 56x56, batch 64, im2col GEMM",
                 "normal", 1.0, 0.02, 100.0, "conv3x3_relu", 1.0, float(np.sqrt(2.0 / 576.0)),
                 conv_hw=56, conv_cin=64),
        Workload("resnet50_conv1x1", 2, 64 * 14 * 14, 256, 1024, 4, 4, ROUND_NEAREST_EVEN,
                 "ResNet-50 1x1 bottleneck conv 1024->256 at 14x14, batch 64",
                 "normal", 1.0, 0.02, 100.0, "relu_normal", 1.0, float(np.sqrt(2.0 / 1024.0))),
        Workload("mlp_up_768x3072", 3, 32 * 512, 3072, 768, 6, 4, ROUND_NEAREST_EVEN,
                 "Transformer MLP up-projection 768->3072, 32x512 tokens, 6-bit gradients",
                 "student_t3", 1.5, 0.0, 1.0, "normal", 1.0, 0.02),
        Workload("linear_4096x11008_sr", 4, 8192, 11008, 4096, 6, 4, ROUND_STOCHASTIC,
                 "large Transformer linear 4096->11008, 8192 tokens, 6-bit SR gradients",
                 "normal", 2.0, 0.005, 1000.0, "normal", 1.0, 0.02),
    ]
}
WORKLOAD_ORDER = sorted(WORKLOADS, key=lambda n: WORKLOADS[n].index)


def _rng(seed: int, index: int, tid: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, index, tid])))


def outlier_count(frac: float, C: int) -> int:
    if frac <= 0.0:
        return 0
    return max(1, int(np.rint(frac * C)))  # np.rint rounds half to even


def make_grad(M: int, C: int, *, seed: int = 0, index: int = 0, dist: str = "normal",
              sigma_s: float = 1.0, outlier_frac: float = 0.02,
              outlier_factor: float = 100.0) -> np.ndarray:
    """Heavy-tailed output gradient dY [M, C] float32 (recipe in the module doc)."""
    sigma = _rng(seed, index, TID_SIGMA).lognormal(0.0, sigma_s, size=C)
    k = outlier_count(outlier_frac, C)
    if k:
        idx = _rng(seed, index, TID_OUTLIER).choice(C, size=k, replace=False)
        sigma[idx] *= outlier_factor
    r = _rng(seed, index, TID_DY)
    if dist == "normal":
        z = r.standard_normal(size=(M, C))
    elif dist == "student_t3":
        z = r.standard_t(3.0, size=(M, C))
    else:
        raise ValueError(dist)
    z *= sigma[None, :]
    return z.astype(np.float32)


def im2col_3x3(x_nhwc: np.ndarray) -> np.ndarray:
    """Stride-1, pad-1 3x3 im2col of an NHWC tensor, columns in (kh, kw, c) order."""
    n, h, w, c = x_nhwc.shape
    xp = np.zeros((n, h + 2, w + 2, c), dtype=x_nhwc.dtype)
    xp[:, 1:h + 1, 1:w + 1, :] = x_nhwc
    out = np.empty((n, h, w, 9, c), dtype=x_nhwc.dtype)
    for kh in range(3):
        for kw in range(3):
            out[:, :, :, kh * 3 + kw, :] = xp[:, kh:kh + h, kw:kw + w, :]
    return out.reshape(n * h * w, 9 * c)


def make_inputs(name: str, *, M: Optional[int] = None, seed: int = 0) -> dict:
    """dY, X, W (float32) for workload ``name``.

    ``M`` overrides the token/pixel count with the same recipe (for the conv
    workload it must be a multiple of H*W and selects the batch size).
    """
    wl = WORKLOADS[name]
    M = wl.M if M is None else int(M)
    dY = make_grad(M, wl.C_out, seed=seed, index=wl.index, dist=wl.dy_dist,
                   sigma_s=wl.sigma_lognormal_s, outlier_frac=wl.outlier_frac,
                   outlier_factor=wl.outlier_factor)
    rx = _rng(seed, wl.index, TID_X)
    if wl.x_kind == "normal":
        X = (rx.standard_normal(size=(M, wl.C_in)) * wl.x_std).astype(np.float32)
    elif wl.x_kind == "relu_normal":
        X = np.maximum(rx.standard_normal(size=(M, wl.C_in)), 0.0).astype(np.float32)
    elif wl.x_kind == "conv3x3_relu":
        hw = wl.conv_hw * wl.conv_hw
        if M % hw:
            raise ValueError(f"conv workload needs M to be a multiple of {hw}")
        x = np.maximum(rx.standard_normal(size=(M // hw, wl.conv_hw, wl.conv_hw, wl.conv_cin)),
                       0.0).astype(np.float32)
        X = im2col_3x3(x)
    else:
        raise ValueError(wl.x_kind)
    rw = _rng(seed, wl.index, TID_W)
    W = (rw.standard_normal(size=(wl.C_out, wl.C_in)) * wl.w_std).astype(np.float32)
    return {"dY": dY, "X": X, "W": W, "workload": wl, "M": M}


# ---------------------------------------------------------------------------
# L1BNQ layers (Sec. 4: 8-bit fully-quantized L1 batch normalization in the
# ResNets and the Transformer of Sec. 5.1).  The layer's input is a conv (or
# linear) output, so X is signed: z * sigma_c + mean_c with z ~ N(0, 1),
# sigma_c ~ LogNormal(0, 0.5), mean_c ~ N(0, 0.5); gamma ~ N(1, 0.2),
# beta ~ N(0, 0.2); the incoming gradient dy follows make_grad with
# LogNormal(0, 1) channel scales and its default outlier channels.  Tensor ids continue after those above:
# 5 = X, 6 = gamma / beta, 7 = dy base (via make_grad's ids with index + 100).
# ---------------------------------------------------------------------------
TID_BN_X, TID_BN_PARAM = 5, 6


@dataclasses.dataclass(frozen=True)
class BNWorkload:
    name: str
    index: int
    M: int          # N * H * W rows
    C: int          # channels
    description: str


BN_WORKLOADS = {w.name: w for w in [
    BNWorkload("resnet18_bn_56x56x64", 10, 64 * 56 * 56, 64,
               "ResNet-18 stage-1 batch norm, N=64, 56x56, 64 channels"),
    BNWorkload("resnet50_bn_14x14x1024", 11, 64 * 14 * 14, 1024,
               "ResNet-50 stage-3 batch norm, N=64, 14x14, 1024 channels"),
    BNWorkload("transformer_bn_768", 12, 16384, 768,
               "Transformer batch norm over 16384 tokens of width 768"),
]}


def make_bn_inputs(name: str, *, seed: int = 0) -> dict:
    w = BN_WORKLOADS[name]
    rx = _rng(seed, w.index, TID_BN_X)
    sig = rx.lognormal(0.0, 0.5, w.C)
    mean = rx.normal(0.0, 0.5, w.C)
    X = (rx.standard_normal((w.M, w.C)) * sig + mean).astype(np.float32)
    rp = _rng(seed, w.index, TID_BN_PARAM)
    gamma = rp.normal(1.0, 0.2, w.C).astype(np.float32)
    beta = rp.normal(0.0, 0.2, w.C).astype(np.float32)
    dy = make_grad(w.M, w.C, seed=seed, index=w.index + 100, dist="normal", sigma_s=1.0)
    return {"X": X, "gamma": gamma, "beta": beta, "dy": dy, "M": w.M, "C": w.C}


# ---------------------------------------------------------------------------
# Two-layer chain of the Transformer MLP: the down-projection (3072 -> 768)
# backward produces, as its input gradient, the output gradient of the
# up-projection (768 -> 3072, the mlp_up_768x3072 workload).  The chain's own
# tensors: dY of the down-projection [16384, 768] (the MLP recipe: Student-t(3)
# times LogNormal(0, 1.5) channel scales), its weight W_dn [768, 3072] ~
# N(0, 0.02) and its input X_dn [16384, 3072] ~ N(0, 1) (tensor ids 8, 9, 10).
# ---------------------------------------------------------------------------
def make_chain_inputs(seed: int = 0) -> dict:
    up = make_inputs("mlp_up_768x3072", seed=seed)
    M = up["M"]
    wl = up["workload"]
    dy_dn = make_grad(M, wl.C_in, seed=seed, index=wl.index + 200, dist="student_t3", sigma_s=1.5,
                      outlier_frac=0.0)
    w_dn = (_rng(seed, wl.index, 9).standard_normal((wl.C_in, wl.C_out)) * 0.02).astype(np.float32)
    x_dn = _rng(seed, wl.index, 10).standard_normal((M, wl.C_out)).astype(np.float32)
    return {"dY_dn": dy_dn, "W_dn": w_dn, "X_dn": x_dn, "W_up": up["W"], "X_up": up["X"], "M": M,
            "d_model": wl.C_in, "d_ff": wl.C_out, "bits": wl.bits, "num_groups": wl.num_groups}
