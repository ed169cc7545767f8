"""Producer-side channel ranges from the convolution input gradient
(sq_conv_dgrad_ranged) and the conv quantizer fed by them
(sq_quantize_grad_conv_from_ranges), anchored on the oracle: dX equals the
oracle's conv input gradient bit for bit, every slab maximum equals the
maximum of the oracle's |dX| over the slab's rows (bit patterns), and the next
layer's codes (on the padded pixel grid), groups and scale equal the oracle's
quantizer on the oracle's dX.  Both paths are covered: the streaming kernel
(per-block slabs) and the other conv kernels (32-row slab pass).  Inputs are
seeded and synthetic."""
import numpy as np
import pytest

import oracle
from paper_2411_10948_amd import workloads
from tests.test_gpu_parity import _dev, _grad

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sq():
    import torch
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    from paper_2411_10948_amd import shiftquant
    shiftquant.load()
    oracle.set_threads(16)
    return shiftquant


def _expected_grid(q, N, Ho, Wo, C, ld, KH, KW, PH, PW, H, W):
    Hp, Wp = H + 2 * PH, (W + 2 * PW + 15) // 16 * 16
    grid = np.zeros((C, ld), np.int8)
    pos = (np.arange(N)[:, None, None] * Hp * Wp + np.arange(Ho)[None, :, None] * Wp
           + np.arange(Wo)[None, None, :]).reshape(-1)
    grid[:, pos] = q.T
    return grid


CASES = [  # N, H, W, C_out, C_in, KH, KW, PH, PW, bits, N_G, rounding (the next layer: 3x3, pad 1)
    (4, 56, 56, 64, 64, 3, 3, 1, 1, 4, 4, 0),    # streaming kernel, the ResNet-18 layer on 4 images
    (3, 17, 23, 48, 32, 3, 3, 1, 1, 6, 4, 1),     # streaming kernel, ragged block, C_out < 64
    (2, 14, 14, 96, 80, 3, 3, 1, 1, 6, 4, 0),     # C_in > 64: the other conv kernels, 32-row slabs
    (2, 20, 20, 64, 48, 5, 5, 2, 2, 4, 4, 0),     # a 5x5 window
]


@pytest.mark.parametrize("case", CASES, ids=["x".join(map(str, c)) for c in CASES])
def test_conv_dgrad_ranges_feed_the_next_quantizer(sq, case):
    import torch
    N, H, W, C_out, C_in, KH, KW, PH, PW, bits, ng, mode = case
    print(f"[conv ranges] {case}", flush=True)
    Ho, Wo = H + 2 * PH - KH + 1, W + 2 * PW - KW + 1
    M, P = N * Ho * Wo, N * H * W
    dY = _grad(M, C_out, seed=M + C_in)
    rng = np.random.default_rng(P + C_out)
    Wt = (rng.standard_normal((C_out, KH * KW * C_in)) * 0.05).astype(np.float32)
    p = sq.Params.make(bits, ng, mode, 7, 3)
    plan = sq.ConvBackwardPlan(N, H, W, C_out, C_in, KH, KW, PH, PW, p, dx_ranges=True)
    wq_t, ws = sq.quantize_tensor(_dev(Wt), 8, transpose=True)
    plan.quantize(_dev(dY))
    plan.dgrad(wq_t, ws)
    slabs, R = plan.range_slabs, plan.range_rows
    assert slabs == (P + R - 1) // R
    # the next layer (3x3, pad 1, C_out' = C_in) quantizes dX with those ranges
    nxt = sq.ConvBackwardPlan(N, H, W, C_in, 8, 3, 3, 1, 1, p)
    nxt.quantize_from_ranges(plan.dX, plan.dX_ranges, range_slabs=slabs)
    torch.cuda.synchronize()

    q_ref, g_ref, s_ref, _ = oracle.quantize_grad(dY, bits, ng, mode, 7, 3)
    wq_ref, ws_ref = oracle.quantize_tensor(Wt, 8)
    A_ref = oracle.conv_dgrad(q_ref, g_ref, ng, wq_ref, N, H, W, KH, KW, PH, PW)
    dX_ref = oracle.dequant_dgrad(A_ref, s_ref["d0"], ws_ref["d0"], ng)
    np.testing.assert_array_equal(plan.dX.cpu().numpy().view(np.uint32), dX_ref.view(np.uint32))
    # slab s covers rows [s R, (s + 1) R)
    assert 1 <= slabs <= sq.sq_gemm_dgrad_range_slabs(P)
    if (C_in > 64 or KH != 3) and slabs:
        assert R == 32   # the other conv kernels: 32-row slabs
    xb = dX_ref.view(np.uint32) & 0x7FFFFFFF
    pad = slabs * R - P
    ref = np.concatenate([xb, np.zeros((pad, C_in), np.uint32)]).reshape(slabs, R, C_in).max(axis=1)
    np.testing.assert_array_equal(plan.dX_ranges[:slabs].cpu().numpy().view(np.uint32), ref)
    # the next layer's quantizer
    q2, g2, s2, _ = oracle.quantize_grad(dX_ref, bits, ng, mode, 7, 3)
    np.testing.assert_array_equal(nxt.group.cpu().numpy(), g2)
    h = sq.scale_to_host(nxt.scale)
    assert np.float32(h["step"]) == np.float32(s2["d0"]) and h["flags"] == s2["flags"]
    rows_, x_ld, q_ld = sq.sq_conv_wgrad_layout(N, H, W, 8, 3, 3, 1, 1)
    np.testing.assert_array_equal(nxt.q_tp.cpu().numpy(),
                                  _expected_grid(q2, N, H, W, C_in, nxt.q_tp.shape[1], 3, 3, 1, 1, H, W))


def test_conv_dgrad_ranges_resnet18_full_size(sq):
    # the benchmarked ResNet-18 layer (64 x 56 x 56 x 64) in a two-layer chain
    import torch
    print("[conv ranges] resnet18 full size", flush=True)
    d = workloads.make_inputs("resnet18_conv3x3")
    wl = d["workload"]
    N, H, W, C = 64, 56, 56, 64
    p = sq.Params.make(wl.bits, wl.num_groups, wl.round_mode)
    plan = sq.ConvBackwardPlan(N, H, W, C, C, 3, 3, 1, 1, p, dx_ranges=True)
    wq_t, ws = sq.quantize_tensor(_dev(d["W"]), 8, transpose=True)
    plan.quantize(_dev(d["dY"]))
    plan.dgrad(wq_t, ws)
    nxt = sq.ConvBackwardPlan(N, H, W, C, C, 3, 3, 1, 1, p)
    nxt.quantize_from_ranges(plan.dX, plan.dX_ranges, range_slabs=plan.range_slabs)
    own = sq.ConvBackwardPlan(N, H, W, C, C, 3, 3, 1, 1, p)
    own.quantize(plan.dX)
    torch.cuda.synchronize()
    slabs = plan.range_slabs
    assert slabs <= 512
    q_ref, g_ref, s_ref, _ = oracle.quantize_grad(d["dY"], wl.bits, wl.num_groups, wl.round_mode)
    wq_ref, ws_ref = oracle.quantize_tensor(d["W"], 8)
    dX_ref = oracle.dequant_dgrad(oracle.conv_dgrad(q_ref, g_ref, wl.num_groups, wq_ref, N, H, W, 3, 3, 1, 1),
                                  s_ref["d0"], ws_ref["d0"], wl.num_groups)
    np.testing.assert_array_equal(plan.dX.cpu().numpy().view(np.uint32), dX_ref.view(np.uint32))
    rg = plan.dX_ranges[:slabs].cpu().numpy().view(np.uint32)
    np.testing.assert_array_equal(rg.max(axis=0), (dX_ref.view(np.uint32) & 0x7FFFFFFF).max(axis=0))
    q2, g2, s2, _ = oracle.quantize_grad(dX_ref, wl.bits, wl.num_groups, wl.round_mode)
    np.testing.assert_array_equal(nxt.group.cpu().numpy(), g2)
    np.testing.assert_array_equal(nxt.q_tp.cpu().numpy(),
                                  _expected_grid(q2, N, H, W, C, nxt.q_tp.shape[1], 3, 3, 1, 1, H, W))
    # identical to the quantizer's own abs-max pass
    for name in ("q_fold", "q_tp", "group", "layout", "scale"):
        assert torch.equal(getattr(nxt, name), getattr(own, name)), name
