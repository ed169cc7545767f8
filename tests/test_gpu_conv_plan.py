"""The ResNet-18 3x3 conv backward step at full size (batch 64, 56 x 56,
64 -> 64 channels, 4-bit gradients, round to nearest even) run the way the
benchmark times it: ConvBackwardPlan with the implicit-im2col input and weight
gradients, on the benchmark's seeded inputs, with the layer input packed from
the centre tap of the im2col'd activations.

Against the oracle: every gradient code (on the padded pixel grid the weight
gradient reads), every group and the scale bit for bit; the shift-folded codes
on sampled rows; every pixel of the input gradient and every row of the
weight gradient, int32 accumulators bit for bit and fp32 outputs bit for bit
(within the 1e-6 relative bar).  A second plan that also keeps the int32
accumulators must give the same fp32 outputs bit for bit."""
import numpy as np
import pytest

import oracle
from paper_2411_10948_amd import workloads
from tests.test_gpu_parity import RTOL, _dev, check_fold

pytestmark = pytest.mark.gpu

N, H, W, C, KH, KW, PH, PW = 64, 56, 56, 64, 3, 3, 1, 1


@pytest.fixture(scope="module")
def sq():
    import torch
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    from paper_2411_10948_amd import shiftquant
    shiftquant.load()
    return shiftquant


def test_resnet18_conv_plan_full_size(sq):
    import torch
    print("[conv plan] resnet18 3x3, 64 x 56 x 56 x 64, as benchmarked", flush=True)
    d = workloads.make_inputs("resnet18_conv3x3")
    wl = d["workload"]
    assert (wl.M, wl.C_out, wl.conv_hw, wl.conv_cin) == (N * H * W, C, H, C)
    params = sq.Params.make(wl.bits, wl.num_groups, wl.round_mode, wl.sr_seed, wl.sr_offset)
    dev = torch.device("cuda:0")
    dY = _dev(d["dY"])
    wq_t, ws = sq.quantize_tensor(_dev(d["W"]), 8, transpose=True)
    Xc = np.ascontiguousarray(d["X"][:, 4 * C:5 * C])   # the layer input: the centre tap (pad 1)
    xq_raw, xs = sq.quantize_tensor(_dev(Xc), 8, transpose=True)
    xq_t = sq.conv_pack_input(xq_raw, N, H, W, KH, KW, PH, PW)

    plan = sq.ConvBackwardPlan(N, H, W, C, C, KH, KW, PH, PW, params, device=dev)
    plan.run(dY, wq_t, ws, xq_t, xs)
    plan_acc = sq.ConvBackwardPlan(N, H, W, C, C, KH, KW, PH, PW, params, device=dev, want_acc=True)
    plan_acc.run(dY, wq_t, ws, xq_t, xs)
    torch.cuda.synchronize()
    assert torch.equal(plan.dX, plan_acc.dX) and torch.equal(plan.dW, plan_acc.dW)

    # gradient codes, groups and scale
    q_ref, g_ref, s_ref, _ = oracle.quantize_grad(d["dY"], wl.bits, wl.num_groups, wl.round_mode,
                                                  wl.sr_seed, wl.sr_offset)
    np.testing.assert_array_equal(plan.group.cpu().numpy(), g_ref)
    gs = sq.scale_to_host(plan.scale)
    assert np.float32(gs["step"]) == np.float32(s_ref["d0"])
    # the padded pixel grid: pixel (n, oh, ow) at n Hp Wp + oh Wp + ow, zeros elsewhere
    rows, ld_x, ld_q = sq.sq_conv_wgrad_layout(N, H, W, C, KH, KW, PH, PW)
    Hp, Wp = H + 2 * PH, (W + 2 * PW + 15) // 16 * 16
    grid = np.zeros((C, ld_q), np.int8)
    pos = (np.arange(N)[:, None, None] * Hp * Wp + np.arange(H)[None, :, None] * Wp
           + np.arange(W)[None, None, :]).reshape(-1)
    grid[:, pos] = q_ref.T
    np.testing.assert_array_equal(plan.q_tp.cpu().numpy(), grid)
    check_fold(plan, q_ref, g_ref, wl.bits, wl.num_groups, np.unique(np.r_[0, N * H * W - 1,
                                                                          np.random.default_rng(3).integers(0, N * H * W, 64)]))

    # input codes: the centre tap's per-tensor scale is the im2col'd tensor's
    wq_ref, ws_ref = oracle.quantize_tensor(d["W"], 8)
    xq_ref, xs_ref = oracle.quantize_tensor(d["X"], 8)
    assert np.float32(sq.scale_to_host(xs)["step"]) == np.float32(xs_ref["d0"])

    oracle.set_threads(16)
    # input gradient: every pixel
    A_ref = oracle.conv_dgrad(q_ref, g_ref, wl.num_groups, wq_ref, N, H, W, KH, KW, PH, PW)
    dX_ref = oracle.dequant_dgrad(A_ref, s_ref["d0"], ws_ref["d0"], wl.num_groups)
    np.testing.assert_array_equal(plan_acc.acc_dX.cpu().numpy(), A_ref)
    np.testing.assert_allclose(plan.dX.cpu().numpy(), dX_ref, rtol=RTOL, atol=0)
    assert np.array_equal(plan.dX.cpu().numpy().view(np.uint32), dX_ref.view(np.uint32))

    # weight gradient: every row, from the convolution's definition on the
    # layer input (the centre-tap columns of the im2col'd codes) ...
    xin = np.ascontiguousarray(xq_ref[:, 4 * C:5 * C])
    B_ref = oracle.conv_wgrad(q_ref, xin, N, H, W, KH, KW, PH, PW)
    dW_ref = oracle.dequant_wgrad(B_ref, g_ref, s_ref["d0"], xs_ref["d0"])
    np.testing.assert_array_equal(plan_acc.acc_dW.cpu().numpy(), B_ref)
    np.testing.assert_allclose(plan.dW.cpu().numpy(), dW_ref, rtol=RTOL, atol=0)
    assert np.array_equal(plan.dW.cpu().numpy().view(np.uint32), dW_ref.view(np.uint32))
    # ... which equals the explicit im2col product on sampled rows (every outlier channel among them)
    outliers = np.nonzero(g_ref < wl.num_groups - 1)[0]
    rows_w = np.unique(np.r_[0, C - 1, outliers[:4], np.random.default_rng(4).integers(0, C, 3)])
    np.testing.assert_array_equal(oracle.wgrad(q_ref, xq_ref, rows_w), B_ref[rows_w])
