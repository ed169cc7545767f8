"""Parity of the implicit-im2col conv weight gradient (sq_conv_wgrad) with the
CPU oracle, through the C-ABI: int32 accumulators bit for bit, fp32 dW within
1e-6 relative.  Inputs are seeded and synthetic (heavy-tailed gradients,
post-ReLU activations quantized to 8 bits)."""
import numpy as np
import pytest

import oracle
from tests.test_gpu_parity import RTOL, _dev, _grad

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sq():
    import torch
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    from paper_2411_10948_amd import shiftquant
    shiftquant.load()
    return shiftquant


WGRAD_CASES = [  # N, H, W, C_out, C_in, KH, KW, PH, PW, bits, N_G
    (2, 9, 7, 64, 64, 3, 3, 1, 1, 4, 4),      # same-size 3x3, width not a multiple of 16
    (1, 13, 11, 48, 40, 3, 3, 1, 1, 6, 4),    # channels not multiples of 16
    (1, 10, 12, 96, 160, 3, 3, 0, 1, 4, 4),   # unpadded rows, padded columns, C_out > 64
    (2, 6, 5, 32, 24, 1, 1, 0, 0, 8, 3),      # 1 x 1 window
    (1, 8, 8, 64, 64, 5, 5, 2, 2, 4, 4),      # 5 x 5 window
    (1, 7, 9, 130, 64, 2, 3, 1, 0, 6, 4),     # even window height, one-sided padding
    (3, 4, 4, 200, 72, 3, 3, 1, 1, 8, 4),     # 8-bit codes
    (1, 5, 16, 64, 64, 3, 3, 1, 1, 4, 4),     # padded width exactly 32
    (4, 14, 14, 256, 128, 3, 3, 1, 1, 4, 4),  # a ResNet stage-3 shape, large tiles
    # 64 input channels, 3-wide windows, split K: the window kernel that
    # reads one input copy and shifts in registers
    (4, 14, 14, 64, 64, 3, 3, 1, 1, 4, 4),    # 2 K splits
    (3, 20, 23, 40, 64, 3, 3, 1, 1, 6, 4),    # fewer than 64 output channels, 4 splits
    (4, 12, 12, 64, 64, 5, 3, 2, 1, 4, 4),    # 5 tap rows per split (2 splits)
    (2, 30, 30, 64, 64, 3, 3, 0, 0, 8, 4),    # unpadded rows and columns, 8-bit codes
]


def _layer(N, H, W, C_out, C_in, KH, KW, PH, PW, seed):
    Ho, Wo = H + 2 * PH - KH + 1, W + 2 * PW - KW + 1
    rng = np.random.default_rng(seed)
    dY = _grad(N * Ho * Wo, C_out, seed=seed)
    X = np.maximum(rng.standard_normal((N * H * W, C_in)), 0.0).astype(np.float32)
    return dY, X


def _run(sq, dY, X, case, mode=0):
    import torch
    N, H, W, C_out, C_in, KH, KW, PH, PW, bits, ng = case
    codes = sq.quantize_grad(_dev(dY), bits, ng, mode, 7, 0)
    xq_t, xs_scale = sq.quantize_tensor(_dev(X), 8, transpose=True)
    xs = sq.conv_pack_input(xq_t, N, H, W, KH, KW, PH, PW)
    dW, acc = sq.conv_wgrad(codes, xs, xs_scale, N, H, W, C_in, KH, KW, PH, PW, want_acc=True)
    # the quantizer writing the padded codes directly (padding zero-filled once)
    _, _, qld = sq.sq_conv_wgrad_layout(N, H, W, C_in, KH, KW, PH, PW)
    q_tp = torch.zeros((C_out, qld), dtype=torch.int8, device="cuda")
    q_fold = torch.zeros_like(codes.q_fold)
    group = torch.empty_like(codes.group)
    scale = sq.new_scale("cuda")
    layout = torch.zeros_like(codes.layout)
    ws = torch.empty(max(sq.sq_quantize_grad_workspace_size(dY.shape[0], C_out, codes.params), 256),
                     dtype=torch.uint8, device="cuda")
    sq.sq_quantize_grad_conv(_dev(dY), N, H, W, KH, KW, PH, PW, codes.params, q_fold, q_tp, group, scale, layout, ws)
    dW2, _ = sq.conv_wgrad(codes, xs, xs_scale, N, H, W, C_in, KH, KW, PH, PW, want_acc=False, q_tp=q_tp)
    torch.cuda.synchronize()
    assert torch.equal(q_fold, codes.q_fold) and torch.equal(group, codes.group) and torch.equal(scale, codes.scale)
    assert torch.equal(q_tp, sq.conv_pack_grad(codes, N, H, W, KH, KW, PH, PW))
    assert torch.equal(dW, dW2)
    return codes, acc.cpu().numpy(), dW.cpu().numpy()


@pytest.mark.parametrize("case", WGRAD_CASES, ids=["x".join(map(str, c)) for c in WGRAD_CASES])
def test_conv_wgrad_parity(sq, case):
    N, H, W, C_out, C_in, KH, KW, PH, PW, bits, ng = case
    print(f"conv wgrad {case}", flush=True)
    dY, X = _layer(N, H, W, C_out, C_in, KH, KW, PH, PW, seed=sum(case))
    codes, acc, dW = _run(sq, dY, X, case)
    q_ref, g_ref, s_ref, _ = oracle.quantize_grad(dY, bits, ng, 0, 7, 0)
    xq_ref, xs_ref = oracle.quantize_tensor(X, 8)
    np.testing.assert_array_equal(codes.group.cpu().numpy(), g_ref)
    B_ref = oracle.conv_wgrad(q_ref, xq_ref, N, H, W, KH, KW, PH, PW)
    bad = np.argwhere(acc != B_ref)
    assert bad.size == 0, f"{len(bad)} conv wgrad accumulators differ, first at {bad[:4].tolist()}"
    dW_ref = oracle.dequant_wgrad(B_ref, g_ref, s_ref["d0"], xs_ref["d0"])
    np.testing.assert_allclose(dW, dW_ref, rtol=RTOL, atol=0)


def test_conv_wgrad_stochastic_codes(sq):
    case = (1, 9, 9, 72, 64, 3, 3, 1, 1, 6, 4)
    print("conv wgrad SR", flush=True)
    N, H, W, C_out, C_in, KH, KW, PH, PW, bits, ng = case
    dY, X = _layer(N, H, W, C_out, C_in, KH, KW, PH, PW, seed=5)
    _, acc, _ = _run(sq, dY, X, case, mode=1)
    q_ref, _, _, _ = oracle.quantize_grad(dY, bits, ng, 1, 7, 0)
    xq_ref, _ = oracle.quantize_tensor(X, 8)
    np.testing.assert_array_equal(acc, oracle.conv_wgrad(q_ref, xq_ref, N, H, W, KH, KW, PH, PW))


def test_conv_wgrad_full_resnet18_layer(sq):
    # the full 64 x 56 x 56 x 64 layer of the benchmark; the reference is the
    # wgrad of the explicit im2col (equal to the conv wgrad by the oracle's
    # pins) as a float64 product, exact here: every partial sum of
    # products of 4-bit and 8-bit codes stays below 2^53
    case = (64, 56, 56, 64, 64, 3, 3, 1, 1, 4, 4)
    print("conv wgrad full resnet18 layer", flush=True)
    N, H, W, C_out, C_in, KH, KW, PH, PW, bits, ng = case
    dY, X = _layer(N, H, W, C_out, C_in, KH, KW, PH, PW, seed=18)
    codes, acc, dW = _run(sq, dY, X, case)
    q_ref, g_ref, s_ref, _ = oracle.quantize_grad(dY, bits, ng, 0, 7, 0)
    xq_ref, xs_ref = oracle.quantize_tensor(X, 8)
    x4 = np.zeros((N, H + 2, W + 2, C_in), np.float64)
    x4[:, 1:H + 1, 1:W + 1, :] = xq_ref.reshape(N, H, W, C_in)
    cols = np.concatenate([x4[:, r:r + H, s:s + W, :] for r in range(3) for s in range(3)], axis=3)
    B_ref = (q_ref.astype(np.float64).T @ cols.reshape(N * H * W, 9 * C_in))
    assert np.abs(B_ref).max() < 2.0 ** 31
    np.testing.assert_array_equal(acc, B_ref.astype(np.int64))
    dW_ref = oracle.dequant_wgrad(B_ref.astype(np.int32), g_ref, s_ref["d0"], xs_ref["d0"])
    np.testing.assert_allclose(dW, dW_ref, rtol=RTOL, atol=0)


PACK_CASES = [  # N, H, W, C_in, KH, KW, PH, PW, ld_xq extra
    (2, 5, 7, 3, 3, 3, 1, 1, 0),      # odd left padding, rows of 7 pixels
    (3, 6, 16, 5, 3, 3, 1, 1, 16),    # a content row ends at a chunk edge
    (1, 9, 30, 2, 5, 5, 2, 2, 32),    # 2-pixel padding, 3 chunks per grid row
    (2, 4, 13, 4, 1, 1, 0, 0, 0),     # no padding, Wp = 16 > W
    (1, 3, 33, 1, 3, 7, 0, 6, 48),    # padding wider than a word, Wp = 48
]


@pytest.mark.parametrize("case", PACK_CASES)
def test_conv_pack_input_layout(sq, case):
    # the packed input is the padded grid of each channel, zeros elsewhere
    # (every byte of the row, through its leading dimension)
    import torch
    N, H, W, C_in, KH, KW, PH, PW, extra = case
    rng = np.random.default_rng(sum(case))
    xq = rng.integers(-127, 128, (N * H * W, C_in)).astype(np.int8)
    ld_xq = (N * H * W + 15) // 16 * 16 + extra
    # bytes past N H W in each row are garbage the pack must not copy
    xq_t = torch.from_numpy(rng.integers(-127, 128, (C_in, ld_xq)).astype(np.int8)).cuda()
    xq_t[:, :N * H * W] = torch.from_numpy(xq.T.copy()).cuda()
    xs = sq.conv_pack_input(xq_t, N, H, W, KH, KW, PH, PW)
    torch.cuda.synchronize()
    rows, ld, qld = sq.sq_conv_wgrad_layout(N, H, W, C_in, KH, KW, PH, PW)
    Hp, Wp = H + 2 * PH, (W + 2 * PW + 15) // 16 * 16
    assert rows == C_in and ld % 16 == 0 and ld == qld + (KH - 1) * Wp + 64
    grid = np.zeros((C_in, ld), np.int8)
    for n in range(N):
        for h in range(H):
            for w in range(W):
                grid[:, n * Hp * Wp + (h + PH) * Wp + (w + PW)] = xq[(n * H + h) * W + w]
    np.testing.assert_array_equal(xs.cpu().numpy(), grid)


def test_conv_wgrad_rejects_bad_geometry(sq):
    import torch
    case = (1, 5, 5, 16, 8, 3, 3, 1, 1, 4, 4)
    dY, X = _layer(*case[:9], seed=1)
    codes = sq.quantize_grad(_dev(dY), 4, 4)
    xq_t, xs_scale = sq.quantize_tensor(_dev(X), 8, transpose=True)
    xs = sq.conv_pack_input(xq_t, 1, 5, 5, 3, 3, 1, 1)
    with pytest.raises(sq.ShiftQuantError):
        sq.conv_wgrad(codes, xs, xs_scale, 1, 5, 5, 8, 3, 3, 3, 1)       # padding >= window
    with pytest.raises(sq.ShiftQuantError):
        sq.conv_pack_input(xq_t, 1, 1, 5, 3, 3, 0, 1)                   # window taller than the input
    torch.cuda.synchronize()
