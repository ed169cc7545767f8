"""The conv input quantizer (sq_quantize_input_conv) through the C-ABI: the
per-tensor 8-bit codes of the oracle, placed on the padded input grid of the
implicit-im2col weight gradient (every byte of the buffer compared, padding
zero), and the same buffer as packing sq_quantize_tensor's codes with
sq_conv_pack_input.  Inputs are seeded and synthetic (post-ReLU activations,
as the layer input of a conv after a ReLU)."""
import numpy as np
import pytest

import oracle
from tests.test_gpu_parity import _dev, _f32bits

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sq():
    import torch
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    from paper_2411_10948_amd import shiftquant
    shiftquant.load()
    return shiftquant


CASES = [  # N, H, W, C_in, KH, KW, PH, PW
    (1, 4, 56, 64, 3, 3, 1, 1),     # ResNet-18 width, one tile row spans image rows (offset 1 mod 8)
    (2, 5, 56, 8, 3, 3, 1, 1),      # 8 channels, several images
    (1, 3, 8, 16, 3, 3, 1, 1),      # one 8-pixel group per image row
    (3, 2, 16, 24, 5, 5, 2, 3),     # offset 3 mod 8
    (1, 7, 24, 72, 3, 3, 0, 2),     # unpadded rows, channels past one 64-channel tile
    (2, 3, 40, 8, 3, 7, 1, 5),      # offset 5 mod 8
    (1, 2, 136, 16, 3, 3, 1, 1),    # rows longer than a 128-pixel tile
    (2, 9, 32, 16, 3, 9, 1, 7),     # offset 7 mod 8
    (2, 6, 16, 32, 1, 1, 0, 0),     # 1 x 1 window: aligned offset 0
    (1, 4, 16, 16, 9, 9, 4, 8),     # offset a multiple of 8 (aligned 8-byte stores)
    (2, 5, 7, 3, 3, 3, 1, 1),       # width and channels not multiples of 8 (byte stores)
    (1, 6, 14, 12, 3, 3, 1, 1),     # channels not a multiple of 8
    (1, 5, 12, 8, 3, 3, 1, 1),      # width not a multiple of 8
]


def _grid(xq, N, H, W, C_in, KH, PH, PW, ld):
    Hp, Wp = H + 2 * PH, (W + 2 * PW + 15) // 16 * 16
    g = np.zeros((C_in, ld), np.int8)
    for n in range(N):
        for h in range(H):
            row = xq[(n * H + h) * W:(n * H + h + 1) * W].T
            base = n * Hp * Wp + (h + PH) * Wp + PW
            g[:, base:base + W] = row
    return g


def _input(N, H, W, C_in, seed):
    rng = np.random.default_rng(seed)
    return np.maximum(rng.standard_normal((N * H * W, C_in)), 0.0).astype(np.float32)


@pytest.mark.parametrize("case", CASES, ids=["x".join(map(str, c)) for c in CASES])
def test_quantize_input_conv_parity(sq, case):
    import torch
    N, H, W, C_in, KH, KW, PH, PW = case
    print(f"conv input quantizer {case}", flush=True)
    X = _input(N, H, W, C_in, sum(case))
    xs, xq, s = sq.quantize_input_conv(_dev(X), N, H, W, KH, KW, PH, PW, 8, want_rows=True)
    torch.cuda.synchronize()
    q_ref, s_ref = oracle.quantize_tensor(X, 8)
    rows, ld, _ = sq.sq_conv_wgrad_layout(N, H, W, C_in, KH, KW, PH, PW)
    assert xs.shape == (rows, ld)
    np.testing.assert_array_equal(xs.cpu().numpy(), _grid(q_ref, N, H, W, C_in, KH, PH, PW, ld))
    np.testing.assert_array_equal(xq.cpu().numpy(), q_ref)
    h = sq.scale_to_host(s)
    assert h["bits"][:3] == [_f32bits(s_ref["r_max"]), _f32bits(s_ref["inv0"]), _f32bits(s_ref["d0"])]
    # the same buffer as packing the codes of the per-tensor quantizer
    xq_t, _ = sq.quantize_tensor(_dev(X), 8, transpose=True)
    assert torch.equal(xs, sq.conv_pack_input(xq_t, N, H, W, KH, KW, PH, PW))


@pytest.mark.parametrize("ld_pad,misalign", [(8, 0), (3, 1)])
def test_quantize_input_conv_strided_input(sq, ld_pad, misalign):
    # X with a padded leading dimension (16-byte rows: the 8-channel kernel),
    # and with an odd one at a 4-byte offset (the generic kernel's byte stores)
    import torch
    N, H, W, C_in, KH, KW, PH, PW = 2, 5, 24, 16, 3, 3, 1, 1
    print(f"conv input quantizer, ld pad {ld_pad}, offset {misalign}", flush=True)
    X = _input(N, H, W, C_in, 40 + ld_pad)
    xs, xq, s = sq.quantize_input_conv(_dev(X, ld_pad, misalign), N, H, W, KH, KW, PH, PW, 8, want_rows=True)
    torch.cuda.synchronize()
    q_ref, _ = oracle.quantize_tensor(X, 8)
    _, ld, _ = sq.sq_conv_wgrad_layout(N, H, W, C_in, KH, KW, PH, PW)
    np.testing.assert_array_equal(xs.cpu().numpy(), _grid(q_ref, N, H, W, C_in, KH, PH, PW, ld))
    np.testing.assert_array_equal(xq.cpu().numpy(), q_ref)


def test_quantize_input_conv_zero_tensor(sq):
    # an all-zero input: zero codes, the scale's zero flag, the grid untouched
    import torch
    N, H, W, C_in = 1, 3, 16, 8
    X = np.zeros((N * H * W, C_in), np.float32)
    xs, xq, s = sq.quantize_input_conv(_dev(X), N, H, W, 3, 3, 1, 1, 8, want_rows=True)
    torch.cuda.synchronize()
    assert not xs.any().item() and not xq.any().item()
    _, s_ref = oracle.quantize_tensor(X, 8)
    assert sq.scale_to_host(s)["bits"][:3] == [_f32bits(s_ref["r_max"]), _f32bits(s_ref["inv0"]),
                                                 _f32bits(s_ref["d0"])]


def test_quantize_input_conv_full_resnet18_layer(sq):
    # the input of the benchmark's conv layer (64 x 56 x 56 x 64) straight onto
    # the grid equals packing the per-tensor codes, and the weight gradient
    # taken from it equals the one of the packed step, bit for bit
    import torch
    from paper_2411_10948_amd import workloads
    print("conv input quantizer, full resnet18 layer", flush=True)
    wl = workloads.WORKLOADS["resnet18_conv3x3"]
    d = workloads.make_inputs(wl.name)
    H = W = wl.conv_hw
    N, C_in = d["M"] // (H * W), wl.conv_cin
    X = d["X"][:, 4 * C_in:5 * C_in].copy()   # centre tap of the im2col'd rows = the layer input
    xs, _, s = sq.quantize_input_conv(_dev(X), N, H, W, 3, 3, 1, 1, 8)
    xq_t, s2 = sq.quantize_tensor(_dev(X), 8, transpose=True)
    packed = sq.conv_pack_input(xq_t, N, H, W, 3, 3, 1, 1)
    torch.cuda.synchronize()
    assert torch.equal(xs, packed) and torch.equal(s, s2)
    q_ref, _ = oracle.quantize_tensor(X, 8)
    rng = np.random.default_rng(3)
    for n in np.unique(np.r_[0, N - 1, rng.integers(0, N, 4)]):
        sl = slice(n * H * W, (n + 1) * H * W)
        Hp, Wp = H + 2, 64
        img = xs[:, n * Hp * Wp:(n + 1) * Hp * Wp].cpu().numpy().reshape(C_in, Hp, Wp)
        np.testing.assert_array_equal(img[:, 1:H + 1, 1:W + 1], q_ref[sl].T.reshape(C_in, H, W))
        assert not img[:, 0].any() and not img[:, H + 1].any() and not img[:, :, 0].any() and not img[:, :, W + 1:].any()


def test_conv_plan_quantize_input_equals_packed_step(sq):
    # the plan's step with the input quantized onto its grid equals the step
    # that packs sq_quantize_tensor's codes (dX and dW bit for bit)
    import torch
    N, H, W, C_out, C_in = 2, 9, 16, 64, 64
    params = sq.Params.make(4, 4, 0, 7, 0)
    rng = np.random.default_rng(11)
    dY = (rng.standard_t(3, (N * H * W, C_out)) * 1e-3).astype(np.float32)
    X = _input(N, H, W, C_in, 12)
    Wt = (rng.standard_normal((C_out, 9 * C_in)) * 0.05).astype(np.float32)
    wq_t, ws = sq.quantize_tensor(_dev(Wt), 8, transpose=True)
    xq_t, xsc = sq.quantize_tensor(_dev(X), 8, transpose=True)
    a = sq.ConvBackwardPlan(N, H, W, C_out, C_in, 3, 3, 1, 1, params)
    b = sq.ConvBackwardPlan(N, H, W, C_out, C_in, 3, 3, 1, 1, params)
    a.run_packed(_dev(dY), wq_t, ws, xq_t, xsc)
    b.quantize_input(_dev(X))
    b.run(_dev(dY), wq_t, ws, b.x_grid, b.x_scale)
    torch.cuda.synchronize()
    assert torch.equal(a.x_grid, b.x_grid) and torch.equal(xsc, b.x_scale)
    assert torch.equal(a.dX, b.dX) and torch.equal(a.dW, b.dW)
