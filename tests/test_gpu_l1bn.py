"""Parity of the HIP L1BNQ layer (Sec. 4, App. C) and of the quantizer fed by
producer-side channel ranges with the CPU oracle, through the C-ABI.

Integer state (mean / sigma codes, sign and deviation sums, groups, scale
bits, codes) and the fp32 outputs y, dx, dgamma and dbeta must match bit
for bit (both sides run the same IEEE operations in the same order, with the
binary64 channel constants rounded once).  Inputs are seeded and synthetic:
post-ReLU or signed activations quantized to 8 bits, gradients with
log-normal channel scales.
"""
import numpy as np
import pytest

import oracle

pytestmark = pytest.mark.gpu

RTOL = 1e-6


@pytest.fixture(scope="module")
def sq():
    import torch
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    from paper_2411_10948_amd import shiftquant
    shiftquant.load()
    return shiftquant


def _inputs(M, C, seed, relu=True):
    rng = np.random.default_rng(seed)
    X = rng.normal(0.3, 1.0, (M, C)) * np.exp(rng.normal(0, 0.5, C))
    if relu:
        X = np.maximum(X, 0.0)
    gamma = rng.normal(1.0, 0.3, C)
    beta = rng.normal(0.0, 0.5, C)
    dy = rng.normal(size=(M, C)) * np.exp(rng.normal(0, 1.0, C))
    return X.astype(np.float32), gamma.astype(np.float32), beta.astype(np.float32), dy.astype(np.float32)


def _run(sq, X, gamma, beta, dy, bits=8, ng=4, mode=0, seed=3, offset=7):
    import torch
    M, C = X.shape
    xq_dev, xs = sq.quantize_tensor(torch.from_numpy(X).cuda(), 8, transpose=False)
    xq_dev = xq_dev[:, :C]
    y, st = sq.l1bn_forward(xq_dev, xs, torch.from_numpy(gamma).cuda(), torch.from_numpy(beta).cuda())
    b = sq.l1bn_backward(torch.from_numpy(dy).cuda(), st, bits, ng, mode, seed, offset, want_ranges=True)
    torch.cuda.synchronize()
    return xq_dev, xs, y, st, b


def _check_against_oracle(sq, X, gamma, beta, dy, bits=8, ng=4, mode=0, seed=3, offset=7):
    M, C = X.shape
    xq_dev, xs, y, st, b = _run(sq, X, gamma, beta, dy, bits, ng, mode, seed, offset)
    xq_ref, xs_ref = oracle.quantize_tensor(X, 8)
    np.testing.assert_array_equal(xq_dev.cpu().numpy(), xq_ref)
    f = oracle.l1bn_forward(xq_ref, xs_ref["d0"], gamma, beta)
    ch = sq.l1bn_channels_to_host(st.chan)
    lay = sq.l1bn_layer_to_host(st.layer)
    for k in ("mu", "sigma", "sign_sum", "dev_sum"):
        np.testing.assert_array_equal(ch[k][:C], f[k], err_msg=k)
    for k in ("gamma_q", "beta_q", "kappa"):
        np.testing.assert_array_equal(ch[k][:C].view(np.uint32), f[k].view(np.uint32), err_msg=k)
    assert lay["dev_max"] == f["dev_max"] and lay["rows"] == M
    assert lay["flags"] == (2 if f["dev_max"] == 0 else 0)
    np.testing.assert_array_equal(np.float32(lay["x_step"]), np.float32(xs_ref["d0"]))
    yd = y.cpu().numpy()
    _bits_equal(yd, f["y"], "y")

    r = oracle.l1bn_backward(dy, f, xq_ref, bits, ng, mode, seed, offset)
    np.testing.assert_array_equal(b["group"].cpu().numpy(), r["group"])
    gs = sq.scale_to_host(b["gscale"])
    assert np.float32(gs["step"]) == np.float32(r["gscale"]["d0"])
    assert gs["flags"] == r["gscale"]["flags"]
    dx = b["dx"].cpu().numpy()
    _bits_equal(dx, r["dx"], "dx")
    for k in ("dgamma", "dbeta"):
        _bits_equal(b[k].cpu().numpy(), r[k], k)
    # producer-side ranges: their maximum over slabs is max |dx| of each
    # channel of the oracle's dx, and no slab exceeds it
    rg = b["ranges"].cpu().numpy().view(np.uint32)
    assert rg.shape == (sq.sq_l1bn_range_slabs(M, C), C)
    ref_max = (np.ascontiguousarray(r["dx"]).view(np.uint32) & 0x7FFFFFFF).max(axis=0)
    np.testing.assert_array_equal(rg.max(axis=0), ref_max)
    return dx, b, r


def _bits_equal(got, ref, name):
    """fp32 arrays equal bit for bit (every NaN payload and signed zero)."""
    g = np.ascontiguousarray(got, np.float32).view(np.uint32)
    r = np.ascontiguousarray(ref, np.float32).view(np.uint32)
    bad = np.argwhere(g != r)
    assert bad.size == 0, (f"{name}: {len(bad)} values differ, first at {bad[:3].tolist()}: "
                           f"{got.reshape(g.shape)[tuple(bad[0])]} vs {ref.reshape(r.shape)[tuple(bad[0])]}")


L1BN_CASES = [
    (37, 5, True), (1000, 64, True), (4099, 48, False), (300, 200, True), (1, 16, True),
    (777, 17, False), (2500, 4100, True),
]


@pytest.mark.parametrize("M,C,relu", L1BN_CASES)
def test_l1bn_parity(sq, M, C, relu):
    print(f"l1bn M={M} C={C} relu={relu}", flush=True)
    X, gamma, beta, dy = _inputs(M, C, seed=M * 31 + C, relu=relu)
    _check_against_oracle(sq, X, gamma, beta, dy)


@pytest.mark.parametrize("bits,ng,mode", [(6, 4, 0), (8, 4, 1), (4, 2, 1), (8, 1, 0)])
def test_l1bn_gradient_quantizer_variants(sq, bits, ng, mode):
    print(f"l1bn variants b={bits} ng={ng} mode={mode}", flush=True)
    X, gamma, beta, dy = _inputs(3001, 96, seed=bits * 10 + ng + mode)
    _check_against_oracle(sq, X, gamma, beta, dy, bits, ng, mode, seed=11, offset=2)


def test_l1bn_constant_channels(sq):
    print("l1bn constant", flush=True)
    M, C = 129, 32
    X = np.tile(np.linspace(-1, 1, C, dtype=np.float32), (M, 1))
    rng = np.random.default_rng(5)
    gamma = rng.normal(1, 0.3, C).astype(np.float32)
    beta = rng.normal(0, 0.5, C).astype(np.float32)
    dy = rng.normal(size=(M, C)).astype(np.float32)
    dx, b, _ = _check_against_oracle(sq, X, gamma, beta, dy)
    assert np.all(dx == 0)


def test_l1bn_resnet18_layer_full_size(sq):
    # the batch norm after a 3x3 conv of ResNet-18's first stage: N=64, 56x56, 64 channels
    print("l1bn resnet18 full size", flush=True)
    X, gamma, beta, dy = _inputs(64 * 56 * 56, 64, seed=18)
    _check_against_oracle(sq, X, gamma, beta, dy)


@pytest.mark.parametrize("bits,ng,mode", [(4, 4, 0), (6, 4, 1)])
def test_quantize_from_producer_ranges_equals_quantize(sq, bits, ng, mode):
    # the layer's dx with the ranges it wrote, quantized for the conv below:
    # codes, groups and scale equal the oracle's quantizer on the oracle's dx,
    # and everything equals the quantizer's own abs-max pass
    import torch
    from tests.test_gpu_parity import check_quant
    print(f"from ranges b={bits} mode={mode}", flush=True)
    X, gamma, beta, dy = _inputs(5003, 64, seed=bits + mode)
    dx_h, b, r = _check_against_oracle(sq, X, gamma, beta, dy)
    dx, ranges = b["dx"], b["ranges"]
    a = sq.quantize_grad(dx, bits, ng, mode, seed=4, offset=9)
    c = sq.quantize_grad_from_ranges(dx, ranges, bits, ng, mode, seed=4, offset=9)
    torch.cuda.synchronize()
    check_quant(sq, c, r["dx"], bits, ng, mode, 4, 9)
    for name in ("q_fold", "q_t", "group", "layout"):
        assert torch.equal(getattr(a, name), getattr(c, name)), name
    assert torch.equal(a.scale, c.scale)


def test_quantize_from_ranges_arbitrary_slabs(sq):
    # ranges cut at arbitrary row subsets (one slab per 100 rows, plus an
    # all-zero slab) give the same codes as the quantizer's own pass
    import torch
    print("from ranges arbitrary slabs", flush=True)
    rng = np.random.default_rng(8)
    M, C = 1234, 300
    dY = (rng.normal(size=(M, C)) * np.exp(rng.normal(0, 1.5, C))).astype(np.float32)
    bits = np.abs(dY).view(np.uint32)
    cuts = list(range(0, M, 100)) + [M]
    slabs = [bits[a:b].max(axis=0) for a, b in zip(cuts[:-1], cuts[1:])] + [np.zeros(C, np.uint32)]
    ranges = torch.from_numpy(np.stack(slabs).view(np.int32)).cuda()
    d = torch.from_numpy(dY).cuda()
    a = sq.quantize_grad(d, 6, 4)
    c = sq.quantize_grad_from_ranges(d, ranges, 6, 4)
    torch.cuda.synchronize()
    from tests.test_gpu_parity import check_quant
    check_quant(sq, c, dY, 6, 4, 0, 0, 0)   # against the oracle's quantizer of dY
    for name in ("q_fold", "q_t", "group", "layout"):
        assert torch.equal(getattr(a, name), getattr(c, name)), name
    assert torch.equal(a.scale, c.scale)
