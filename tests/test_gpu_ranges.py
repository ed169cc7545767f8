"""Producer-side channel ranges from the loss-propagation GEMM (sq_gemm_dgrad_ranged),
anchored on the oracle: dX equals the oracle's dX bit for bit (and
sq_gemm_dgrad's), every 32-row slab maximum equals the maximum of the oracle's
|dX| over those rows (bit patterns), and quantizing dX with those ranges gives
the oracle quantizer's codes, groups and scale on the oracle's dX (and exactly
the quantizer's own abs-max pass).  Inputs are seeded and synthetic."""
import numpy as np
import pytest

import oracle
from tests.test_gpu_parity import _dev, _grad, check_quant

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sq():
    import torch
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    from paper_2411_10948_amd import shiftquant
    shiftquant.load()
    return shiftquant


RANGE_CASES = [  # M, C_out, C_in, bits, N_G  (tile: large / small / skinny, fold windows)
    (1000, 256, 1024, 4, 4),
    (777, 300, 200, 6, 4),      # appended fold windows, ragged M and C
    (40, 128, 96, 4, 4),        # a single row tile of the skinny kind
    (4099, 768, 3072, 6, 4),    # the MLP chain's down-projection, large tiles
    (65, 64, 48, 8, 3),
    (8000, 1024, 1536, 6, 4),   # 128 x 384 tiles (192 large tiles would leave CUs idle), fold windows
    (8000 - 40, 1024, 1536, 4, 4),   # the same tiles, one window, ragged rows
]


@pytest.mark.parametrize("case", RANGE_CASES, ids=["x".join(map(str, c)) for c in RANGE_CASES])
def test_dgrad_ranges(sq, case):
    import torch
    M, C_out, C_in, bits, ng = case
    print(f"dgrad ranges {case}", flush=True)
    rng = np.random.default_rng(M + C_in)
    dY = _grad(M, C_out, seed=M)
    Wt = (rng.standard_normal((C_out, C_in)) * 0.02).astype(np.float32)
    codes = sq.quantize_grad(_dev(dY), bits, ng)
    wq_t, ws = sq.quantize_tensor(_dev(Wt), 8, transpose=True)
    _, dX0 = sq.gemm_dgrad(codes, wq_t, ws)
    slabs = sq.sq_gemm_dgrad_range_slabs(M)
    assert slabs == (M + 31) // 32
    dX = torch.empty((M, C_in), dtype=torch.float32, device="cuda")
    ranges = torch.full((slabs, C_in), -1, dtype=torch.int32, device="cuda")
    wsz = sq.sq_gemm_dgrad_workspace_size(M, C_out, C_in, codes.params)
    ws_d = torch.empty(max(wsz, 256), dtype=torch.uint8, device="cuda")
    sq.sq_gemm_dgrad_ranged(codes.q_fold, codes.layout, codes.group, codes.scale, wq_t, ws, M, C_out, C_in,
                            codes.params, None, dX, ranges, ws_d)
    torch.cuda.synchronize()
    assert torch.equal(dX, dX0)
    # the oracle's dX of the same layer
    oracle.set_threads(16)
    q_ref, g_ref, s_ref, _ = oracle.quantize_grad(dY, bits, ng)
    wq_ref, ws_ref = oracle.quantize_tensor(Wt, 8)
    dX_ref = oracle.dequant_dgrad(oracle.dgrad(q_ref, g_ref, ng, wq_ref), s_ref["d0"], ws_ref["d0"], ng)
    np.testing.assert_array_equal(dX.cpu().numpy().view(np.uint32), dX_ref.view(np.uint32))
    xb = dX_ref.view(np.uint32) & 0x7FFFFFFF
    pad = slabs * 32 - M
    ref = np.concatenate([xb, np.zeros((pad, C_in), np.uint32)]).reshape(slabs, 32, C_in).max(axis=1)
    np.testing.assert_array_equal(ranges.cpu().numpy().view(np.uint32), ref)
    # the next layer's quantizer fed these ranges
    a = sq.quantize_grad(dX, bits, ng)
    b = sq.quantize_grad_from_ranges(dX, ranges, bits, ng)
    torch.cuda.synchronize()
    check_quant(sq, b, dX_ref, bits, ng, 0, 0, 0)
    for name in ("q_fold", "q_t", "group", "layout"):
        assert torch.equal(getattr(a, name), getattr(b, name)), name
    assert torch.equal(a.scale, b.scale)
