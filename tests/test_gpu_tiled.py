"""Parity of the tile-major code layout (SQ_LAYOUT_TILED) with the CPU oracle,
through the C-ABI: the quantizer's codes, groups, scale and shift-folded
operand, the K padding it zero-fills, the transposed tensor codes, and the
dgrad / wgrad int32 accumulators (bit for bit) and fp32 outputs (bit for bit,
within the 1e-6 relative bar) on every row, at sizes that span several
tiles, ragged edges, fold windows, split K and every tile shape the GEMM
picks.  Inputs are seeded and synthetic."""
import numpy as np
import pytest

import oracle
from paper_2411_10948_amd import workloads
from tests.test_gpu_parity import _dev, _grad, check_layer, check_quant

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sq():
    import torch
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    from paper_2411_10948_amd import shiftquant
    shiftquant.load()
    oracle.set_threads(16)
    return shiftquant


QUANT_CASES = [  # M, C, bits, N_G, rounding
    (1, 1, 4, 4, 0), (5, 3, 4, 4, 0), (129, 67, 4, 4, 0), (300, 130, 6, 4, 0), (1000, 257, 6, 4, 1),
    (777, 300, 8, 4, 0), (64, 64, 4, 4, 0), (130, 1024, 6, 4, 1),
]


@pytest.mark.parametrize("M,C,bits,ng,mode", QUANT_CASES)
def test_tiled_quantizer(sq, M, C, bits, ng, mode):
    import torch
    print(f"[tiled quantizer] M={M} C={C} b={bits} N_G={ng} mode={mode}", flush=True)
    dY = _grad(M, C, seed=M * 7 + C)
    codes = sq.quantize_grad(_dev(dY), bits, ng, mode, 3, 5, tiled=True)
    torch.cuda.synchronize()
    check_quant(sq, codes, dY, bits, ng, mode, 3, 5)   # codes (through q_t), groups, scale, fold (all rows)
    # K padding written as zeros: q_fold columns [C, roundup(C, 64)), q_t columns [M, roundup(M, 64))
    qf = sq.untile(codes.q_fold).cpu().numpy()
    assert not qf[:, C:sq.round_up(C, 64)].any()
    qt = sq.untile(codes.q_t).cpu().numpy()
    assert not qt[:, M:sq.round_up(M, 64)].any()
    # the row-major quantizer writes the same matrices
    rm = sq.quantize_grad(_dev(dY), bits, ng, mode, 3, 5)
    torch.cuda.synchronize()
    assert np.array_equal(qf[:, :C], rm.q_fold[:, :C].cpu().numpy())
    assert np.array_equal(qt[:, :M], rm.q_t[:, :M].cpu().numpy())


@pytest.mark.parametrize("rows,cols", [(1, 1), (100, 37), (1000, 257), (4099, 130)])
def test_tiled_tensor_codes(sq, rows, cols):
    import torch
    rng = np.random.default_rng(rows + cols)
    T = rng.normal(0, 0.5, (rows, cols)).astype(np.float32)
    q, s = sq.quantize_tensor(_dev(T), 8, transpose=True, tiled=True)
    torch.cuda.synchronize()
    ref, sref = oracle.quantize_tensor(T, 8)
    u = sq.untile(q).cpu().numpy()
    assert np.array_equal(u[:, :rows].T, ref)
    assert not u[:, rows:sq.round_up(rows, 64)].any()
    assert np.float32(sq.scale_to_host(s)["step"]) == np.float32(sref["d0"])


GEMM_CASES = [  # M, C_out, C_in, bits, N_G, rounding: every row compared
    (256, 256, 256, 4, 4, 0),       # the small linear layer
    (1000, 256, 1024, 4, 4, 0),     # ragged M
    (777, 300, 200, 6, 4, 0),       # appended fold windows, ragged M, C_out, C_in
    (40, 128, 96, 4, 4, 0),         # a single skinny row tile
    (65, 64, 48, 8, 3, 1),          # one-window 8-bit with 3 groups, stochastic rounding
    (4099, 768, 3072, 6, 4, 0),     # large tiles with fold windows
    (8000, 1024, 1536, 6, 4, 1),    # tall 128 x 384 tiles
    (12544, 256, 1024, 4, 4, 0),    # the ResNet-50 1x1 layer (weight gradient split over K)
    (3000, 3072, 768, 6, 4, 0),     # MLP-like, wgrad split over K with large tiles
]


@pytest.mark.parametrize("case", GEMM_CASES, ids=["x".join(map(str, c)) for c in GEMM_CASES])
def test_tiled_layer(sq, case):
    M, C_out, C_in, bits, ng, mode = case
    print(f"[tiled layer] {case}", flush=True)
    rng = np.random.default_rng(M + C_out + C_in)
    dY = _grad(M, C_out, seed=M + 1)
    W = (rng.standard_normal((C_out, C_in)) * 0.02).astype(np.float32)
    X = rng.standard_normal((M, C_in)).astype(np.float32)
    r = check_layer(sq, dY, W, X, bits, ng, mode, 9, 2, tiled=True)
    assert r["exact_dX"] and r["exact_dW"]


def test_tiled_dgrad_ranges(sq):
    # producer-side ranges from the tile-major dgrad, anchored on the oracle:
    # dX and its 32-row slab maxima against the oracle's dX, and the next
    # quantizer fed those ranges against the oracle's quantizer on that dX
    import torch
    M, C_out, C_in, bits, ng = 4099, 768, 3072, 6, 4
    print("[tiled dgrad ranges]", flush=True)
    rng = np.random.default_rng(5)
    dY = _grad(M, C_out, seed=77)
    W = (rng.standard_normal((C_out, C_in)) * 0.02).astype(np.float32)
    codes = sq.quantize_grad(_dev(dY), bits, ng, tiled=True)
    wq_t, ws = sq.quantize_tensor(_dev(W), 8, transpose=True, tiled=True)
    slabs = sq.sq_gemm_dgrad_range_slabs(M)
    dX = torch.empty((M, C_in), dtype=torch.float32, device="cuda")
    ranges = torch.full((slabs, C_in), -1, dtype=torch.int32, device="cuda")
    wsz = sq.sq_gemm_dgrad_workspace_size(M, C_out, C_in, codes.params)
    ws_d = torch.empty(max(wsz, 256), dtype=torch.uint8, device="cuda")
    sq.sq_gemm_dgrad_ranged(codes.q_fold, codes.layout, codes.group, codes.scale, wq_t, ws, M, C_out, C_in,
                            codes.params, None, dX, ranges, ws_d)
    nxt = sq.quantize_grad_from_ranges(dX, ranges, bits, ng)
    torch.cuda.synchronize()
    q_ref, g_ref, s_ref, _ = oracle.quantize_grad(dY, bits, ng)
    wq_ref, ws_ref = oracle.quantize_tensor(W, 8)
    dX_ref = oracle.dequant_dgrad(oracle.dgrad(q_ref, g_ref, ng, wq_ref), s_ref["d0"], ws_ref["d0"], ng)
    assert np.array_equal(dX.cpu().numpy().view(np.uint32), dX_ref.view(np.uint32))
    xb = dX_ref.view(np.uint32) & 0x7FFFFFFF
    pad = slabs * 32 - M
    ref = np.concatenate([xb, np.zeros((pad, C_in), np.uint32)]).reshape(slabs, 32, C_in).max(axis=1)
    np.testing.assert_array_equal(ranges.cpu().numpy().view(np.uint32), ref)
    check_quant(sq, nxt, dX_ref, bits, ng, 0, 0, 0)
