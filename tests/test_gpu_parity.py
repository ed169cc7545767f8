"""Parity of the HIP path (through the C-ABI) with the CPU oracle.

Integers -- codes, group ids, scale bit patterns, int32 accumulators -- must
match bit for bit; fp32 outputs within 1e-6 relative (the same IEEE
operations run in the same order on both sides, so they are expected to be
identical).  All inputs are seeded and synthetic.
"""
import numpy as np
import pytest

import oracle
from paper_2411_10948_amd import workloads

pytestmark = pytest.mark.gpu

RTOL = 1e-6


@pytest.fixture(scope="module")
def sq():
    import torch
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    from paper_2411_10948_amd import shiftquant
    shiftquant.load()
    return shiftquant


def _qmax(bits):
    return (1 << (bits - 1)) - 1


def _T(bits):
    Q, T = _qmax(bits), 0
    while Q * (1 << (T + 1)) <= 127:
        T += 1
    return T


def _f32bits(x):
    return int(np.array([x], np.float32).view(np.uint32)[0])


def _dev(a, ld_pad=0, misalign=0):
    import torch
    a = np.ascontiguousarray(a)
    if ld_pad == 0 and misalign == 0:
        return torch.from_numpy(a).cuda()
    rows, cols = a.shape
    buf = torch.zeros(rows * (cols + ld_pad) + misalign, dtype=torch.float32, device="cuda")
    view = buf[misalign:misalign + rows * (cols + ld_pad)].view(rows, cols + ld_pad)[:, :cols]
    view.copy_(torch.from_numpy(a).cuda())
    return view


def expected_fold(g, num_groups, bits, pad=64):
    """The fold of the dgrad operand as include/shiftquant.h documents it.

    Shifts sh = N_G - 1 - g are cut into windows [B, B + T]; the window with
    the most channels (lowest B on ties) keeps the channels' own columns, the
    other non-empty windows become appended regions, visited in descending B.
    Returns the regions (base, members, is_main) in visiting order, the
    appended-column list, and per channel (t, pos).
    """
    T, S = _T(bits), num_groups - 1
    sh = S - g.astype(np.int64)
    n = np.bincount(sh, minlength=S + 1) if sh.size else np.zeros(S + 1, np.int64)
    best, bstar = -1, 0
    for B in range(0, max(0, S - T) + 1):
        c = int(n[B:min(S, B + T) + 1].sum())
        if c > best:
            best, bstar = c, B
    wins = [(lo, min(S, lo + T), False) for lo in range(bstar + T + 1, S + 1, T + 1)][::-1]
    wins.append((bstar, min(S, bstar + T), True))
    hi = bstar - 1
    while hi >= 0:
        lo = max(0, hi - T)
        wins.append((lo, hi, False))
        hi = lo - 1
    regions = []
    for lo, hi, is_main in wins:
        members = [int(c) for c in np.nonzero((sh >= lo) & (sh <= hi))[0]]
        if members or is_main:
            regions.append((lo, members, is_main))
    cols, t, pos = [], np.zeros(sh.size, np.int64), np.full(sh.size, -1, np.int64)
    for base, members, is_main in regions:
        for c in members:
            t[c] = sh[c] - base
        if not is_main:
            for c in members:
                pos[c] = len(cols)
                cols.append(c)
            cols += [-1] * ((-len(members)) % pad)
    return regions, cols, t, pos


def check_fold(codes, q_ref, g_ref, bits, ng, rows=None):
    """Layout words and the shift-folded operand (all rows, or the given ones)."""
    C = q_ref.shape[1]
    regions, cols, t, pos = expected_fold(g_ref, ng, bits)
    lay = codes.layout.cpu().numpy()
    ext_max = len(lay) - 32 - C
    base_col = (C + 63) // 64 * 64
    nr = len(regions)
    main_r = [i for i, r in enumerate(regions) if r[2]][0]
    flat, starts = 0, []
    for base, members, is_main in regions:
        starts.append(flat)
        flat += base_col if is_main else (len(members) + 63) // 64 * 64
    H = sum((len(r[1]) + 63) // 64 * 64 for r in regions[:main_r])
    assert lay[0] == nr and lay[1] == len(cols) and lay[2] == base_col, lay[:8]
    assert lay[3] == regions[-1][0] and lay[4] == H, lay[:8]
    assert list(lay[8:8 + nr]) == starts
    assert list(lay[16:16 + nr]) == [0] + [regions[i - 1][0] - regions[i][0] for i in range(1, nr)]
    assert len(cols) <= ext_max
    assert list(lay[32:32 + len(cols)]) == cols
    assert np.array_equal(lay[32 + ext_max:32 + ext_max + C], ((pos + 1) << 4) | t)
    if q_ref.shape[0] == 0:
        return
    fold = codes.q_fold
    if codes.params.tiled:   # tile-major: compare the row-major matrix it encodes
        from paper_2411_10948_amd import shiftquant
        fold = shiftquant.untile(fold)
    if rows is None:
        qf = fold.cpu().numpy().astype(np.int64)
        shifted = q_ref.astype(np.int64) << t[None, :]
    else:
        import torch
        qf = fold.index_select(0, torch.as_tensor(rows, device="cuda")).cpu().numpy().astype(np.int64)
        shifted = q_ref[rows].astype(np.int64) << t[None, :]
    main = pos < 0
    assert np.array_equal(qf[:, :C][:, main], shifted[:, main]), "main fold columns"
    assert not qf[:, :C][:, ~main].any(), "main columns of appended channels must be 0"
    for c in np.nonzero(~main)[0]:
        assert np.array_equal(qf[:, base_col + pos[c]], shifted[:, c]), f"appended column of channel {c}"


def check_quant(sq, codes, dY, bits, ng, mode, seed, offset, fold_rows=None):
    q_ref, g_ref, s_ref, _ = oracle.quantize_grad(dY, bits, ng, mode, seed, offset)
    M, C = dY.shape
    q = codes.codes().cpu().numpy()
    g = codes.group.cpu().numpy()
    assert np.array_equal(g, g_ref), "group ids differ"
    bad = np.argwhere(q != q_ref)
    assert bad.size == 0, f"{len(bad)} codes differ, first at {bad[:5].tolist()}"
    s = sq.scale_to_host(codes.scale)
    assert s["bits"][0] == _f32bits(s_ref["r_max"])
    assert s["bits"][1] == _f32bits(s_ref["inv0"])
    assert s["bits"][2] == _f32bits(s_ref["d0"])
    assert s["flags"] == s_ref["flags"]
    check_fold(codes, q_ref, g_ref, bits, ng, fold_rows)
    return q_ref, g_ref, s_ref


def _rows(sq, t, tiled):
    """A code matrix as row-major (a copy when tile-major)."""
    return sq.untile(t) if tiled else t


def check_layer(sq, dY, W, X, bits, ng, mode=0, seed=0, offset=0, dgrad_rows=None, wgrad_rows=None,
                want_acc=True, fold_rows=None, tiled=False):
    import torch
    M, C_out = dY.shape
    C_in = W.shape[1]
    codes = sq.quantize_grad(_dev(dY), bits, ng, mode, seed, offset, tiled=tiled)
    wq_t, ws = sq.quantize_tensor(_dev(W), 8, transpose=True, tiled=tiled)
    xq_t, xs = sq.quantize_tensor(_dev(X), 8, transpose=True, tiled=tiled)
    acc_d, dX = sq.gemm_dgrad(codes, wq_t, ws, want_acc=want_acc)
    acc_w, dW = sq.gemm_wgrad(codes, xq_t, xs, want_acc=want_acc)
    torch.cuda.synchronize()
    q_ref, g_ref, s_ref = check_quant(sq, codes, dY, bits, ng, mode, seed, offset, fold_rows)

    wq_ref, ws_ref = oracle.quantize_tensor(W, 8)
    xq_ref, xs_ref = oracle.quantize_tensor(X, 8)
    assert np.array_equal(_rows(sq, wq_t, tiled)[:, :C_out].t().cpu().numpy(), wq_ref)
    assert np.array_equal(_rows(sq, xq_t, tiled)[:, :M].t().cpu().numpy(), xq_ref)
    for got, ref in ((ws, ws_ref), (xs, xs_ref)):
        h = sq.scale_to_host(got)
        assert h["bits"][:3] == [_f32bits(ref["r_max"]), _f32bits(ref["inv0"]), _f32bits(ref["d0"])]
        assert h["flags"] == ref["flags"]

    rows_d = np.arange(M) if dgrad_rows is None else np.asarray(dgrad_rows)
    rows_w = np.arange(C_out) if wgrad_rows is None else np.asarray(wgrad_rows)
    A_ref = oracle.dgrad(q_ref, g_ref, ng, wq_ref, None if dgrad_rows is None else rows_d)
    B_ref = oracle.wgrad(q_ref, xq_ref, None if wgrad_rows is None else rows_w)
    dX_ref = oracle.dequant_dgrad(A_ref, s_ref["d0"], ws_ref["d0"], ng)
    dW_ref = oracle.dequant_wgrad(B_ref, g_ref[rows_w], s_ref["d0"], xs_ref["d0"])

    rows_d_t = torch.as_tensor(rows_d, device="cuda", dtype=torch.long)
    rows_w_t = torch.as_tensor(rows_w, device="cuda", dtype=torch.long)
    if want_acc:
        assert np.array_equal(acc_d.index_select(0, rows_d_t).cpu().numpy(), A_ref), "dgrad int32 differs"
        assert np.array_equal(acc_w.index_select(0, rows_w_t).cpu().numpy(), B_ref), "wgrad int32 differs"
    dXg = dX.index_select(0, rows_d_t).cpu().numpy()
    dWg = dW.index_select(0, rows_w_t).cpu().numpy()
    np.testing.assert_allclose(dXg, dX_ref, rtol=RTOL, atol=0)
    np.testing.assert_allclose(dWg, dW_ref, rtol=RTOL, atol=0)
    return {"codes": codes, "dX": dX, "dW": dW, "acc_d": acc_d, "acc_w": acc_w,
            "exact_dX": bool(np.array_equal(dXg.view(np.uint32), dX_ref.view(np.uint32))),
            "exact_dW": bool(np.array_equal(dWg.view(np.uint32), dW_ref.view(np.uint32)))}


def _grad(M, C, seed, s=2.0, frac=0.03, factor=100.0, dist="normal"):
    return workloads.make_grad(M, C, seed=seed, sigma_s=s, outlier_frac=frac, outlier_factor=factor, dist=dist)


# ---------------------------------------------------------------------------
# quantizer
# ---------------------------------------------------------------------------
QUANT_SHAPES = [(1, 1), (1, 7), (5, 3), (64, 64), (129, 67), (300, 130), (257, 96), (1000, 257), (130, 1024)]


@pytest.mark.parametrize("shape", QUANT_SHAPES, ids=[f"{m}x{c}" for m, c in QUANT_SHAPES])
@pytest.mark.parametrize("bits,ng", [(4, 4), (6, 4), (8, 4), (2, 8), (5, 1), (7, 3)])
@pytest.mark.parametrize("mode", [0, 1])
def test_quantize_grad_parity(sq, shape, bits, ng, mode):
    import torch
    M, C = shape
    dY = _grad(M, C, seed=M * 7 + C + bits)
    codes = sq.quantize_grad(_dev(dY), bits, ng, mode, seed=11, offset=5)
    torch.cuda.synchronize()
    check_quant(sq, codes, dY, bits, ng, mode, 11, 5)


@pytest.mark.parametrize("ld_pad,misalign", [(3, 0), (4, 0), (0, 1), (5, 3)])
@pytest.mark.parametrize("mode", [0, 1])
def test_quantize_grad_strided_input(sq, ld_pad, misalign, mode):
    import torch
    dY = _grad(200, 77, seed=3)
    codes = sq.quantize_grad(_dev(dY, ld_pad, misalign), 6, 4, mode, seed=2, offset=9)
    torch.cuda.synchronize()
    check_quant(sq, codes, dY, 6, 4, mode, 2, 9)


def test_quantize_degenerate_tensors(sq):
    import torch
    cases = {
        "zeros": np.zeros((70, 33), np.float32),
        "tiny": np.full((70, 33), 2.0 ** -100, np.float32),
        "at_threshold": np.full((70, 33), 2.0 ** -96, np.float32),
        "single": np.array([[-3.5]], np.float32),
    }
    nan = _grad(70, 33, seed=1)
    nan[17, 5] = np.nan
    cases["nan"] = nan
    inf = _grad(70, 33, seed=2)
    inf[69, 32] = -np.inf
    cases["inf"] = inf
    huge = _grad(70, 33, seed=4)
    huge[0, 0] = 3.0e38
    cases["huge"] = huge
    subn = _grad(70, 33, seed=5) * np.float32(1e-35)
    cases["subnormal_scale"] = subn.astype(np.float32)
    for name, dY in cases.items():
        for mode in (0, 1):
            codes = sq.quantize_grad(_dev(dY), 4, 4, mode, seed=1, offset=1)
            torch.cuda.synchronize()
            check_quant(sq, codes, dY, 4, 4, mode, 1, 1)
    # empty token dimension
    codes = sq.quantize_grad(torch.zeros((0, 8), device="cuda"), 4, 4)
    torch.cuda.synchronize()
    s = sq.scale_to_host(codes.scale)
    assert s["flags"] == sq.FLAG_ZERO
    assert np.all(codes.group.cpu().numpy() == 3)


def test_stochastic_rounding_streams(sq):
    import torch
    dY = _grad(64, 40, seed=9)
    x = _dev(dY)
    a = sq.quantize_grad(x, 4, 4, 1, seed=3, offset=10).codes().clone()
    b = sq.quantize_grad(x, 4, 4, 1, seed=3, offset=10).codes().clone()
    c = sq.quantize_grad(x, 4, 4, 1, seed=3, offset=11).codes().clone()
    d = sq.quantize_grad(x, 4, 4, 1, seed=4, offset=10).codes().clone()
    torch.cuda.synchronize()
    assert torch.equal(a, b)
    assert not torch.equal(a, c) and not torch.equal(a, d)


@pytest.mark.parametrize("transpose", [0, 1])
@pytest.mark.parametrize("shape", [(1, 1), (33, 17), (300, 129), (64, 1000)])
@pytest.mark.parametrize("bits", [8, 4])
def test_quantize_tensor_parity(sq, transpose, shape, bits):
    import torch
    rng = np.random.default_rng(shape[0] + shape[1])
    T = (rng.standard_normal(shape) * 0.02).astype(np.float32)
    q, s = sq.quantize_tensor(_dev(T), bits, transpose=bool(transpose))
    torch.cuda.synchronize()
    q_ref, s_ref = oracle.quantize_tensor(T, bits)
    got = q[:, :shape[0]].t() if transpose else q[:, :shape[1]]
    assert np.array_equal(got.cpu().numpy(), q_ref)
    h = sq.scale_to_host(s)
    assert h["bits"][:3] == [_f32bits(s_ref["r_max"]), _f32bits(s_ref["inv0"]), _f32bits(s_ref["d0"])]


# ---------------------------------------------------------------------------
# GEMMs on small layers (several tiles, ragged tails, every fold case)
# ---------------------------------------------------------------------------
LAYERS = [(1, 1, 1), (7, 5, 3), (130, 67, 45), (256, 256, 256), (300, 200, 129), (513, 130, 260),
          (64, 1100, 40)]


@pytest.mark.parametrize("layer", LAYERS, ids=[f"{m}x{co}x{ci}" for m, co, ci in LAYERS])
@pytest.mark.parametrize("bits,ng", [(4, 4), (6, 4), (8, 4), (7, 3), (2, 8), (5, 1)])
def test_layer_parity(sq, layer, bits, ng):
    M, C_out, C_in = layer
    rng = np.random.default_rng(M + C_out + C_in + bits)
    dY = _grad(M, C_out, seed=M + bits, s=2.5)
    W = (rng.standard_normal((C_out, C_in)) * 0.02).astype(np.float32)
    X = rng.standard_normal((M, C_in)).astype(np.float32)
    mode = 1 if (M + bits) % 2 else 0
    check_layer(sq, dY, W, X, bits, ng, mode=mode, seed=7, offset=3)


def _grouped_grad(M, groups, seed):
    """dY whose channel c has range exactly 0.75 * 2^-groups[c], so that (with a
    channel in group 0) its ShiftQuant group is groups[c]."""
    rng = np.random.default_rng(seed)
    scale = 0.75 * np.exp2(-np.asarray(groups, np.float64))
    dY = rng.uniform(-1.0, 1.0, (M, len(groups))) * scale[None, :]
    hit = rng.integers(0, M, len(groups))
    dY[hit, np.arange(len(groups))] = scale * np.where(rng.random(len(groups)) < 0.5, -1.0, 1.0)
    return dY.astype(np.float32)


def _group_pattern(name, C, ng, seed):
    rng = np.random.default_rng(seed)
    last = ng - 1
    if name == "all_g0":
        g = np.zeros(C, np.int64)
    elif name == "mostly_g0":
        g = np.where(rng.random(C) < 0.8, 0, last)
    elif name == "middle":
        g = np.where(rng.random(C) < 0.7, min(1, last), rng.integers(0, ng, C))
    elif name == "bimodal":
        g = np.where(rng.random(C) < 0.5, 0, last)
    else:   # spread
        g = rng.integers(0, ng, C)
    g[0] = 0
    return g


FOLD_PATTERNS = ["all_g0", "mostly_g0", "middle", "bimodal", "spread"]


@pytest.mark.parametrize("layer", [(200, 130, 70), (256, 192, 128)], ids=["ragged", "aligned"])
@pytest.mark.parametrize("pattern", FOLD_PATTERNS)
@pytest.mark.parametrize("bits,ng", [(6, 4), (8, 4), (7, 3), (2, 8), (3, 8), (8, 6)])
def test_fold_windows(sq, layer, pattern, bits, ng):
    # channel groups forced so that the main window sits at the bottom, in the
    # middle or at the top of the shift range, with appended windows above,
    # below or on both sides
    M, C_out, C_in = layer
    g = _group_pattern(pattern, C_out, ng, seed=C_out + bits)
    dY = _grouped_grad(M, g, seed=M + ng)
    q_ref, g_ref, _, _ = oracle.quantize_grad(dY, bits, ng, 0, 0, 0)
    assert np.array_equal(g_ref, g)
    rng = np.random.default_rng(bits * 10 + ng)
    W = (rng.standard_normal((C_out, C_in)) * 0.02).astype(np.float32)
    X = rng.standard_normal((M, C_in)).astype(np.float32)
    check_layer(sq, dY, W, X, bits, ng, mode=(M + bits) % 2)


@pytest.mark.parametrize("bits,ng", [(6, 4), (8, 4)])
def test_fold_windows_many_channels(sq, bits, ng):
    # more than 16 * 1024 channels: the finalize kernel ranks appended
    # channels over several chunks of rounds
    M, C = 40, 20000
    g = _group_pattern("spread", C, ng, seed=11)
    dY = _grouped_grad(M, g, seed=12)
    import torch
    codes = sq.quantize_grad(_dev(dY), bits, ng, 0, 0, 0)
    torch.cuda.synchronize()
    q_ref, g_ref, _ = check_quant(sq, codes, dY, bits, ng, 0, 0, 0)
    assert np.array_equal(g_ref, g)


@pytest.mark.parametrize("pattern", ["mostly_g0", "spread"])
def test_fold_windows_large_tiles(sq, pattern):
    # the same on the large-tile pipelined GEMM (K >= 1024, >= 256 output tiles)
    M, C_out, C_in, bits, ng = 4096, 1024, 4096, 6, 4
    g = _group_pattern(pattern, C_out, ng, seed=3)
    dY = _grouped_grad(M, g, seed=4)
    rng = np.random.default_rng(6)
    W = (rng.standard_normal((C_out, C_in)) * 0.02).astype(np.float32)
    X = rng.standard_normal((M, C_in)).astype(np.float32)
    rows_d = np.unique(np.r_[0, 255, 256, M - 1, rng.integers(0, M, 20)])
    rows_w = np.unique(np.r_[0, C_out - 1, rng.integers(0, C_out, 10)])
    check_layer(sq, dY, W, X, bits, ng, dgrad_rows=rows_d, wgrad_rows=rows_w, fold_rows=rows_d)


@pytest.mark.parametrize("shape,bits", [((8000, 1024, 1536), 6), ((8000 - 77, 1024, 1536 - 40), 4)],
                         ids=["8000x1024x1536-b6", "7923x1024x1496-b4"])
def test_dgrad_tall_tiles(sq, shape, bits):
    # 128 x 384 tiles: the 256 x 256 tiling would leave CUs idle (192 tiles),
    # the tall one fills more of them; 6-bit codes take the appended fold
    # windows, the second shape has ragged tiles in both directions
    M, C_out, C_in = shape
    g = _group_pattern("spread", C_out, 4, seed=8)
    dY = _grouped_grad(M, g, seed=9)
    rng = np.random.default_rng(10)
    W = (rng.standard_normal((C_out, C_in)) * 0.02).astype(np.float32)
    X = rng.standard_normal((M, C_in)).astype(np.float32)
    rows_d = np.unique(np.r_[0, 127, 128, M - 2, M - 1, rng.integers(0, M, 24)])
    rows_w = np.unique(np.r_[0, C_out - 1, rng.integers(0, C_out, 6)])
    check_layer(sq, dY, W, X, bits, 4, dgrad_rows=rows_d, wgrad_rows=rows_w, fold_rows=rows_d)


def test_wgrad_tall_tiles(sq):
    # the weight gradient of a 2048 -> 4096 layer over 2048 tokens: 128 large
    # tiles (no split), 192 tall ones; per-row group scales in the epilogue
    M, C_out, C_in = 2048, 4096, 2048
    g = _group_pattern("spread", C_out, 4, seed=11)
    dY = _grouped_grad(M, g, seed=12)
    rng = np.random.default_rng(13)
    W = (rng.standard_normal((C_out, C_in)) * 0.02).astype(np.float32)
    X = rng.standard_normal((M, C_in)).astype(np.float32)
    rows_w = np.unique(np.r_[0, 127, 128, C_out - 1, np.nonzero(g < 3)[0][:6], rng.integers(0, C_out, 10)])
    rows_d = np.unique(np.r_[0, M - 1, rng.integers(0, M, 6)])
    check_layer(sq, dY, W, X, 6, 4, dgrad_rows=rows_d, wgrad_rows=rows_w)


def test_fp32_only_outputs_match_with_acc(sq):
    import torch
    M, C_out, C_in = 300, 200, 129
    rng = np.random.default_rng(1)
    dY = _grad(M, C_out, seed=1)
    W = (rng.standard_normal((C_out, C_in)) * 0.02).astype(np.float32)
    X = rng.standard_normal((M, C_in)).astype(np.float32)
    codes = sq.quantize_grad(_dev(dY), 6, 4)
    wq_t, ws = sq.quantize_tensor(_dev(W), 8)
    xq_t, xs = sq.quantize_tensor(_dev(X), 8)
    a1, dX1 = sq.gemm_dgrad(codes, wq_t, ws, want_acc=True)
    _, dX2 = sq.gemm_dgrad(codes, wq_t, ws, want_acc=False)
    b1, dW1 = sq.gemm_wgrad(codes, xq_t, xs, want_acc=True)
    _, dW2 = sq.gemm_wgrad(codes, xq_t, xs, want_acc=False)
    b3, dW3 = sq.gemm_wgrad(codes, xq_t, xs, want_acc=True, want_out=False)
    torch.cuda.synchronize()
    assert torch.equal(dX1, dX2) and torch.equal(dW1, dW2) and torch.equal(b1, b3) and dW3 is None
    # standalone dequantization of the accumulators gives the fused outputs
    outd = torch.empty_like(dX1)
    sq.sq_dequant(a1, 0, None, codes.scale, ws, 4, outd)
    outw = torch.empty_like(dW1)
    sq.sq_dequant(b1, 1, codes.group, codes.scale, xs, 4, outw)
    torch.cuda.synchronize()
    assert torch.equal(outd, dX1) and torch.equal(outw, dW1)


def test_wgrad_split_k(sq):
    # long token dimension, small output: the wgrad splits K over many blocks
    M, C_out, C_in = 20000, 64, 96
    rng = np.random.default_rng(5)
    dY = _grad(M, C_out, seed=5)
    W = (rng.standard_normal((C_out, C_in)) * 0.05).astype(np.float32)
    X = np.maximum(rng.standard_normal((M, C_in)), 0).astype(np.float32)
    assert sq.sq_gemm_wgrad_workspace_size(M, C_out, C_in, sq.Params.make(4)) > 0
    check_layer(sq, dY, W, X, 4, 4, dgrad_rows=[0, 1, 5000, 19999])
    check_layer(sq, dY, W, X, 4, 4, dgrad_rows=[3, 19998], want_acc=False)


@pytest.mark.parametrize("shape", [(4096, 1024, 2048), (4136, 1024, 2048), (5120, 1280, 1344)])
def test_wgrad_large_tiles_split_k(sq, shape):
    # few 256 x 256 output tiles and a long token dimension: the wgrad splits
    # K over large tiles (4 or 5 slices); 4136 tokens leave a ragged last K
    # tile, which takes the register-staged kernel
    M, C_out, C_in = shape
    rng = np.random.default_rng(M + C_in)
    dY = _grad(M, C_out, seed=C_in)
    W = (rng.standard_normal((C_out, C_in)) * 0.05).astype(np.float32)
    X = np.maximum(rng.standard_normal((M, C_in)), 0).astype(np.float32)
    assert sq.sq_gemm_wgrad_workspace_size(M, C_out, C_in, sq.Params.make(4)) > 0
    check_layer(sq, dY, W, X, 4, 4, dgrad_rows=[0, 1, M // 2, M - 1],
                wgrad_rows=[0, 1, 255, 256, C_out // 2, C_out - 1])
    check_layer(sq, dY, W, X, 6, 4, dgrad_rows=[2, M - 2], wgrad_rows=[3, C_out - 2], want_acc=False)


@pytest.mark.parametrize("shape", [(4096, 40, 200), (8192, 64, 197), (2048, 1, 64), (16384, 64, 576)])
def test_wgrad_narrow_outputs(sq, shape):
    # at most 64 output rows and a token count that is a multiple of 64: the
    # 64-row tile with split-K, and the reduce with and without 4-aligned rows
    M, C_out, C_in = shape
    rng = np.random.default_rng(C_in)
    dY = _grad(M, C_out, seed=C_out)
    W = (rng.standard_normal((C_out, C_in)) * 0.05).astype(np.float32)
    X = np.maximum(rng.standard_normal((M, C_in)), 0).astype(np.float32)
    check_layer(sq, dY, W, X, 4, 4, dgrad_rows=[0, 1, M // 2, M - 1])


# ---------------------------------------------------------------------------
# convolution input gradient with implicit im2col / col2im
# ---------------------------------------------------------------------------
CONV_GPU_CASES = [  # N, H, W, C_out, C_in, KH, KW, PH, PW, bits, N_G
    (2, 9, 7, 64, 64, 3, 3, 1, 1, 4, 4),      # same-size 3x3: several tiles, ragged last tile
    (1, 13, 11, 48, 40, 3, 3, 1, 1, 6, 4),    # fold with appended windows; C_out, C_in not multiples of 64
    (1, 10, 12, 96, 160, 3, 3, 0, 1, 4, 4),   # unpadded rows, padded columns; C_in > 64
    (2, 6, 5, 32, 24, 1, 1, 0, 0, 8, 3),      # 1 x 1 window
    (1, 8, 8, 64, 64, 5, 5, 2, 2, 4, 4),      # 5 x 5 window
    (1, 7, 9, 130, 64, 2, 3, 1, 0, 6, 4),     # even window height, one-sided padding
    (3, 4, 4, 200, 72, 3, 3, 1, 1, 8, 4),     # 8-bit codes: several appended windows
    (1, 5, 63, 64, 64, 3, 3, 1, 1, 4, 4),     # widest image whose row window is staged whole
    (1, 4, 64, 64, 64, 3, 3, 1, 1, 4, 4),     # one column wider: per-tap loads
    (2, 5, 6, 64, 32, 1, 3, 0, 1, 6, 4),      # 1 x 3 window
]


def _conv_layer(N, H, W, C_out, C_in, KH, KW, PH, PW, seed):
    Ho, Wo = H + 2 * PH - KH + 1, W + 2 * PW - KW + 1
    rng = np.random.default_rng(seed)
    dY = _grad(N * Ho * Wo, C_out, seed=seed)
    Wt = (rng.standard_normal((C_out, KH * KW * C_in)) * np.sqrt(2.0 / (KH * KW * C_in))).astype(np.float32)
    return dY, Wt


def check_conv(sq, case, pix=None, mode=0):
    import torch
    N, H, W, C_out, C_in, KH, KW, PH, PW, bits, ng = case
    dY, Wt = _conv_layer(N, H, W, C_out, C_in, KH, KW, PH, PW, seed=sum(case))
    codes = sq.quantize_grad(_dev(dY), bits, ng, mode, 7, 0)
    wq_t, ws = sq.quantize_tensor(_dev(Wt), 8, transpose=True)
    acc, dX = sq.conv_dgrad(codes, wq_t, ws, N, H, W, KH, KW, PH, PW, want_acc=True)
    _, dX2 = sq.conv_dgrad(codes, wq_t, ws, N, H, W, KH, KW, PH, PW, want_acc=False)
    torch.cuda.synchronize()
    q_ref, g_ref, s_ref = check_quant(sq, codes, dY, bits, ng, mode, 7, 0, fold_rows=None if pix is None else [0])
    wq_ref, ws_ref = oracle.quantize_tensor(Wt, 8)
    A_ref = oracle.conv_dgrad(q_ref, g_ref, ng, wq_ref, N, H, W, KH, KW, PH, PW, pix)
    dX_ref = oracle.dequant_dgrad(A_ref, s_ref["d0"], ws_ref["d0"], ng)
    rows = torch.arange(N * H * W, device="cuda") if pix is None else torch.as_tensor(pix, device="cuda")
    got = acc.index_select(0, rows).cpu().numpy()
    bad = np.argwhere(got != A_ref)
    assert bad.size == 0, f"{len(bad)} conv dgrad accumulators differ, first at {bad[:4].tolist()}"
    np.testing.assert_allclose(dX.index_select(0, rows).cpu().numpy(), dX_ref, rtol=RTOL, atol=0)
    assert torch.equal(dX, dX2)


@pytest.mark.parametrize("case", CONV_GPU_CASES, ids=["x".join(map(str, c)) for c in CONV_GPU_CASES])
def test_conv_dgrad_parity(sq, case):
    check_conv(sq, case)


def test_conv_dgrad_stochastic_codes(sq):
    check_conv(sq, (1, 9, 9, 72, 64, 3, 3, 1, 1, 6, 4), mode=1)


def test_conv_dgrad_full_resnet18_layer(sq):
    # the full 64 x 56 x 56 x 64 layer; pixels sampled on image borders,
    # corners, tile boundaries and interiors
    N, H, W = 64, 56, 56
    rng = np.random.default_rng(11)
    picks = []
    for n in (0, 1, 31, 63):
        for ih, iw in ((0, 0), (0, 55), (55, 0), (55, 55), (0, 27), (27, 0), (55, 31), (13, 55), (28, 28)):
            picks.append((n * H + ih) * W + iw)
    picks += [255, 256, 511, 512, 3135, 3136] + list(rng.integers(0, N * H * W, 200))
    check_conv(sq, (N, H, W, 64, 64, 3, 3, 1, 1, 4, 4), pix=np.array(sorted(set(int(p) for p in picks))))


def test_conv_dgrad_rejects_bad_geometry(sq):
    import torch
    dY, Wt = _conv_layer(1, 5, 5, 16, 8, 3, 3, 1, 1, seed=1)
    codes = sq.quantize_grad(_dev(dY), 4, 4)
    wq_t, ws = sq.quantize_tensor(_dev(Wt), 8, transpose=True)
    with pytest.raises(sq.ShiftQuantError):
        sq.conv_dgrad(codes, wq_t, ws, 1, 5, 5, 3, 3, 3, 1)      # padding >= window
    with pytest.raises(sq.ShiftQuantError):
        sq.conv_dgrad(codes, wq_t, ws, 1, 1, 5, 3, 3, 0, 1)      # window taller than the input
    torch.cuda.synchronize()


@pytest.mark.parametrize("bits,ng,shape", [(4, 4, (300, 200, 96)), (6, 4, (257, 130, 64)), (8, 6, (129, 300, 80)),
                                           (5, 1, (64, 64, 64)), (6, 3, (1000, 1024, 256))])
def test_dgrad_grouped_matches_shiftmm(sq, bits, ng, shape):
    # the GEMM-based implementation (per-group sub-GEMMs after rearrangement,
    # then shift and sum) gives the ShiftMM accumulator and dX bit for bit
    import torch
    M, C_out, C_in = shape
    rng = np.random.default_rng(M + C_out)
    dY = _grad(M, C_out, seed=C_in + bits, s=2.5)
    W = (rng.standard_normal((C_out, C_in)) * 0.05).astype(np.float32)
    codes = sq.quantize_grad(_dev(dY), bits, ng)
    wq_t, ws = sq.quantize_tensor(_dev(W), 8, transpose=True)
    a1, d1 = sq.gemm_dgrad(codes, wq_t, ws, want_acc=True)
    a2, d2 = sq.gemm_dgrad_grouped(codes, wq_t, ws, want_acc=True)
    torch.cuda.synchronize()
    assert torch.equal(a1, a2) and torch.equal(d1, d2)
    q_ref, g_ref, s_ref, _ = oracle.quantize_grad(dY, bits, ng)
    wq_ref, _ = oracle.quantize_tensor(W, 8)
    rows = np.unique(np.r_[0, M - 1, rng.integers(0, M, 8)])
    A_ref = oracle.dgrad(q_ref, g_ref, ng, wq_ref, rows)
    assert np.array_equal(a2.index_select(0, torch.as_tensor(rows, device="cuda")).cpu().numpy(), A_ref)


# ---------------------------------------------------------------------------
# forward pass: ShiftQuant activations, per-channel weights (Sec. 5.1)
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("shape", [(1, 1), (7, 5), (64, 300), (257, 96), (1000, 33)])
@pytest.mark.parametrize("axis", [0, 1])
@pytest.mark.parametrize("transpose", [0, 1])
def test_quantize_channels_parity(sq, shape, axis, transpose):
    import torch
    rows, cols = shape
    rng = np.random.default_rng(rows * 3 + cols + axis)
    T = (rng.standard_normal(shape) * np.exp(2 * rng.standard_normal((rows, 1)))).astype(np.float32)
    if rows > 2 and cols > 2:
        T[1, :] = 0.0            # a zero row
        T[:, 2] = 0.0            # a zero column
        T[rows - 1, cols - 1] = np.inf
    q, scales = sq.quantize_channels(_dev(T), 4 if axis else 8, axis, bool(transpose))
    torch.cuda.synchronize()
    q_ref, s_ref = oracle.quantize_channels(T, 4 if axis else 8, axis)
    got = q.cpu().numpy()
    got = got[:, :rows].T if transpose else got[:, :cols]
    assert np.array_equal(got, q_ref)
    h = scales.cpu().numpy()
    for ch, s in enumerate(s_ref):
        assert list(h[ch, :3].view(np.uint32)) == [_f32bits(s["r_max"]), _f32bits(s["inv0"]), _f32bits(s["d0"])]
        assert int(h[ch, 3:4].view(np.uint32)[0]) == s["flags"]


FORWARD_CASES = [(200, 96, 64, 4, 4), (333, 130, 72, 6, 4), (129, 256, 300, 8, 6), (1000, 768, 512, 6, 3),
                 (64, 64, 64, 4, 1), (4096, 1024, 1024, 4, 4)]


@pytest.mark.parametrize("case", FORWARD_CASES, ids=["x".join(map(str, c)) for c in FORWARD_CASES])
def test_forward_parity(sq, case):
    # Y = X W^T: X in ShiftQuant groups over its channels, W per output channel
    import torch
    M, C_in, C_out, bits, ng = case
    rng = np.random.default_rng(M + C_in)
    X = _grad(M, C_in, seed=C_out, s=1.5)
    W = (rng.standard_normal((C_out, C_in)) * np.exp(rng.standard_normal((C_out, 1)))).astype(np.float32)
    xc = sq.quantize_grad(_dev(X), bits, ng)
    wq, ws = sq.quantize_channels(_dev(W), 8, 0, False)
    acc, Y = sq.gemm_forward(xc, wq, ws, want_acc=True)
    torch.cuda.synchronize()
    xq_ref, g_ref, xs_ref = check_quant(sq, xc, X, bits, ng, 0, 0, 0, fold_rows=[0, M - 1])
    wq_ref, ws_ref = oracle.quantize_channels(W, 8, 0)
    rows = np.arange(M) if M * C_in * C_out < 2e8 else np.unique(np.r_[0, M - 1, rng.integers(0, M, 20)])
    A_ref = oracle.dgrad(xq_ref, g_ref, ng, np.ascontiguousarray(wq_ref.T), rows)
    d_w = np.array([s["d0"] for s in ws_ref], np.float32)
    Y_ref = oracle.dequant_cols(A_ref, xs_ref["d0"], d_w, ng)
    rt = torch.as_tensor(rows, device="cuda")
    assert np.array_equal(acc.index_select(0, rt).cpu().numpy(), A_ref)
    np.testing.assert_allclose(Y.index_select(0, rt).cpu().numpy(), Y_ref, rtol=RTOL, atol=0)
    # standalone dequantization (kind 2) of the accumulator gives the fused output
    out = torch.empty_like(Y)
    sq.sq_dequant(acc, 2, None, xc.scale, ws, ng, out)
    torch.cuda.synchronize()
    assert torch.equal(out, Y)


def test_loss_propagation_per_input_channel_weights(sq):
    # dX = dY W with W quantized per input channel: the forward call with the
    # gradient's codes, W^T codes and their per-column scales
    import torch
    M, C_out, C_in, bits, ng = 700, 200, 160, 6, 4
    rng = np.random.default_rng(12)
    dY = _grad(M, C_out, seed=12)
    W = (rng.standard_normal((C_out, C_in)) * np.exp(rng.standard_normal((1, C_in)))).astype(np.float32)
    codes = sq.quantize_grad(_dev(dY), bits, ng)
    wq_t, ws = sq.quantize_channels(_dev(W), 8, 1, True)      # [C_in, C_out], one scale per input channel
    acc, dX = sq.gemm_forward(codes, wq_t, ws, want_acc=True)
    torch.cuda.synchronize()
    q_ref, g_ref, s_ref = check_quant(sq, codes, dY, bits, ng, 0, 0, 0)
    wq_ref, ws_ref = oracle.quantize_channels(W, 8, 1)
    A_ref = oracle.dgrad(q_ref, g_ref, ng, wq_ref)
    dX_ref = oracle.dequant_cols(A_ref, s_ref["d0"], np.array([s["d0"] for s in ws_ref], np.float32), ng)
    assert np.array_equal(acc.cpu().numpy(), A_ref)
    np.testing.assert_allclose(dX.cpu().numpy(), dX_ref, rtol=RTOL, atol=0)


def test_degenerate_layers(sq):
    rng = np.random.default_rng(2)
    W = (rng.standard_normal((40, 24)) * 0.02).astype(np.float32)
    X = rng.standard_normal((50, 24)).astype(np.float32)
    zeros = np.zeros((50, 40), np.float32)
    r = check_layer(sq, zeros, W, X, 4, 4)
    assert not r["dX"].any() and not r["dW"].any()
    nan = _grad(50, 40, seed=3)
    nan[3, 3] = np.nan
    r = check_layer(sq, nan, W, X, 6, 4)
    assert not r["dX"].any()
    Wz = np.zeros_like(W)
    check_layer(sq, _grad(50, 40, seed=4), Wz, X, 4, 4)


# ---------------------------------------------------------------------------
# The five layer workloads: reduced token counts (full oracle) ...
# ---------------------------------------------------------------------------
REDUCED = {"linear_256": 256, "resnet18_conv3x3": 3136, "resnet50_conv1x1": 1000,
           "mlp_up_768x3072": 600, "linear_4096x11008_sr": 200}


@pytest.mark.parametrize("name", workloads.WORKLOAD_ORDER)
def test_workload_reduced(sq, name):
    wl = workloads.WORKLOADS[name]
    d = workloads.make_inputs(name, M=REDUCED[name])
    M = d["M"]
    dgrad_rows = None
    wgrad_rows = None
    if wl.C_out * wl.C_in * M > 2e9:
        dgrad_rows = np.unique(np.r_[0, 1, M // 2, M - 2, M - 1, np.arange(64, M, 97)])
        rng = np.random.default_rng(1)
        wgrad_rows = np.unique(np.r_[0, wl.C_out - 1, rng.integers(0, wl.C_out, 24)])
    r = check_layer(sq, d["dY"], d["W"], d["X"], wl.bits, wl.num_groups, wl.round_mode, wl.sr_seed,
                    wl.sr_offset, dgrad_rows, wgrad_rows)
    assert r["exact_dX"] and r["exact_dW"]


# Parameter variants of the MLP layer (the bench's --bits / --num-groups /
# --rounding runs): b in {4, 6, 8}, N_G in 1..6, both rounding modes.
VARIANTS = [(b, g, 0) for b in (4, 6, 8) for g in range(1, 7)] + [(4, 4, 1), (6, 6, 1), (8, 3, 1), (8, 6, 1)]


@pytest.mark.parametrize("bits,ng,mode", VARIANTS, ids=[f"b{b}-ng{g}-{'sr' if m else 'rtn'}" for b, g, m in VARIANTS])
def test_parameter_variants(sq, bits, ng, mode):
    d = workloads.make_inputs("mlp_up_768x3072", M=600)
    M, C_out = d["M"], d["dY"].shape[1]
    rng = np.random.default_rng(bits * 10 + ng)
    dgrad_rows = np.unique(np.r_[0, M - 1, rng.integers(0, M, 12)])
    wgrad_rows = np.unique(np.r_[0, C_out - 1, rng.integers(0, C_out, 12)])
    r = check_layer(sq, d["dY"], d["W"], d["X"], bits, ng, mode, 3, 1, dgrad_rows, wgrad_rows)
    assert r["exact_dX"] and r["exact_dW"]


def test_parameter_variant_full_size(sq):
    # the widest variant the benchmark runs: 8-bit codes in 6 groups, full MLP layer
    d = workloads.make_inputs("mlp_up_768x3072")
    M, C_out = d["M"], d["dY"].shape[1]
    rng = np.random.default_rng(86)
    dgrad_rows = np.unique(np.r_[0, M - 1, rng.integers(0, M, 16)])
    wgrad_rows = np.unique(np.r_[0, C_out - 1, rng.integers(0, C_out, 8)])
    r = check_layer(sq, d["dY"], d["W"], d["X"], 8, 6, 0, 0, 0, dgrad_rows, wgrad_rows, fold_rows=dgrad_rows)
    assert r["exact_dX"] and r["exact_dW"]


# ... and full size, in the launch configuration the benchmark times, with
# every code compared and sampled GEMM rows computed by the oracle.
@pytest.mark.parametrize("name", workloads.WORKLOAD_ORDER)
def test_workload_full_size(sq, name):
    import torch
    wl = workloads.WORKLOADS[name]
    d = workloads.make_inputs(name)
    M, C_out, C_in = d["M"], wl.C_out, wl.C_in
    # the launch configuration bench.py times: tile-major code matrices
    print(f"[full-size parity] {name} M={M} C_out={C_out} C_in={C_in} (tile-major)", flush=True)
    p = sq.Params.make(wl.bits, wl.num_groups, wl.round_mode, wl.sr_seed, wl.sr_offset, sq.LAYOUT_TILED)
    plan = sq.BackwardPlan(M, C_out, C_in, p, want_acc=True)
    dY = _dev(d["dY"])
    wq_t, ws = sq.quantize_tensor(_dev(d["W"]), 8, tiled=True)
    xq_t, xs = sq.quantize_tensor(_dev(d["X"]), 8, tiled=True)
    plan.run(dY, wq_t, ws, xq_t, xs)
    torch.cuda.synchronize()

    q_ref, g_ref, s_ref, _ = oracle.quantize_grad(d["dY"], wl.bits, wl.num_groups, wl.round_mode,
                                                  wl.sr_seed, wl.sr_offset)
    q = sq.untile(plan.q_t)[:, :M].t().cpu().numpy()
    assert np.array_equal(plan.group.cpu().numpy(), g_ref)
    assert np.array_equal(q, q_ref)
    fold_rows = np.unique(np.r_[0, M - 1, np.random.default_rng(2).integers(0, M, 64)])
    check_fold(plan, q_ref, g_ref, wl.bits, wl.num_groups, fold_rows)
    wq_ref, ws_ref = oracle.quantize_tensor(d["W"], 8)
    xq_ref, xs_ref = oracle.quantize_tensor(d["X"], 8)
    assert np.array_equal(sq.untile(wq_t)[:, :C_out].t().cpu().numpy(), wq_ref)
    assert np.array_equal(sq.untile(xq_t)[:, :M].t().cpu().numpy(), xq_ref)

    # every row, except on the large linear layer (8192 x 11008 x 4096: 3.7e11
    # multiply-adds per product, minutes for the oracle): a quarter of the
    # input-gradient rows and a tenth of the weight-gradient rows, every tile
    # row boundary and every outlier channel among them
    oracle.set_threads(16)
    rng = np.random.default_rng(0)
    rows_d = np.arange(M)
    rows_w = np.arange(C_out)
    if M * C_out * C_in > 1e11:
        rows_d = np.unique(np.r_[0, M - 1, np.arange(255, M, 256), np.arange(256, M, 256), rng.integers(0, M, 2048)])
        outliers = np.nonzero(g_ref < wl.num_groups - 1)[0]
        rows_w = np.unique(np.r_[0, C_out - 1, outliers, np.arange(255, C_out, 256), np.arange(256, C_out, 256),
                                 rng.integers(0, C_out, 1024)])
    A_ref = oracle.dgrad(q_ref, g_ref, wl.num_groups, wq_ref, rows_d)
    B_ref = oracle.wgrad(q_ref, xq_ref, rows_w)
    dX_ref = oracle.dequant_dgrad(A_ref, s_ref["d0"], ws_ref["d0"], wl.num_groups)
    dW_ref = oracle.dequant_wgrad(B_ref, g_ref[rows_w], s_ref["d0"], xs_ref["d0"])
    rd = torch.as_tensor(rows_d, device="cuda")
    rw = torch.as_tensor(rows_w, device="cuda")
    assert np.array_equal(plan.acc_dX.index_select(0, rd).cpu().numpy(), A_ref)
    assert np.array_equal(plan.acc_dW.index_select(0, rw).cpu().numpy(), B_ref)
    np.testing.assert_allclose(plan.dX.index_select(0, rd).cpu().numpy(), dX_ref, rtol=RTOL, atol=0)
    np.testing.assert_allclose(plan.dW.index_select(0, rw).cpu().numpy(), dW_ref, rtol=RTOL, atol=0)
    assert np.array_equal(plan.dX.index_select(0, rd).cpu().numpy().view(np.uint32), dX_ref.view(np.uint32))
    assert np.array_equal(plan.dW.index_select(0, rw).cpu().numpy().view(np.uint32), dW_ref.view(np.uint32))
    # properties that hold at any size, checked on the whole outputs
    assert torch.isfinite(plan.dX).all() and torch.isfinite(plan.dW).all()
    assert sq.untile(plan.q_t)[:, :M].abs().max().item() == (1 << (wl.bits - 1)) - 1
