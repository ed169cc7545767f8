"""sq_quantize_grad_noalloc (the gradient quantizer with the library's fixed
device scratch instead of a workspace) against sq_quantize_grad, through the
C-ABI: codes, transposed codes, groups, scale and fold layout bit for bit, on
two calls in a row, the second with a smaller gradient (the scratch keeps the
first call's contents).  Inputs are seeded and synthetic."""
import numpy as np
import pytest

from paper_2411_10948_amd import workloads

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sq():
    import torch
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    from paper_2411_10948_amd import shiftquant
    shiftquant.load()
    return shiftquant


def _outputs(sq, M, C, p, dev):
    import torch
    lay_bytes, min_ld = sq.sq_grad_layout_size(C, p)
    q_fold = torch.full((M, min_ld), 77, dtype=torch.int8, device=dev)
    q_t = torch.full((C, sq.round_up(M, 16)), 77, dtype=torch.int8, device=dev)
    group = torch.full((C,), 9, dtype=torch.uint8, device=dev)
    scale = sq.new_scale(dev)
    layout = torch.full((lay_bytes // 4,), -5, dtype=torch.int32, device=dev)
    return q_fold, q_t, group, scale, layout


def _both(sq, dY, p):
    import torch
    dev = dY.device
    M, C = dY.shape
    a = _outputs(sq, M, C, p, dev)
    b = _outputs(sq, M, C, p, dev)
    ws = torch.empty(max(sq.sq_quantize_grad_workspace_size(M, C, p), 256), dtype=torch.uint8, device=dev)
    sq.sq_quantize_grad(dY, p, *a, ws)
    sq.sq_quantize_grad_noalloc(dY, p, *b)
    torch.cuda.synchronize()
    for name, x, y in zip(("q_fold", "q_t", "group", "scale", "layout"), a, b):
        assert torch.equal(x, y), name
    return a


CASES = [  # (M, C), bits, N_G, rounding: the second call of each pair is smaller
    ((4096, 3072), (300, 200), 6, 4, 0),    # appended fold windows, ragged second call
    ((8192, 11008), (1000, 1100), 6, 4, 1),  # the large linear layer's gradient (stochastic rounding)
    ((5000, 64), (17, 5), 4, 4, 0),
]


@pytest.mark.parametrize("first,second,bits,ng,mode", CASES)
def test_noalloc_equals_workspace_entry(sq, first, second, bits, ng, mode):
    import torch
    print(f"[noalloc] {first} then {second} b={bits} N_G={ng} mode={mode}", flush=True)
    p = sq.Params.make(bits, ng, mode, 5, 11)
    for i, (M, C) in enumerate((first, second)):
        dY = workloads.make_grad(M, C, seed=M + C + i, sigma_s=2.0, outlier_frac=0.005, outlier_factor=1000.0)
        _both(sq, torch.from_numpy(dY).cuda(), p)
