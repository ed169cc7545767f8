"""A whole backward step captured as a HIP graph and replayed: the library
allocates, clears and synchronizes nothing inside a call, so a step is
capturable.  Each replay, with eager work and synchronizations between the
replays and the outputs overwritten before each, must reproduce the eager
step bit for bit (codes, groups, scale, layout, dX, dW)."""
import numpy as np
import pytest

from paper_2411_10948_amd import workloads
from tests.test_gpu_parity import _dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sq():
    import torch
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    from paper_2411_10948_amd import shiftquant
    shiftquant.load()
    return shiftquant


def _outputs(plan):
    return [plan.q_fold, plan.group, plan.scale, plan.layout, plan.dX, plan.dW] + \
           ([plan.q_t] if getattr(plan, "q_t", None) is not None else []) + \
           ([plan.q_tp] if getattr(plan, "q_tp", None) is not None else [])


def _replay_and_check(sq, plan, step, other):
    import torch
    ref = [t.clone() for t in _outputs(plan)]
    cs = torch.cuda.Stream()
    cs.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(cs):
        step(cs)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=cs):
        step(cs)
    torch.cuda.synchronize()
    for r in range(3):
        # eager work of the program between replays; then NaN in dX and dW and
        # garbage in the groups and scale, which every step rewrites, and the
        # code and layout buffers back to zeros (their state before a first
        # call: padding that the quantizer never writes stays zero)
        other()
        torch.cuda.synchronize()
        plan.dX.fill_(float("nan"))
        plan.dW.fill_(float("nan"))
        plan.group.fill_(251)
        plan.scale.fill_(-3)
        for t in _outputs(plan)[6:] + [plan.q_fold, plan.layout]:
            t.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for i, (a, b) in enumerate(zip(_outputs(plan), ref)):
            assert torch.equal(a.view(torch.uint8) if a.dtype == torch.float32 else a,
                               b.view(torch.uint8) if b.dtype == torch.float32 else b), f"replay {r}, output {i}"
    del g


@pytest.mark.parametrize("layout", ["tiled", "rows"])
def test_linear_step_graph_replay(sq, layout):
    # appended fold windows (b = 6, N_G = 4), stochastic rounding, split-K wgrad
    import torch
    print(f"[graph] linear step, {layout} codes", flush=True)
    M, C_out, C_in = 4096, 1100, 300
    dY = workloads.make_grad(M, C_out, seed=5, sigma_s=2.0, outlier_frac=0.005, outlier_factor=1000.0)
    rng = np.random.default_rng(6)
    W = (rng.standard_normal((C_out, C_in)) * 0.05).astype(np.float32)
    X = np.maximum(rng.standard_normal((M, C_in)), 0.0).astype(np.float32)
    tiled = layout == "tiled"
    p = sq.Params.make(6, 4, 1, 9, 3, sq.LAYOUT_TILED if tiled else sq.LAYOUT_ROWS)
    plan = sq.BackwardPlan(M, C_out, C_in, p)
    wq, ws = sq.quantize_tensor(_dev(W), 8, transpose=True, tiled=tiled)
    xq, xs = sq.quantize_tensor(_dev(X), 8, transpose=True, tiled=tiled)
    dYd = _dev(dY)
    plan.run(dYd, wq, ws, xq, xs)
    torch.cuda.synchronize()
    other_plan = sq.BackwardPlan(M, C_out, C_in, p)
    dY2 = dYd * 0.5
    _replay_and_check(sq, plan, lambda st: plan.run(dYd, wq, ws, xq, xs, st),
                      lambda: other_plan.run(dY2, wq, ws, xq, xs))


def test_conv_step_graph_replay(sq):
    import torch
    print("[graph] conv step", flush=True)
    N, H, W, C = 2, 12, 16, 64
    rng = np.random.default_rng(8)
    dY = workloads.make_grad(N * H * W, C, seed=7, sigma_s=2.0, outlier_frac=0.005, outlier_factor=1000.0)
    X = np.maximum(rng.standard_normal((N * H * W, C)), 0.0).astype(np.float32)
    Wt = (rng.standard_normal((C, 9 * C)) * 0.05).astype(np.float32)
    p = sq.Params.make(4, 4, 0)
    plan = sq.ConvBackwardPlan(N, H, W, C, C, 3, 3, 1, 1, p)
    wq, ws = sq.quantize_tensor(_dev(Wt), 8, transpose=True)
    plan.quantize_input(_dev(X))
    dYd = _dev(dY)
    plan.run(dYd, wq, ws, plan.x_grid, plan.x_scale)
    torch.cuda.synchronize()
    other = sq.ConvBackwardPlan(N, H, W, C, C, 3, 3, 1, 1, p)
    other.quantize_input(_dev(X))
    dY2 = dYd * 2.0
    _replay_and_check(sq, plan, lambda st: plan.run(dYd, wq, ws, plan.x_grid, plan.x_scale, st),
                      lambda: other.run(dY2, wq, ws, other.x_grid, other.x_scale))
