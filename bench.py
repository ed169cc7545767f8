#!/usr/bin/env python3
"""Benchmark of the ShiftQuant backward step on one MI355X.

One step = sq_quantize_grad (dY -> codes, groups, scale) -> sq_gemm_dgrad
(fp32 dX) -> sq_gemm_wgrad (fp32 dW) on one stream, inputs resident in HBM.
W and X are quantized once, untimed: in training their codes come from the
forward pass.

Prints ONE JSON line.  `value` is whole-step throughput in TOPS, counting the
two integer GEMMs as 4 * M * C_out * C_in ops (quantizer element work is not
counted as ops).  `roofline` describes the step's dominant kernel, timed with
HIP events on the launch stream inside the timed region; `cpu_baseline` times
the CPU oracle on a bounded slice of the same workload.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0        # MI355X HBM3E
PEAK_INT8_TOPS = 5000.0      # MI355X dense int8 matrix-core peak
DEFAULT_WORKLOAD = "linear_4096x11008_sr"
SCRUB_BYTES = 512 << 20      # larger than the 256 MB last-level cache
# the same conv layer with the input gradient taken by the implicit-im2col
# conv dgrad (dX itself, NHWC, instead of the 9x larger im2col'd dX_col)
FUSED_CONV = {"resnet18_conv3x3_fused": "resnet18_conv3x3"}
KERNEL_SOURCES = ["paper_2411_10948_amd/csrc/sq_gemm.hip", "paper_2411_10948_amd/csrc/sq_quant.hip",
                  "paper_2411_10948_amd/csrc/sq_internal.h", "paper_2411_10948_amd/csrc/sq_abi.hip",
                  "paper_2411_10948_amd/build.py"]   # the compiler flags shape the kernels too


def _code_only(text: str) -> str:
    """C++ source without comments and blank lines (comments do not change the kernels)."""
    import re
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    lines = (re.sub(r"//.*$", "", line).rstrip() for line in text.splitlines())
    return "\n".join(line for line in lines if line)


def kernel_source_hash(read=None) -> str:
    """Hash of the kernel sources' code and of the build script (its flags
    shape the kernels too); read(rel) -> text overrides reading the files."""
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        if read is None:
            with open(os.path.join(ROOT, rel), encoding="utf-8") as f:
                text = f.read()
        else:
            text = read(rel)
        h.update((text if rel.endswith(".py") else _code_only(text)).encode())
    return h.hexdigest()[:16]


def measured_traffic(workload: str, kernel: str):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if it
    was taken on the current kernel sources (else None)."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    try:
        with open(path) as f:
            rec = json.load(f)
        ent = rec.get(workload, {}).get(kernel)
        if not ent or ent.get("kernel_source_hash") != kernel_source_hash():
            return None
        return ent.get("hbm_bytes_per_launch")
    except (OSError, ValueError):
        return None


def host_cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def host_threads() -> int:
    """Cores this process may use: OMP_NUM_THREADS when set (the GPU machine sets
    it to its CPU share), else the affinity mask."""
    env = os.environ.get("OMP_NUM_THREADS", "")
    if env.isdigit() and int(env) > 0:
        return int(env)
    return len(os.sched_getaffinity(0))


def cpu_baseline_one(inputs, wl, threads: int, budget_s: float, conv=False):
    """The CPU oracle (plain C; OpenMP over independent outputs) on the first
    rows of the same layer (whole images for the implicit-im2col conv step)."""
    import numpy as np
    import oracle
    oracle.set_threads(threads)
    dY, W, X = inputs["dY"], inputs["W"], inputs["X"]
    M = dY.shape[0]
    hw = wl.conv_hw * wl.conv_hw

    def run(rows):
        t0 = time.perf_counter()
        if conv:
            q, g, gs, _ = oracle.quantize_grad(dY[:rows], wl.bits, wl.num_groups, wl.round_mode, wl.sr_seed,
                                               wl.sr_offset)
            wq, ws = oracle.quantize_tensor(W, 8)
            xq, xs = oracle.quantize_tensor(X[:rows], 8)
            A = oracle.conv_dgrad(q, g, wl.num_groups, wq, rows // hw, wl.conv_hw, wl.conv_hw, 3, 3, 1, 1)
            # the layer input is the centre tap of the im2col'd rows (pad 1)
            xr = np.ascontiguousarray(xq[:, 4 * wl.conv_cin:5 * wl.conv_cin])
            B = oracle.conv_wgrad(q, xr, rows // hw, wl.conv_hw, wl.conv_hw, 3, 3, 1, 1)
            oracle.dequant_dgrad(A, gs["d0"], ws["d0"], wl.num_groups)
            oracle.dequant_wgrad(B, g, gs["d0"], xs["d0"])
        else:
            oracle.backward(dY[:rows], W, X[:rows], wl.bits, wl.num_groups, wl.round_mode, wl.sr_seed,
                            wl.sr_offset)
        return time.perf_counter() - t0

    unit = hw if conv else 1
    rows = max(unit, min(M, 8 if not conv else M // 256) // unit * unit)
    t = run(rows)
    if t < 0.5 * budget_s:
        rows = int(min(M, max(rows, rows * budget_s / max(t, 1e-3)))) // unit * unit
        t = run(rows)
    oracle.set_threads(1)
    ops = 4 * rows * wl.C_out * wl.C_in
    what = "quantize+conv dgrad+conv wgrad+dequant" if conv else "quantize+dgrad+wgrad+dequant"
    return {"value": ops / t / 1e12, "unit": "TOPS", "cores": threads, "kind": "oracle",
            "sample": f"oracle {what} on the first {rows} of {M} token rows "
                      f"({ops / 1e9:.2f} Gop in {t:.2f} s, {threads} thread{'s' if threads > 1 else ''})"}


def cpu_baseline(inputs, wl, conv=False):
    """All host cores (the reported figure) and one thread beside it."""
    n = host_threads()
    allc = cpu_baseline_one(inputs, wl, n, 8.0, conv)
    one = cpu_baseline_one(inputs, wl, 1, 8.0, conv) if n > 1 else dict(allc)
    allc["cpu_model"] = host_cpu_model()
    allc["single_thread"] = {"value": one["value"], "unit": "TOPS", "cores": 1, "sample": one["sample"]}
    return allc


def run_forward(args, torch, sq, wl, inputs):
    """Forward pass of the same layer (Sec. 5.1): X quantized with ShiftQuant
    (groups over its channels, the workload's b and N_G, round-half-even),
    W per output channel (8-bit, untimed: in training the weights change once
    per step), Y = X W^T as ShiftMM with per-column weight scales."""
    dev = torch.device("cuda:0")
    M, C_in, C_out = inputs["M"], wl.C_in, wl.C_out
    X = torch.from_numpy(inputs["X"]).to(dev)
    W = torch.from_numpy(inputs["W"]).to(dev)
    params = sq.Params.make(wl.bits, wl.num_groups, 0)
    wq, wsc = sq.quantize_channels(W, 8, 0, False)
    del W
    lay_bytes, min_ld = sq.sq_grad_layout_size(C_in, params)
    xq = torch.zeros((M, min_ld), dtype=torch.int8, device=dev)
    group = torch.empty(C_in, dtype=torch.uint8, device=dev)
    xscale = sq.new_scale(dev)
    layout = torch.zeros(lay_bytes // 4, dtype=torch.int32, device=dev)
    ws_q = torch.empty(max(sq.sq_quantize_grad_workspace_size(M, C_in, params), 256), dtype=torch.uint8, device=dev)
    ws_f = torch.empty(max(sq.sq_gemm_dgrad_workspace_size(M, C_in, C_out, params), 256), dtype=torch.uint8,
                       device=dev)
    Y = torch.empty((M, C_out), dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream()

    def quant():
        sq.sq_quantize_grad(X, params, xq, None, group, xscale, layout, ws_q, stream)

    def fwd():
        sq.sq_gemm_forward(xq, layout, group, xscale, wq, wsc, M, C_in, C_out, params, None, Y, ws_f, stream)

    def timed(fn, K):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record(stream)
        for _ in range(K):
            fn()
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) / K

    for _ in range(args.warmup):
        quant()
        fwd()
    step = lambda: (quant(), fwd())
    ms_step = timed(step, args.steps)
    t_q, t_f = timed(quant, args.steps), timed(fwd, args.steps)
    ops = 2 * M * C_in * C_out
    parts = {"sq_quantize_grad(X)": {"ms": t_q, "bytes": 5 * M * C_in, "ops": 0},
             "sq_gemm_forward": {"ms": t_f, "bytes": M * C_in + C_in * C_out + 4 * M * C_out, "ops": ops}}
    dom = max(parts, key=lambda k: parts[k]["ms"])
    d = parts[dom]
    if d["ops"] and d["ops"] / d["bytes"] > PEAK_INT8_TOPS * 1e12 / (PEAK_HBM_GBS * 1e9):
        roof = {"bound": "mfma", "achieved": d["ops"] / (d["ms"] * 1e-3) / 1e12, "peak": PEAK_INT8_TOPS,
                "unit": "TOPS"}
    else:
        roof = {"bound": "hbm", "achieved": d["bytes"] / (d["ms"] * 1e-3) / 1e9, "peak": PEAK_HBM_GBS, "unit": "GB/s"}
    roof.update({"frac": roof["achieved"] / roof["peak"], "traffic": None, "kernel": dom,
                 "algorithmic_bytes": d["bytes"], "algorithmic_ops": d["ops"], "avg_ms": d["ms"]})
    out = {"metric": "ShiftQuant forward TOPS (quantize X + ShiftMM forward GEMM)",
           "value": ops / (ms_step * 1e-3) / 1e12, "unit": "TOPS", "n_gpus": 1, "steps": args.steps,
           "warmup": args.warmup, "ms_per_step": ms_step, "higher_is_better": True, "scaling": "weak",
           "vs_baseline": None, "dtype": "int8", "data": "synthetic",
           "config": {"workload": args.workload, "step": "forward", "M": M, "C_in": C_in, "C_out": C_out,
                      "bits": wl.bits, "num_groups": wl.num_groups, "rounding": "nearest-even",
                      "weights": "8-bit per output channel", "parallelism": "none"},
           "breakdown_ms": {k: v["ms"] for k, v in parts.items()}, "roofline": roof}
    if not args.no_cpu_baseline:
        import numpy as np
        import oracle
        Xh, Wh = inputs["X"], inputs["W"]
        rows = max(1, min(M, 64))
        t0 = time.perf_counter()
        xq_o, g_o, xs_o, _ = oracle.quantize_grad(Xh[:rows], wl.bits, wl.num_groups)
        wq_o, wsc_o = oracle.quantize_channels(Wh, 8, 0)
        A_o = oracle.dgrad(xq_o, g_o, wl.num_groups, np.ascontiguousarray(wq_o.T))
        oracle.dequant_cols(A_o, xs_o["d0"], np.array([s["d0"] for s in wsc_o], np.float32), wl.num_groups)
        t = time.perf_counter() - t0
        out["cpu_baseline"] = {"value": 2 * rows * C_in * C_out / t / 1e12, "unit": "TOPS", "cores": 1,
                               "kind": "oracle", "sample": f"oracle quantize X + forward product + dequant on the "
                                                          f"first {rows} of {M} rows ({t:.2f} s, 1 thread)"}
    print(json.dumps(out), flush=True)
    return 0


def run_l1bn(args, torch, sq):
    """Fully-quantized L1 batch normalization (Sec. 4), one training step of
    the layer: the conv output X quantized to 8 bits per tensor, the L1BNQ
    forward, and the L1BNQ backward (ShiftQuant of dy, dx, dgamma, dbeta and
    the channel ranges of dx for the quantizer of the layer below).  HBM-bound:
    the figure of merit is algorithmic GB/s (X read 4 B, y written 4 B, dy read
    4 B, codes read 1 B, dx written 4 B per element)."""
    from paper_2411_10948_amd import workloads
    name = args.workload if args.workload in workloads.BN_WORKLOADS else "resnet18_bn_56x56x64"
    w = workloads.BN_WORKLOADS[name]
    inp = workloads.make_bn_inputs(name)
    M, C = w.M, w.C
    bits = args.bits or 8
    ng = args.num_groups or 4
    mode = int(args.rounding == "sr")
    print(f"[bench] {name}: M={M} C={C} gradient b={bits} N_G={ng} round={'SR' if mode else 'RTN'}",
          file=sys.stderr, flush=True)
    dev = torch.device("cuda:0")
    X = torch.from_numpy(inp["X"]).to(dev)
    gamma = torch.from_numpy(inp["gamma"]).to(dev)
    beta = torch.from_numpy(inp["beta"]).to(dev)
    dy = torch.from_numpy(inp["dy"]).to(dev)
    p = sq.Params.make(bits, ng, mode, 0, 0)
    ldx = sq.round_up(C, 16)
    xq = torch.zeros((M, ldx), dtype=torch.int8, device=dev)[:, :C]
    xs = sq.new_scale(dev)
    ws_x = torch.empty(max(sq.sq_quantize_tensor_workspace_size(M, C), 256), dtype=torch.uint8, device=dev)
    y = torch.empty((M, C), dtype=torch.float32, device=dev)
    chan = torch.zeros(C * sq.L1BN_CHANNEL_WORDS, dtype=torch.int32, device=dev)
    layer = torch.zeros(16, dtype=torch.int32, device=dev)
    ws_f = torch.empty(max(sq.sq_l1bn_forward_workspace_size(M, C), 256), dtype=torch.uint8, device=dev)
    dx = torch.empty((M, C), dtype=torch.float32, device=dev)
    dgamma = torch.empty(C, dtype=torch.float32, device=dev)
    dbeta = torch.empty(C, dtype=torch.float32, device=dev)
    group = torch.empty(C, dtype=torch.uint8, device=dev)
    gscale = sq.new_scale(dev)
    ranges = torch.empty((sq.sq_l1bn_range_slabs(M, C), C), dtype=torch.int32, device=dev)
    ws_b = torch.empty(sq.sq_l1bn_backward_workspace_size(M, C, p), dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream()

    def quant():
        sq.sq_quantize_tensor(X, 8, False, xq, xs, ws_x, stream)

    def fwd():
        sq.sq_l1bn_forward(xq, xs, gamma, beta, y, chan, layer, ws_f, stream)

    def bwd():
        sq.sq_l1bn_backward(dy, p, xq, chan, layer, dx, dgamma, dbeta, group, gscale, ranges, ws_b, stream)

    def step():
        quant()
        fwd()
        bwd()

    def timed(fn, K):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record(stream)
        for _ in range(K):
            fn()
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) / K

    for _ in range(args.warmup):
        step()
    ms_step = timed(step, args.steps)
    parts = {"sq_quantize_tensor(X)": {"ms": timed(quant, args.steps), "bytes": 5 * M * C},
             "sq_l1bn_forward": {"ms": timed(fwd, args.steps), "bytes": 5 * M * C},
             "sq_l1bn_backward": {"ms": timed(bwd, args.steps), "bytes": 9 * M * C}}
    total_bytes = 17 * M * C
    dom = max(parts, key=lambda k: parts[k]["ms"])
    d = parts[dom]
    roof = {"bound": "hbm", "achieved": d["bytes"] / (d["ms"] * 1e-3) / 1e9, "peak": PEAK_HBM_GBS, "unit": "GB/s"}
    roof.update({"frac": roof["achieved"] / roof["peak"], "traffic": None, "kernel": dom,
                 "algorithmic_bytes": d["bytes"], "algorithmic_ops": 0, "avg_ms": d["ms"]})
    value = total_bytes / (ms_step * 1e-3) / 1e9
    out = {"metric": "L1BNQ training step (quantize X + forward + backward) algorithmic GB/s",
           "value": value, "unit": "GB/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
           "ms_per_step": ms_step, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
           "dtype": "int8", "data": "synthetic",
           "config": {"workload": name, "step": "l1bn", "M": M, "C": C, "input_bits": 8, "grad_bits": bits,
                      "num_groups": ng, "rounding": "stochastic" if mode else "nearest-even", "parallelism": "none"},
           "pct_hbm_peak": 100.0 * value / PEAK_HBM_GBS,
           "breakdown_ms": {k: v["ms"] for k, v in parts.items()}, "roofline": roof}
    if not args.no_cpu_baseline:
        import oracle
        rows = min(M, 1 << 18)
        Xh, dyh = inp["X"][:rows], inp["dy"][:rows]
        t0 = time.perf_counter()
        xq_o, xs_o = oracle.quantize_tensor(Xh, 8)
        f = oracle.l1bn_forward(xq_o, xs_o["d0"], inp["gamma"], inp["beta"])
        oracle.l1bn_backward(dyh, f, xq_o, bits, ng, mode)
        t = time.perf_counter() - t0
        out["cpu_baseline"] = {"value": 17 * rows * C / t / 1e9, "unit": "GB/s", "cores": 1, "kind": "oracle",
                               "sample": f"oracle quantize X + L1BNQ forward + backward on the first {rows} of {M} "
                                         f"rows ({t:.2f} s, 1 thread)"}
    print(json.dumps(out), flush=True)
    return 0


def run_chain(args, torch, sq):
    """Two layers of the Transformer MLP backward in sequence: the
    down-projection (3072 -> 768) and then the up-projection (768 -> 3072),
    whose output gradient is the down-projection's input gradient.  With
    --fused-ranges the down-projection's dgrad also writes the channel ranges
    of its dX and the up-projection's quantizer takes them instead of reading
    dX once more for its abs-max; otherwise both quantizers run in full."""
    from paper_2411_10948_amd import workloads
    inp = workloads.make_chain_inputs()
    M, d, f = inp["M"], inp["d_model"], inp["d_ff"]
    dev = torch.device("cuda:0")
    p = sq.Params.make(inp["bits"], inp["num_groups"], 0)
    dY = torch.from_numpy(inp["dY_dn"]).to(dev)
    wdn_t, wdn_s = sq.quantize_tensor(torch.from_numpy(inp["W_dn"]).to(dev), 8, transpose=True)
    xdn_t, xdn_s = sq.quantize_tensor(torch.from_numpy(inp["X_dn"]).to(dev), 8, transpose=True)
    wup_t, wup_s = sq.quantize_tensor(torch.from_numpy(inp["W_up"]).to(dev), 8, transpose=True)
    xup_t, xup_s = sq.quantize_tensor(torch.from_numpy(inp["X_up"]).to(dev), 8, transpose=True)
    fused = args.fused_ranges
    dn = sq.BackwardPlan(M, d, f, p, device=dev, dx_ranges=fused)
    up = sq.BackwardPlan(M, f, d, p, device=dev)
    stream = torch.cuda.current_stream()

    def step():
        dn.run(dY, wdn_t, wdn_s, xdn_t, xdn_s, stream)
        if fused:
            up.quantize_from_ranges(dn.dX, dn.dX_ranges, stream)
        else:
            up.quantize(dn.dX, stream)
        up.dgrad(wup_t, wup_s, stream)
        up.wgrad(xup_t, xup_s, stream)

    def timed(fn, K):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record(stream)
        for _ in range(K):
            fn()
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) / K

    for _ in range(args.warmup):
        step()
    ms = timed(step, args.steps)
    t_qup = timed((lambda: up.quantize_from_ranges(dn.dX, dn.dX_ranges, stream)) if fused
                  else (lambda: up.quantize(dn.dX, stream)), args.steps)
    t_dgdn = timed(lambda: dn.dgrad(wdn_t, wdn_s, stream), args.steps)
    ops = 2 * 4 * M * d * f
    alg_q = 5 * M * f
    out = {"metric": "ShiftQuant backward TOPS (quantize+dgrad+wgrad) and % of int8 MFMA peak",
           "value": ops / (ms * 1e-3) / 1e12, "unit": "TOPS", "n_gpus": 1, "steps": args.steps,
           "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
           "vs_baseline": None, "dtype": "int8", "data": "synthetic",
           "config": {"workload": "mlp_chain_down_up_768x3072", "step": "chain", "M": M, "d_model": d, "d_ff": f,
                      "bits": inp["bits"], "num_groups": inp["num_groups"], "rounding": "nearest-even",
                      "up_proj_ranges": "from the down-projection's dgrad epilogue" if fused else "abs-max pass",
                      "parallelism": "none"},
           "breakdown_ms": {"up-projection quantize": t_qup, "down-projection dgrad": t_dgdn},
           "up_quantize_gbs": alg_q / (t_qup * 1e-3) / 1e9,
           "up_quantize_frac_hbm": alg_q / (t_qup * 1e-3) / 1e9 / PEAK_HBM_GBS}
    print(json.dumps(out), flush=True)
    return 0


def per_step_times(torch, stream, step, K):
    """K steps, each bracketed by its own event pair on the launch stream.
    Before each, outside the events, a 512 MB write evicts the last-level
    cache, so no step finds its inputs cache-resident."""
    scrub = torch.empty(SCRUB_BYTES // 4, dtype=torch.float32, device="cuda")
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(K)]
    torch.cuda.synchronize()
    for k in range(K):
        scrub.fill_(float(k))
        ev[k][0].record(stream)
        step()
        ev[k][1].record(stream)
    torch.cuda.synchronize()
    del scrub
    return [a.elapsed_time(b) for a, b in ev]


def summarize_steps(times, ops):
    import numpy as np
    t = np.asarray(times, np.float64)
    med = float(np.median(t))
    return {"mode": "event pair per step, 512 MB cache scrub before each (outside the events)",
            "scrub_bytes": SCRUB_BYTES, "steps": len(times), "median_ms": med,
            "p10_ms": float(np.percentile(t, 10)), "p90_ms": float(np.percentile(t, 90)),
            "value_at_median": ops / (med * 1e-3) / 1e12}


def run_conv_chain(args, torch, sq):
    """Two ResNet-18 stage-1 conv layers backward in sequence (64 x 56 x 56,
    64 -> 64 channels, 3x3, pad 1, 4-bit gradients): the upper layer's input
    gradient is the lower layer's output gradient.  With --fused-ranges the
    upper layer's conv dgrad also writes the channel ranges of its dX and the
    lower layer's quantizer takes them instead of its own abs-max pass over dX."""
    import numpy as np
    from paper_2411_10948_amd import workloads
    d = workloads.make_inputs("resnet18_conv3x3")
    wl = d["workload"]
    N, H, W, C = 64, 56, 56, 64
    dev = torch.device("cuda:0")
    p = sq.Params.make(wl.bits, wl.num_groups, wl.round_mode)
    dY = torch.from_numpy(d["dY"]).to(dev)
    W2 = torch.from_numpy(d["W"]).to(dev)
    W1 = torch.flip(W2, dims=(0,)).contiguous()      # a second layer's weights (same distribution)
    w2_t, w2_s = sq.quantize_tensor(W2, 8, transpose=True)
    w1_t, w1_s = sq.quantize_tensor(W1, 8, transpose=True)
    Xc = torch.from_numpy(np.ascontiguousarray(d["X"][:, 4 * C:5 * C])).to(dev)
    xq_raw, xs = sq.quantize_tensor(Xc, 8, transpose=True)
    del W1, W2
    fused = args.fused_ranges
    packed = args.conv_input == "pack"
    up = sq.ConvBackwardPlan(N, H, W, C, C, 3, 3, 1, 1, p, device=dev, dx_ranges=fused)
    lo = sq.ConvBackwardPlan(N, H, W, C, C, 3, 3, 1, 1, p, device=dev)
    stream = torch.cuda.current_stream()
    if not packed:
        # the forward pass's input quantizer writes each layer's grid
        up.quantize_input(Xc, stream)
        lo.quantize_input(Xc, stream)
    del Xc

    def quant_lo():
        if fused:
            lo.quantize_from_ranges(up.dX, up.dX_ranges, stream, range_slabs=up.range_slabs)
        else:
            lo.quantize(up.dX, stream)

    def step():
        # --conv-input pack: each layer packs its input codes onto its grid
        if packed:
            up.run_packed(dY, w2_t, w2_s, xq_raw, xs, stream)
        else:
            up.run(dY, w2_t, w2_s, up.x_grid, up.x_scale, stream)
        quant_lo()
        lo.dgrad(w1_t, w1_s, stream)
        if packed:
            lo.pack_input(xq_raw, stream)
        lo.wgrad(lo.x_grid, xs if packed else lo.x_scale, stream)

    def timed(fn, K):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record(stream)
        for _ in range(K):
            fn()
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) / K

    for _ in range(args.warmup):
        step()
    ms = timed(step, args.steps)
    ops = 2 * 4 * (N * H * W) * C * 9 * C
    out = {"metric": "ShiftQuant backward TOPS (quantize+dgrad+wgrad) and % of int8 MFMA peak",
           "value": ops / (ms * 1e-3) / 1e12, "unit": "TOPS", "n_gpus": 1, "steps": args.steps,
           "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
           "vs_baseline": None, "dtype": "int8", "data": "synthetic",
           "config": {"workload": "resnet18_conv3x3_chain", "step": "conv_chain", "layers": 2, "N": N, "H": H,
                      "W": W, "C": C, "bits": wl.bits, "num_groups": wl.num_groups, "rounding": "nearest-even",
                      "lower_quantizer_ranges": "from the upper layer's conv dgrad" if fused else "abs-max pass",
                      "conv_input_codes": "packed in the step" if packed else "on the grid from the forward quantizer",
                      "parallelism": "none"},
           "breakdown_ms": {"upper conv dgrad": timed(lambda: up.dgrad(w2_t, w2_s, stream), args.steps),
                            "lower quantize": timed(quant_lo, args.steps)}}
    print(json.dumps(out), flush=True)
    return 0


def run_vendor_gemm(args, torch, wl, M):
    """The vendor library's GEMMs on the layer's two backward product shapes,
    for comparison with the ShiftQuant GEMMs: dX = dY W as [M, C_out] x
    [C_out, C_in] and dW = dY^T X as [C_out, M] x [M, C_in], second operand
    column-major (its faster layout), in int8 (torch._int_mm, int32 output)
    and, as the paper's floating-point comparison point, in fp16 and bf16
    (torch.matmul, output in the same type).  Warm, back-to-back launches;
    random codes in [-31, 31] (the same values in every type)."""
    dev = torch.device("cuda:0")
    g = torch.Generator(device=dev)
    g.manual_seed(0)
    shapes = {"dgrad": (M, wl.C_out, wl.C_in), "wgrad": (wl.C_out, M, wl.C_in)}

    def timed(fn):
        for _ in range(args.warmup):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(args.steps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / args.steps

    out = {}
    for name, (m, k, n) in shapes.items():
        a = torch.randint(-31, 32, (m, k), dtype=torch.int8, device=dev, generator=g)
        b = torch.randint(-31, 32, (n, k), dtype=torch.int8, device=dev, generator=g)
        ops = 2.0 * m * n * k
        res = {"shape_mkn": [m, k, n]}
        ms = timed(lambda: torch._int_mm(a, b.t()))
        res["int8"] = {"ms": ms, "TOPS": ops / ms / 1e9}
        for tname, dt in (("fp16", torch.float16), ("bf16", torch.bfloat16)):
            af, bf = a.to(dt), b.to(dt)
            ms = timed(lambda: torch.matmul(af, bf.t()))
            res[tname] = {"ms": ms, "TFLOPS": ops / ms / 1e9}
            del af, bf
        out[name] = res
        del a, b
    ops = 4.0 * M * wl.C_out * wl.C_in
    tot = {t: sum(v[t]["ms"] for v in out.values()) for t in ("int8", "fp16", "bf16")}
    print(json.dumps({"metric": "vendor int8 GEMM (torch._int_mm) TOPS on the backward product shapes",
                      "value": ops / tot["int8"] / 1e9, "unit": "TOPS", "n_gpus": 1, "steps": args.steps,
                      "warmup": args.warmup, "ms_per_step": tot["int8"], "higher_is_better": True, "dtype": "int8",
                      "data": "synthetic", "config": {"workload": wl.name, "M": M, "C_out": wl.C_out,
                                                      "C_in": wl.C_in, "library": "hipBLASLt via torch"},
                      "fp16_ms_per_step": tot["fp16"], "fp16_TFLOPS": ops / tot["fp16"] / 1e9,
                      "bf16_ms_per_step": tot["bf16"], "bf16_TFLOPS": ops / tot["bf16"] / 1e9,
                      "per_product": out, "pct_int8_peak": 100.0 * ops / tot["int8"] / 1e9 / PEAK_INT8_TOPS}))
    return 0


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--bits", type=int, default=None, help="override the workload's gradient bits (variant runs)")
    ap.add_argument("--num-groups", type=int, default=None, help="override the workload's N_G (variant runs)")
    ap.add_argument("--rounding", choices=["rtn", "sr"], default=None,
                    help="override the workload's rounding (variant runs)")
    ap.add_argument("--fused-ranges", action="store_true",
                    help="--step chain / conv_chain: the upper layer's dgrad writes the lower quantizer's ranges")
    ap.add_argument("--step", choices=["backward", "forward", "l1bn", "chain", "conv_chain", "vendor_gemm"],
                    default="backward",
                    help="forward: quantize X with ShiftQuant + Y = X W^T (per-output-channel W); "
                         "vendor_gemm: the vendor int8, fp16 and bf16 GEMMs on the linear layer's two backward product shapes; "
                         "l1bn: the L1BNQ layer (workloads resnet18_bn_56x56x64, resnet50_bn_14x14x1024, "
                         "transformer_bn_768)")
    ap.add_argument("--conv-wgrad", choices=["implicit", "im2col"], default="implicit",
                    help="weight gradient of the fused conv step: implicit im2col (sq_conv_wgrad) or the GEMM on "
                         "the im2col'd activations")
    ap.add_argument("--conv-input", choices=["grid", "pack"], default="grid",
                    help="input codes of the implicit conv wgrad: written onto the padded grid by the forward "
                         "pass's quantizer (sq_quantize_input_conv, untimed like the rest of the forward), or "
                         "packed from sq_quantize_tensor's codes inside the timed step (sq_conv_pack_input)")
    ap.add_argument("--layout", choices=["tiled", "rows"], default="tiled",
                    help="code matrices of the linear layers: tile-major (default) or row-major")
    ap.add_argument("--dgrad", choices=["shiftmm", "grouped"], default="shiftmm",
                    help="grouped: the GEMM-based comparison implementation of the dgrad (Sec. 3.2)")
    ap.add_argument("--graph", action="store_true",
                    help="also time the step captured as a HIP graph and replayed (reported under 'graph')")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="run one 256 MiB device-to-device copy first (reference for HBM byte counters)")
    args = ap.parse_args(argv)
    if args.gpus != 1:
        print(f"bench.py: measures one GPU only; --gpus {args.gpus} is not supported "
              "(the ShiftQuant path runs on one GPU; sharding over tokens is not built)", file=sys.stderr)
        return 2

    import torch
    from paper_2411_10948_amd import shiftquant as sq
    from paper_2411_10948_amd import workloads

    if not os.path.exists(sq.LIB_PATH):
        from paper_2411_10948_amd import build
        build.build()
    sq.load()
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    if args.step == "l1bn":
        return run_l1bn(args, torch, sq)
    if args.step == "chain":
        return run_chain(args, torch, sq)
    if args.step == "conv_chain":
        return run_conv_chain(args, torch, sq)
    conv = args.workload in FUSED_CONV
    wl = workloads.WORKLOADS[FUSED_CONV.get(args.workload, args.workload)]
    # parameter variants of the same layer (same tensors, other b / N_G / rounding)
    import dataclasses
    over = {k: v for k, v in (("bits", args.bits), ("num_groups", args.num_groups),
                                ("round_mode", None if args.rounding is None else int(args.rounding == "sr")))
            if v is not None}
    wl = dataclasses.replace(wl, **over)
    inputs = workloads.make_inputs(wl.name)
    M, C_out, C_in = inputs["M"], wl.C_out, wl.C_in
    print(f"[bench] {args.workload}: M={M} C_out={C_out} C_in={C_in} b={wl.bits} N_G={wl.num_groups} "
          f"round={'SR' if wl.round_mode else 'RTN'}", file=sys.stderr, flush=True)

    if args.step == "vendor_gemm":
        if conv:
            print("bench.py: --step vendor_gemm takes a linear workload", file=sys.stderr)
            return 2
        return run_vendor_gemm(args, torch, wl, M)

    if args.step == "forward":
        if conv or wl.x_kind == "conv3x3_relu":
            print("bench.py: --step forward runs the linear layers (the conv layers' inputs are im2col'd)",
                  file=sys.stderr)
            return 2
        return run_forward(args, torch, sq, wl, inputs)

    dev = torch.device("cuda:0")
    dY = torch.from_numpy(inputs["dY"]).to(dev)
    W = torch.from_numpy(inputs["W"]).to(dev)
    X = torch.from_numpy(inputs["X"]).to(dev)
    # linear layers: tile-major code matrices (the GEMMs' K tiles are then
    # contiguous 1 KB blocks); the conv kernels take row-major codes
    tiled = not conv and args.dgrad == "shiftmm" and args.layout == "tiled"
    params = sq.Params.make(wl.bits, wl.num_groups, wl.round_mode, wl.sr_seed, wl.sr_offset,
                            sq.LAYOUT_TILED if tiled else sq.LAYOUT_ROWS)
    wq_t, ws = sq.quantize_tensor(W, 8, transpose=True, tiled=tiled)
    implicit = conv and args.conv_wgrad == "implicit"
    packed = implicit and args.conv_input == "pack"
    if implicit:
        # the layer input is the centre tap of the im2col'd rows (pad 1); its
        # per-tensor scale equals the im2col'd tensor's (the im2col adds only
        # zeros).  Its codes come from the forward pass: written onto the
        # padded grid by the input quantizer (--conv-input grid), or as
        # sq_quantize_tensor codes that the timed step packs (run_packed).
        X = X[:, 4 * wl.conv_cin:5 * wl.conv_cin].contiguous()
        xq_t, xs = sq.quantize_tensor(X, 8, transpose=True) if packed else (None, None)
    else:
        xq_t, xs = sq.quantize_tensor(X, 8, transpose=True, tiled=tiled)
    del W
    if conv:
        n_img = M // (wl.conv_hw * wl.conv_hw)
        plan = sq.ConvBackwardPlan(n_img, wl.conv_hw, wl.conv_hw, C_out, wl.conv_cin, 3, 3, 1, 1, params, device=dev,
                                   implicit_wgrad=implicit)
    else:
        plan = sq.BackwardPlan(M, C_out, C_in, params, device=dev, grouped_dgrad=args.dgrad == "grouped")
    stream = torch.cuda.current_stream()
    if implicit and not packed:
        plan.quantize_input(X, stream)     # the forward pass's quantizer of the layer input
        xq_t, xs = plan.x_grid, plan.x_scale
    else:
        del X
    if args.calibrate_copy:
        src = torch.empty(64 << 20, dtype=torch.float32, device=dev).fill_(1.0)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)        # reads and writes exactly 256 MiB
        torch.cuda.synchronize()
        del src, dst

    run = plan.run_packed if packed else plan.run
    for _ in range(args.warmup):
        run(dY, wq_t, ws, xq_t, xs, stream)
    torch.cuda.synchronize()

    K = args.steps
    per_step = per_step_times(torch, stream, lambda: run(dY, wq_t, ws, xq_t, xs, stream), K)
    # Timed region: K whole steps on one stream, bracketed by two events only
    # (an event recorded between kernels costs a bubble of several us).
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    for _ in range(K):
        run(dY, wq_t, ws, xq_t, xs, stream)
    stop.record(stream)
    torch.cuda.synchronize()
    ms_step = start.elapsed_time(stop) / K

    graph = None
    if args.graph:
        # the same step captured once as a HIP graph (the library allocates,
        # clears and synchronizes nothing, so a step is capturable) and
        # replayed K times between two events: the same kernels, launched by
        # the runtime as one graph instead of one call at a time
        cs = torch.cuda.Stream()
        cs.wait_stream(stream)
        with torch.cuda.stream(cs):
            run(dY, wq_t, ws, xq_t, xs, cs)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=cs):
            run(dY, wq_t, ws, xq_t, xs, cs)
        torch.cuda.synchronize()
        for _ in range(args.warmup):
            g.replay()
        torch.cuda.synchronize()
        start.record(stream)
        for _ in range(K):
            g.replay()
        stop.record(stream)
        torch.cuda.synchronize()
        ms_graph = start.elapsed_time(stop) / K
        graph = {"ms_per_step": ms_graph, "value": 4 * M * C_out * C_in / (ms_graph * 1e-3) / 1e12,
                 "mode": "one step captured as a HIP graph, replayed K times between two events"}
        del g

    # Per-call averages: each call launched K times back to back between two
    # events on the same stream (the kernels of the dominant call are what the
    # roofline entry reports).
    def per_call(fn):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record(stream)
        for _ in range(K):
            fn()
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) / K

    t_quant = per_call(lambda: plan.quantize(dY, stream))
    t_dgrad = per_call(lambda: plan.dgrad(wq_t, ws, stream))
    if packed:
        t_pack = per_call(lambda: plan.pack_input(xq_t, stream))
        t_wgrad = per_call(lambda: plan.wgrad(plan.x_grid, xs, stream))
    elif implicit:
        t_wgrad = per_call(lambda: plan.wgrad(plan.x_grid, xs, stream))
    else:
        t_wgrad = per_call(lambda: plan.wgrad(xq_t, xs, stream))
    forward_ms = {}
    if implicit and not packed:
        # outside the step: the forward pass's input quantizer, for the record
        forward_ms["sq_quantize_input_conv"] = per_call(lambda: plan.quantize_input(X, stream))
        del X
    ops = 4 * M * C_out * C_in
    value = ops / (ms_step * 1e-3) / 1e12

    # algorithmic bytes / ops per launch (int8 operands read once, outputs written once)
    parts = {
        "sq_quantize_grad": {"ms": t_quant, "bytes": 5 * M * C_out, "ops": 0},
        # the conv dgrad writes dX [N*H*W, C_in / 9] (stride 1, same padding: N*H*W = M)
        "sq_conv_dgrad" if conv else "sq_gemm_dgrad": {
            "ms": t_dgrad, "bytes": M * C_out + C_out * C_in + 4 * M * (C_in // 9 if conv else C_in),
            "ops": 2 * M * C_out * C_in},
        # the implicit conv wgrad reads the layer input [N*H*W, C_in / 9] once
        "sq_conv_wgrad" if implicit else "sq_gemm_wgrad": {
            "ms": t_wgrad, "bytes": M * C_out + M * (C_in // 9 if implicit else C_in) + 4 * C_out * C_in,
            "ops": 2 * M * C_out * C_in},
    }
    if packed:
        # the input codes [C_in / 9, N*H*W] read, the padded grid written
        parts["sq_conv_pack_input"] = {"ms": t_pack, "bytes": M * (C_in // 9) + plan.x_grid.numel(), "ops": 0}
    dom = max(parts, key=lambda k: parts[k]["ms"])
    d = parts[dom]
    balance = PEAK_INT8_TOPS * 1e12 / (PEAK_HBM_GBS * 1e9)
    if d["ops"] and d["ops"] / d["bytes"] > balance:
        achieved = d["ops"] / (d["ms"] * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": achieved, "peak": PEAK_INT8_TOPS, "unit": "TOPS"}
    else:
        achieved = d["bytes"] / (d["ms"] * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s"}
    roof["frac"] = roof["achieved"] / roof["peak"]
    roof["traffic"] = measured_traffic(args.workload, dom)
    roof["kernel"] = dom
    roof["algorithmic_bytes"] = d["bytes"]
    roof["algorithmic_ops"] = d["ops"]
    roof["avg_ms"] = d["ms"]

    out = {
        "metric": "ShiftQuant backward TOPS (quantize+dgrad+wgrad) and % of int8 MFMA peak",
        "value": value,
        "unit": "TOPS",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int8",
        "data": "synthetic",
        "config": {"workload": args.workload, "M": M, "C_out": C_out, "C_in": C_in, "bits": wl.bits,
                   "num_groups": wl.num_groups, "rounding": "stochastic" if wl.round_mode else "nearest-even",
                   "dgrad_output": "dX [N,H,W,C] (implicit im2col + col2im)" if conv else "dX_col [M, C_in]",
                   "dgrad_impl": "shiftmm" if conv else args.dgrad,
                   "wgrad_impl": ("implicit im2col (sq_conv_wgrad)" if implicit else "GEMM on im2col'd X")
                   if conv else "gemm",
                   **({"conv_input_codes": "packed in the step (sq_conv_pack_input)" if packed else
                       "on the padded grid from the forward quantizer (sq_quantize_input_conv)"}
                      if implicit else {}),
                   "code_layout": "tile-major" if tiled else "row-major",
                   "parallelism": "none"},
        "pct_int8_peak": 100.0 * value / PEAK_INT8_TOPS,
        "breakdown_ms": {k: v["ms"] for k, v in parts.items()},
        **({"forward_ms": forward_ms} if forward_ms else {}),
        **({"graph": graph} if graph else {}),
        "roofline": roof,
        "per_step": summarize_steps(per_step, ops),
    }
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle on a slice of the workload", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(inputs, wl, conv=conv)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
