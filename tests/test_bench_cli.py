"""Host-side checks of bench.py's command line (no GPU needed)."""
import bench


def test_more_than_one_gpu_is_refused(capsys):
    assert bench.main(["--gpus", "2"]) == 2
    err = capsys.readouterr().err
    assert "one GPU only" in err and "--gpus 2" in err


def test_default_workload_is_the_large_linear_layer():
    # the largest configuration, the one the int8-peak figure is quoted on
    from paper_2411_10948_amd import workloads
    assert bench.DEFAULT_WORKLOAD == "linear_4096x11008_sr"
    wl = workloads.WORKLOADS[bench.DEFAULT_WORKLOAD]
    assert (wl.M, wl.C_out, wl.C_in, wl.bits, wl.round_mode) == (8192, 11008, 4096, 6, 1)
    assert bench.FUSED_CONV["resnet18_conv3x3_fused"] == "resnet18_conv3x3"


def test_summarize_steps():
    s = bench.summarize_steps([1.0, 2.0, 3.0, 4.0, 5.0], 4e9)
    assert s["median_ms"] == 3.0 and s["p10_ms"] < s["median_ms"] < s["p90_ms"]
    assert abs(s["value_at_median"] - 4e9 / 3e-3 / 1e12) < 1e-9
