"""Host-side checks of bench.py's command line (no GPU needed)."""
import bench


def test_more_than_one_gpu_is_refused(capsys):
    assert bench.main(["--gpus", "2"]) == 2
    err = capsys.readouterr().err
    assert "one GPU only" in err and "--gpus 2" in err


def test_default_workload_is_the_fused_resnet18_conv():
    assert bench.DEFAULT_WORKLOAD == "resnet18_conv3x3_fused"
    assert bench.FUSED_CONV[bench.DEFAULT_WORKLOAD] == "resnet18_conv3x3"
