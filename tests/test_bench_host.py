"""Host logic of bench.py (no GPU): the one-GPU refusal, the argument
defaults, and the rule that measured HBM traffic is reported only while the
counter runs' recorded kernel source matches the current one."""
import os
import shutil

import pytest

import bench


def test_more_than_one_gpu_is_refused(capsys):
    assert bench.main(["--gpus", "2"]) == 2
    err = capsys.readouterr().err
    assert "one GPU" in err and "--gpus 1" in err


def test_defaults_finish_within_minutes():
    a = bench.parse_args([])
    assert (a.gpus, a.steps, a.warmup, a.config) == (1, 50, 5, "flux_dev_1024")
    assert a.waves_per_cu is None and a.block is None      # the library's own launch shape


def test_traffic_reported_only_for_the_profiled_source(tmp_path, monkeypatch):
    src = os.path.join(bench.PROFILES, f"traffic_extrapolate_flux_dev_1024_{bench.LAYOUT}.md")
    if not os.path.exists(src):
        pytest.skip("no traffic profile committed")
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path))
    dst = tmp_path / os.path.basename(src)
    shutil.copy(src, dst)
    text = dst.read_text()
    # the committed profile was taken on the committed kernel source
    assert bench.measured_traffic("flux_dev_1024") == pytest.approx(11296309248, rel=1e-3)
    # a profile of another source is not used
    monkeypatch.setattr(bench, "kernel_sha256", lambda: "0" * 64)
    assert bench.measured_traffic("flux_dev_1024") is None
    monkeypatch.undo()
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path))
    dst.write_text(text.replace("traffic_bytes_per_launch", "traffic_bytes"))
    assert bench.measured_traffic("flux_dev_1024") is None
    assert bench.measured_traffic("no_such_workload") is None
