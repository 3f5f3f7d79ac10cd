"""Host-side checks of bench.py (no GPU): the one-GPU contract and the
counter-traffic bookkeeping."""
import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    res = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                         capture_output=True, text=True, timeout=120)
    assert res.returncode == 2
    assert "one GPU" in res.stderr


def test_traffic_is_null_once_the_kernel_source_changes(monkeypatch):
    for kernel, (src, fetch, write) in bench.TRAFFIC_KIB.items():
        assert src in bench.TRAFFIC_SOURCES
        assert fetch > 0 and write >= 0
    monkeypatch.setitem(bench.TRAFFIC_SOURCES, "linear_decode.hip", "0" * 64)
    assert bench.traffic_bytes("gemv_lut_kernel<1,2,2>") is None
    assert bench.traffic_bytes("no_such_kernel") is None


def test_traffic_scale_from_copy_is_sane():
    # the counters were scaled by a plain copy: both factors near small integers
    assert 0.9 < bench.TRAFFIC_WRITE_SCALE < 1.1
    assert 0.9 < bench.TRAFFIC_FETCH_SCALE < 2.1
