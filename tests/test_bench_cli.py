"""bench.py's host-side contract (no GPU): one GPU only, nearest-rank P99, and measured
traffic reported only for the kernel source it was measured on."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


@pytest.mark.parametrize("args,env", [(["--gpus", "2"], {}), (["--gpus", "8"], {}), ([], {"WORLD_SIZE": "2"})])
def test_more_than_one_gpu_is_refused(args, env):
    e = dict(os.environ, **env)
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], capture_output=True, text=True,
                       env=e, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_p99_is_nearest_rank():
    assert bench.p99(list(range(1, 1001))) == 990
    assert bench.p99(list(range(100, 0, -1))) == 99
    assert bench.p99([7.0]) == 7.0


def test_source_hash_is_stable_and_covers_the_planner():
    assert bench.kernel_source_hash() == bench.kernel_source_hash()
    assert any(p.endswith("lookup.hip") for p in bench.KERNEL_SOURCES)
    assert any(p.endswith("planner.cpp") for p in bench.KERNEL_SOURCES)


def test_traffic_only_for_the_matching_source():
    names = sorted(f for f in os.listdir(os.path.join(ROOT, "profiles")) if f.startswith("traffic_"))
    assert names
    for f in names:
        d = json.load(open(os.path.join(ROOT, "profiles", f)))
        w = f[len("traffic_"):-len(".json")]
        assert bench.load_traffic(w, d["kernel_source_hash"]) == d["hbm_bytes_per_launch"] > 0
        assert bench.load_traffic(w, "0" * 16) is None
        assert d["hbm_bytes_per_launch"] == pytest.approx(d["hbm_read_bytes_per_launch"] + d["hbm_write_bytes_per_launch"])
    assert bench.load_traffic("no-such-workload", bench.kernel_source_hash()) is None


@pytest.mark.parametrize("args", [["--streams", "5"], ["--streams", "0"], ["--table-costs", "x"]])
def test_bad_throughput_options_are_refused_before_the_gpu(args):
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], capture_output=True, text=True,
                       timeout=120)
    assert r.returncode == 2 and r.stdout == ""
    assert "--streams" in r.stderr or "--table-costs" in r.stderr
