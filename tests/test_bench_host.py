"""Host-side parts of bench.py that run without a GPU: the one-GPU guard and
the rule that measured HBM traffic is reported only for the kernel sources
the counters were taken from."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


@pytest.mark.parametrize("argv,env", [(["--gpus", "2"], {}), (["--gpus", "1"], {"WORLD_SIZE": "4"})])
def test_more_than_one_gpu_is_refused(argv, env):
    e = dict(os.environ)
    e.update(env)
    p = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py")] + argv, capture_output=True, text=True,
                       env=e, timeout=120)
    assert p.returncode == 2
    assert "one GPU" in p.stderr
    assert p.stdout == ""  # no JSON line


def test_traffic_only_for_matching_sources(monkeypatch):
    import bench
    from paper_2501_19090_amd import build
    path = os.path.join(ROOT, "profiles", "pifa_gemm1_xwp_attn4096_M4096_traffic.txt")
    with open(path) as f:
        rec = json.load(f)
    if "forward_kernel_digest" in rec:
        monkeypatch.setattr(build, "forward_kernel_digest", lambda: rec["forward_kernel_digest"])
        assert bench.traffic_from_profiles("pifa_gemm1_xwp") == rec["hbm_bytes_per_launch"]
    else:  # a record that does not name the kernels' version is never used
        assert bench.traffic_from_profiles("pifa_gemm1_xwp") is None
    monkeypatch.setattr(build, "forward_kernel_digest", lambda: "0" * 16)
    assert bench.traffic_from_profiles("pifa_gemm1_xwp") is None
    assert bench.traffic_from_profiles("no_such_kernel") is None


def test_traffic_record_is_consistent():
    """The stored per-launch bytes are the raw KiB counts (averaged over the
    kernel's dispatches) times the copy calibration factors (FETCH_SIZE /
    WRITE_SIZE of a copy of known size)."""
    path = os.path.join(ROOT, "profiles", "pifa_gemm1_xwp_attn4096_M4096_traffic.txt")
    with open(path) as f:
        rec = json.load(f)
    fetch_scale = rec["copy_bytes"] / (rec["copy_fetch_kib_raw"] * 1024)
    write_scale = rec["copy_bytes"] / (rec["copy_write_kib_raw"] * 1024)
    assert rec["fetch_scale"] == pytest.approx(fetch_scale, rel=1e-9)
    assert rec["write_scale"] == pytest.approx(write_scale, rel=1e-9)
    assert rec["dispatches"]["fetch"] > 0 and rec["dispatches"]["write"] > 0
    read = rec["fetch_kib_raw"] * 1024 * fetch_scale
    write = rec["write_kib_raw"] * 1024 * write_scale
    assert rec["hbm_bytes_per_launch"] == pytest.approx(read + write, rel=1e-9)
