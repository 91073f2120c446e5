"""Host-side checks of bench.py (no GPU): the one-GPU contract and the roofline arithmetic
the JSON line reports (its lower bound per env-step, documented as 141.5 ps and 353,678
bf16-MFMA-equivalent FLOP for the headline workload)."""
import os
import subprocess
import sys

import pytest

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "exactly one GPU" in r.stderr and r.stdout == ""


def test_headline_lower_bound_per_env_step():
    # MFMA work of the 23-256-256-8 policy per env-step: the three layers' multiply-adds
    assert bench.F_MFMA == 2 * (23 * 256 + 256 * 256 + 256 * 8) == 146944
    # the transcendental peak: 256 CUs x 4 SIMDs x 8 lanes per cycle x 2.4 GHz
    assert bench.P_TRANS == pytest.approx(19.6608e12)
    t_lb = bench.F_MFMA / bench.P_MFMA + bench.F_VALU / bench.P_VALU + bench.N_TRANS / bench.P_TRANS
    assert t_lb == pytest.approx(141.5e-12, rel=1e-3)
    assert t_lb * bench.P_MFMA == pytest.approx(353678, rel=1e-4)


def test_recorded_traffic_follows_the_kernel_sources():
    """The counter summary is used only while its source hash matches the kernel sources
    (otherwise the JSON line reports null), and then gives the per-launch HBM bytes."""
    v = bench.recorded_traffic()
    kv = {}
    for line in open(bench.COUNTERS_FILE):
        if ":" in line and not line.startswith("#"):
            k, s = line.split(":", 1)
            kv[k.strip()] = s.strip()
    if kv.get("source_sha256") == bench.source_hash():
        assert v == float(kv["hbm_bytes_per_launch"]) > 0
        assert v == float(kv["fetch_bytes_per_launch"]) + float(kv["write_bytes_per_launch"])
    else:
        assert v is None
