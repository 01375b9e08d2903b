"""bench.py's host-side contract, without a GPU: one GPU only, the Philox roof it
reports against, and the traffic lookup that only trusts counters taken on the current
kernel sources."""
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_more_than_one_gpu_exits_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode != 0
    line = json.loads(r.stdout.strip().splitlines()[-1])
    assert line["n_gpus"] == 2 and "one GPU" in line["error"]


def test_philox_roof_from_unit_counts():
    # 256 CUs x 64 lanes x 2.4 GHz full-rate lane-ops over 58 lane-ops per block
    assert abs(bench.PHILOX_PEAK_GBLOCKS - 256 * 64 * 2.4 / 58) < 1e-9
    assert 670 < bench.PHILOX_PEAK_GBLOCKS < 690
    assert bench.HBM_PEAK_GBPS == 8000.0


def test_traffic_lookup_refuses_counters_of_other_sources(tmp_path):
    prof = {"source_sha256": "0" * 64, "kernels": {"k@1": {"hbm_bytes": 1.0}}}
    path = tmp_path / "p.json"
    path.write_text(json.dumps(prof))
    assert bench.measured_traffic(str(path)) == {}
    assert bench.measured_traffic(str(tmp_path / "missing.json")) == {}


def test_traffic_lookup_accepts_counters_of_these_sources(tmp_path):
    import hashlib
    h = hashlib.sha256()
    for f in bench.KERNEL_SOURCES:
        h.update(open(os.path.join(ROOT, f), "rb").read())
    prof = {"source_sha256": h.hexdigest(), "kernels": {"k@1": {"hbm_bytes": 311.0e6}}}
    path = tmp_path / "p.json"
    path.write_text(json.dumps(prof))
    assert bench.measured_traffic(str(path)) == {"k@1": 311.0e6}
