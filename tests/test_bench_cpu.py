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
    # 256 CUs x 64 lanes x 2.4 GHz issue slots over 38 slots per block: 18 products at
    # one slot each, 22 xors and 18 key adds at two per slot
    assert bench.PHILOX_ISSUE_SLOTS == 38
    assert abs(bench.PHILOX_PEAK_GBLOCKS - 256 * 64 * 2.4 / 38) < 1e-9
    assert 1030 < bench.PHILOX_PEAK_GBLOCKS < 1040
    assert bench.HBM_PEAK_GBPS == 8000.0


def test_rate_probe_source_counts_match_the_roof():
    # the probe's block is the 58-op block the roof counts: 10 rounds, counter (c,0,0,0)
    src = open(os.path.join(ROOT, "paper_2609_03844_amd", "csrc", "philox_rate.hip")).read()
    assert "for (int r = 0; r < 10; ++r)" in src
    assert "kChains = 8" in src
    # the scheduled kernel draws the library's own per-lane-key block
    assert "sbw::philox_block_lane" in src and "sbw_rate_philox_sched" in src
    assert os.path.basename(bench.RATE_LIBRARY) == "libsbw_rate.so"


def test_cpu_baseline_fields(monkeypatch):
    # the CPU leg on a tiny batch: every field the benchmark line reports is there
    import numpy as np
    import workloads
    monkeypatch.setattr(workloads, "C4", dict(workloads.C4))
    x = np.random.default_rng(0).standard_normal((4, 64)).astype(np.float32)
    prev = np.arange(4, dtype=np.int32)
    toks = {s: np.random.default_rng(1).integers(0, 64, (8, 16)).astype(np.int32)
            for s in ("self_salt", "context")}
    monkeypatch.setattr(bench, "_threads", lambda: 2)
    out = bench.cpu_baseline(x, prev, toks, runs=1)
    for k in ("value", "value_1thread", "unit", "cores", "kind", "sample", "cpu", "nproc",
              "detect_seq_per_s", "runs"):
        assert k in out, k
    assert out["kind"] == "oracle" and out["cores"] == 2
    for s in ("self_salt", "context"):
        assert out["watermark"][s]["gelem_per_s"] > 0
        assert out["detect"][s]["seq_per_s"] > 0 and out["detect"][s]["seq_per_s_1thread"] > 0


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
