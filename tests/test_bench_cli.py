"""Host-side checks of bench.py that need no GPU: the one-GPU contract and the
rule that committed HBM counters are used only while the kernel sources they
were taken from are unchanged."""
import os
import subprocess
import sys

import bench
import workloads as wl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    p = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert p.returncode == 2
    assert "one GPU" in p.stderr and p.stdout == ""


def test_traffic_only_for_matching_sources(tmp_path, monkeypatch):
    w = wl.WORKLOADS["fwd_d512"]
    sha = bench.source_digest("paper_2505_00315_amd/csrc")
    assert sha is not None and len(sha) == 16
    f = tmp_path / "counters.txt"
    f.write_text("# header\n"
                 f"stage=wgrad workload={w.name} source=paper_2505_00315_amd/csrc source_sha={sha} "
                 "fetch_kib=1 write_kib=1 hbm_bytes_per_launch=12345\n"
                 f"stage=select workload={w.name} source=paper_2505_00315_amd/csrc source_sha=0000000000000000 "
                 "fetch_kib=1 write_kib=1 hbm_bytes_per_launch=999\n")
    monkeypatch.setattr(bench, "COUNTERS_FILE", str(f))
    assert bench.traffic_for("wgrad", w) == 12345.0
    assert bench.traffic_for("select", w) is None           # sources changed since
    assert bench.traffic_for("router", w) is None           # no line for the stage
    assert bench.traffic_for("wgrad", wl.WORKLOADS["fwdbwd_d1024"]) is None  # other workload
