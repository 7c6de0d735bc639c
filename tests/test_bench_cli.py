"""bench.py's command line without a GPU: more than one GPU is refused with a
message (one GPU is measured), and the counter summary keyed to another
kernel source is ignored."""
from __future__ import annotations

import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=300, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout.strip() == ""


def test_counter_traffic_follows_the_kernel_source(tmp_path, monkeypatch):
    sys.path.insert(0, ROOT)
    import bench

    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    os.makedirs(tmp_path / "profiles")
    src = tmp_path / "paper_2606_12280_amd" / "csrc"
    os.makedirs(src)
    (src / "gemm.hip").write_text("// kernel v1\n")
    sha = bench.sources_sha(bench.GEMM_SOURCES)
    with open(tmp_path / "profiles" / "gemm_ffn_up_counters.json", "w") as f:
        json.dump({"kernel_source_sha256": sha, "hbm_bytes_per_launch": 123}, f)
    assert bench.counter_traffic("ffn_up") == 123
    (src / "gemm.hip").write_text("// kernel v2\n")
    assert bench.counter_traffic("ffn_up") is None
    assert bench.counter_traffic("ffn_down") is None
