"""bench.py's contract on the host: one GPU only, and profiled counter figures
reported only for the kernel sources they were measured with."""
import hashlib
import json
import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2", "--steps", "1"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def _sha(name):
    with open(os.path.join(ROOT, "paper_2307_02486_amd", "csrc", name), "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def test_profiled_counters_follow_the_kernel_sources(tmp_path, monkeypatch):
    keys = [n.replace(".", "_") + "_sha256_16" for n in bench.PROFILED_SOURCES]
    assert "device_common_h_sha256_16" in keys   # the shared header changes both kernels
    rec = {"attention_bytes_per_launch": 123, "combine_bytes_per_launch": 45, "attention_mfma_busy_pct": 40.0}
    rec.update({k: _sha(n) for k, n in zip(keys, bench.PROFILED_SOURCES)})
    path = tmp_path / "traffic.json"
    monkeypatch.setattr(bench, "PROFILED_TRAFFIC", str(path))
    assert bench.profiled_counters("w") == {}                 # no file
    path.write_text(json.dumps({"w": rec}))
    assert bench.profiled_counters("w") == rec                # sources unchanged
    assert bench.profiled_counters("other") == {}             # workload never profiled
    for key in keys:
        path.write_text(json.dumps({"w": dict(rec, **{key: "0" * 16})}))
        assert bench.profiled_counters("w") == {}             # a kernel changed since: no figures
