"""Host-side logic of bench.py: the measured-traffic lookup and the
single-GPU guard (no GPU needed)."""
import json
import subprocess
import sys

import bench


def test_traffic_is_used_only_for_the_profiled_source(tmp_path):
    p = tmp_path / "traffic.json"
    p.write_text(json.dumps({"kernel_source_sha": bench._kernel_sha(), "long70b": {"bytes_per_launch": 123}}))
    assert bench._attention_traffic(str(p), "long70b") == 123
    assert bench._attention_traffic(str(p), "batched") is None
    p.write_text(json.dumps({"kernel_source_sha": "0" * 16, "long70b": {"bytes_per_launch": 123}}))
    assert bench._attention_traffic(str(p), "long70b") is None
    assert bench._attention_traffic(str(tmp_path / "missing.json"), "long70b") is None


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, "bench.py", "--gpus", "2"], capture_output=True, text=True,
                       cwd=bench.ROOT, timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr
