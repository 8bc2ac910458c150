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


def test_oracle_rate_counts_every_worker_and_cycles_past_one_pass():
    # a pass over the three items takes ~3 ms; the budget forces many passes
    import time

    def work(n):
        time.sleep(0.001)
        return n
    for workers in (1, 2):
        rate, count, dt = bench._oracle_rate(work, [1, 2, 3], 0.2, workers)
        assert count > 3 * workers and dt >= 0.2
        assert 0 < rate <= 3 * workers / 0.001


def test_cpu_baseline_reports_both_modes_on_the_tiny_workload():
    import workloads as W
    w = W.make("tiny", poison=False)
    r = bench.cpu_baseline(w, 0.3)
    assert r["kind"] == "oracle" and r["unit"] == "GB/s" and r["cores"] == bench._host_cores()
    assert r["value"] > 0 and r["single_thread"]["value"] > 0 and r["single_thread"]["cores"] == 1
