"""bench.py's host-side parts on the CPU: the one-GPU rule, the CPU-oracle
leg, the traffic record and the source hash it is keyed by."""
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from workload import generate, small_spec  # noqa: E402


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_cpu_leg_times_the_gpu_window_on_the_host_cores():
    s = generate(small_spec(n=400, groups=4, prefix_len=(5, 30), suffix_len=(3, 20), vocab=9))
    out = bench.cpu_baseline(s, 3, 120, 100, 300, 5.0, replicas=3)
    assert out["kind"] == "oracle" and out["unit"] == "queries/s"
    assert 1 <= out["cores"] <= min(3, bench.host_cores())
    assert out["value"] > 0 and out["per_core"] > 0
    assert f"replicas 0..{out['cores'] - 1}" in out["sample"]
    assert "from query 100 on" in out["sample"] and "200..200 queries" in out["sample"]
    assert out["cpu_model"]


def test_oracle_window_timing_stops_at_its_budget():
    from oracle import oracle as O
    s = generate(small_spec(n=3000, groups=4, prefix_len=(20, 60), suffix_len=(10, 40), vocab=50))
    o = O.run(s, 4, 400, time_from=100, time_budget_s=1e-9)
    assert o["rc"] == 0 and 101 <= o["done"] < s.n  # stops right after the first timed query
    assert o["window_cpu_s"] > 0 and o["window_wall_s"] > 0
    full = O.run(s, 4, 400, n=o["done"])
    assert (full["route"] == o["route"]).all()


def test_host_cores_is_at_most_one_gpus_share():
    assert 1 <= bench.host_cores() <= 16


def test_source_hash_ignores_comments_and_whitespace():
    a = "int f(int x) {\n  return x + 1;  // one more\n}\n/* block\n comment */"
    b = "int f(int x) { return x + 1; }"
    assert bench._code_only(a) == bench._code_only(b)
    assert bench._code_only("int x = 1;") != bench._code_only("int x = 2;")
    h = bench.kernel_source_hash()
    assert len(h) == 16 and h == bench.kernel_source_hash()


def test_traffic_record_used_only_for_the_current_sources_and_window(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    (tmp_path / "profiles").mkdir()
    rec = {"kernel_source_hash": "0" * 16, "bytes_per_launch": 1.0, "batch": 2000, "warmup": 5, "steps": 20}
    (tmp_path / "profiles" / "traffic_w.json").write_text(json.dumps(rec))
    monkeypatch.setattr(bench, "kernel_source_hash", lambda: "1" * 16)
    assert bench.load_traffic("w", 2000, 5, 20) is None
    monkeypatch.setattr(bench, "kernel_source_hash", lambda: "0" * 16)
    assert bench.load_traffic("w", 2000, 5, 20)["bytes_per_launch"] == 1.0
    assert bench.load_traffic("w", 2000, 4, 6) is None  # another window
    assert bench.load_traffic("w", 1000, 5, 20) is None
    assert bench.load_traffic("absent", 2000, 5, 20) is None
