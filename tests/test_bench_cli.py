"""bench.py's contract on the CPU: one GPU only, the counter record tied to
the kernel source it was taken on, and the host-only simulator mode."""
import json
import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _run(*args, timeout=300):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args],
                          capture_output=True, text=True, timeout=timeout)


def test_more_than_one_gpu_is_refused_with_a_message():
    p = _run("--gpus", "2")
    assert p.returncode == 2
    assert "one GPU" in p.stderr
    assert p.stdout == ""


def test_kernel_hash_ignores_comments_and_whitespace_only():
    code = "int f(int x) {\n    return x + 1;   // one more\n}\n"
    same = "int f(int x) {   return x + 1; // a different comment\n\n}\n"
    other = "int f(int x) {\n    return x + 2;\n}\n"
    assert bench.kernel_hash([code]) == bench.kernel_hash([same])
    assert bench.kernel_hash([code]) != bench.kernel_hash([other])


def test_counter_record_of_other_code_gives_no_traffic(tmp_path, monkeypatch):
    rec = {"kernel_sha": "0000000000000000", "bytes_per_launch": 1.0}
    path = tmp_path / "traffic.json"
    path.write_text(json.dumps(rec))
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(path))
    assert bench.measured_traffic(1.0) is None
    rec["kernel_sha"] = bench.kernel_hash()
    path.write_text(json.dumps(rec))
    assert bench.measured_traffic(1.0) == 1.0


def test_committed_counter_record_names_its_kernel_and_calibration():
    with open(bench.TRAFFIC_FILE) as fh:
        rec = json.load(fh)
    assert "fused_ws_kernel" in rec["kernel"]
    assert len(rec["kernel_sha"]) == 16
    cal = rec["calibration"]
    # the read probe's loads match the kernel's; the recorded bytes are the
    # counters divided by those factors
    assert abs(rec["read_bytes_per_launch"]
               - rec["FETCH_SIZE_KiB_per_dispatch"] * 1024 / cal["read_factor"]) < 1e3
    assert abs(rec["write_bytes_per_launch"]
               - rec["WRITE_SIZE_KiB_per_dispatch"] * 1024 / cal["fill_write_factor"]) < 1e3
    assert rec["bytes_per_launch"] >= rec["algorithmic_bytes_per_launch"]


def test_simulate_mode_prints_one_json_line():
    p = _run("--simulate")
    assert p.returncode == 0, p.stderr
    lines = [ln for ln in p.stdout.splitlines() if ln.strip()]
    assert len(lines) == 1
    out = json.loads(lines[0])
    assert out["mode"] == "simulate"
    # Tables 1-3 settings: K = 15, 21, 24 with r = 3, both attacks
    assert {(row["K"], row["attack"]) for row in out["tables_1_3"]} == \
        {(K, a) for K in (15, 21, 24) for a in ("optimal", "weak")}
    assert all(row["files"] == {15: 455, 21: 1330, 24: 2024}[row["K"]] for row in out["tables_1_3"])
    assert len(out["k100_r5"]) == 10
