"""Host-side logic of bench.py, on the CPU: the one-GPU refusal and the rule
that committed HBM counter figures are used only for the kernel sources they
were taken on."""
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr and r.stdout == ""


def test_traffic_record_matches_current_kernels(monkeypatch, tmp_path):
    rec = json.load(open(os.path.join(ROOT, "profiles", "traffic_gateup_mixtral_decode.json")))
    assert abs(rec["read_bytes"] + rec["write_bytes"] - rec["bytes_per_launch"]) <= 2   # each part rounded
    # a record taken on other sources is ignored, a matching one is used
    (tmp_path / "profiles").mkdir()
    fake = dict(rec, kernel_sha256_16="0" * 16)
    (tmp_path / "profiles" / "traffic_gateup_mixtral_decode.json").write_text(json.dumps(fake))
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.traffic_for("gateup", "mixtral_decode", 1) is None
    fake["kernel_sha256_16"] = bench.kernel_hash()
    (tmp_path / "profiles" / "traffic_gateup_mixtral_decode.json").write_text(json.dumps(fake))
    assert bench.traffic_for("gateup", "mixtral_decode", 1) == rec["bytes_per_launch"]
    assert bench.traffic_for("down", "mixtral_decode", 1) is None     # no record
