"""bench.py pieces that need no GPU: the one-GPU guard and the counter-record check."""
import json
import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_exits_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_attention_digest_ignores_comments(tmp_path, monkeypatch):
    src = open(os.path.join(ROOT, "paper_2606_05875_amd", "csrc", "attention.hip")).read()
    base = bench.attention_code_digest()
    fake = tmp_path / "paper_2606_05875_amd" / "csrc"
    fake.mkdir(parents=True)
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    (fake / "attention.hip").write_text("// a new comment line\n" + src.replace("{\n", "{  /* note */\n", 1))
    assert bench.attention_code_digest() == base
    (fake / "attention.hip").write_text(src.replace("kKT = 64", "kKT = 32", 1))
    assert bench.attention_code_digest() != base


def test_traffic_record_is_used_only_for_its_code_and_stride(tmp_path, monkeypatch):
    prof = tmp_path / "profiles"
    prof.mkdir()
    csrc = tmp_path / "paper_2606_05875_amd" / "csrc"
    csrc.mkdir(parents=True)
    (csrc / "attention.hip").write_text("int f() { return 1; }\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    digest = bench.attention_code_digest()
    rec = {"attention_code_sha256": digest, "kv_row_stride": 1152, "bytes_per_call": 123}
    (prof / "attention_c4_hbm_traffic.md").write_text("# record\n\n" + json.dumps(rec) + "\n")
    assert bench.measured_traffic("c4", 1152) == 123
    assert bench.measured_traffic("c4", 1024) is None          # another cache row stride
    assert bench.measured_traffic("c2", 1152) is None          # no record for that workload
    (csrc / "attention.hip").write_text("int f() { return 2; }\n")
    assert bench.measured_traffic("c4", 1152) is None          # the kernel changed since
