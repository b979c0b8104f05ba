"""The benchmark's command-line contract, checked on the CPU: more than one
GPU is refused with a message before any device work, and the GEMM traffic
record is reported only while its source hash matches the GEMM source."""
import json
import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120, cwd=ROOT)
    assert r.returncode != 0
    assert "--gpus 1" in (r.stdout + r.stderr)


def test_gemm_traffic_follows_the_source_hash(tmp_path, monkeypatch):
    rec = json.load(open(os.path.join(ROOT, "profiles", "gemm_f32_mfma_gpt2_124m_b16_traffic.json")))
    src = os.path.join(ROOT, "paper_2606_24780_amd", "csrc", "gemm.hip")
    assert rec["gemm_source_sha256"] == bench.code_sha256(src)
    traffic, alg = bench.gemm_traffic()
    assert traffic == rec["traffic_bytes_per_launch"] and alg == rec["algorithmic_bytes_per_launch"]
    # comments and blank lines do not change the hash; code does
    text = open(src, encoding="utf-8").read()
    a = tmp_path / "a.hip"
    a.write_text(text + "\n// a comment\n\n")
    assert bench.code_sha256(str(a)) == bench.code_sha256(src)
    a.write_text(text + "\nint extra;\n")
    assert bench.code_sha256(str(a)) != bench.code_sha256(src)
