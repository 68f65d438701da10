"""Host-side checks of bench.py that need no GPU: it refuses more than one
GPU with a message, and the calibrated traffic record it reports is read from
the committed counter summary only while that summary was taken on the
current contraction source (its recorded hash), with fetch plus writes adding
up to the reported traffic."""
import hashlib
import json
import os
import re
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_traffic_record_matches_the_contraction_source():
    md = open(os.path.join(ROOT, "profiles", "rotation_gemm_traffic.md")).read()
    rec = json.loads(re.search(r"```json\s*(\{.*?\})\s*```", md, re.S).group(1))
    src = os.path.join(ROOT, "paper_2609_37842_amd", "csrc", "gemm.hip")
    sha = hashlib.sha256(open(src, "rb").read()).hexdigest()
    got = bench.profiled_traffic()
    if rec["gemm_hip_sha256"] == sha:
        assert got == rec
        assert rec["traffic_bytes_per_launch"] == rec["fetch_bytes_per_launch"] + rec["write_bytes_per_launch"]
    else:
        assert got is None          # a stale summary is never reported as the kernel's traffic


def test_bench_defaults_are_the_headline_workload():
    a = bench.parse([])
    assert a.gpus == 1 and a.batch == 1250 and a.queries_per_step == 16 and a.blocks == 12
    assert a.prec == "f16" and a.pca_prec == "fast"
