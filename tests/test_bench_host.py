"""Host-side pieces of bench.py (no GPU): the algorithmic byte count of the
LM-head call, the code hash that ties committed counters to the kernel
source, and the one-GPU guard."""
import json
import os
import subprocess
import sys

import pytest

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_lmhead_bytes_formula():
    class S:
        V, d, N = 126464, 4096, 77
    # W once (bf16), the scored hidden rows (bf16), conf + argmax + lse (4 B each)
    assert bench.lmhead_bytes(S) == 2 * 126464 * 4096 + 2 * 77 * 4096 + 12 * 77
    assert bench.lmhead_bytes(S) == 1036624796


def test_code_only_drops_comments_and_keeps_code():
    src = "int a = 1;  // one\n/* block\n   comment */\nint b = a / 2; /* x */ int c;\n\n   // only a comment\n"
    assert bench._code_only(src) == "int a = 1;\nint b = a / 2;  int c;"


def test_code_hash_ignores_comment_edits(tmp_path, monkeypatch):
    csrc = tmp_path / "paper_2606_08411_amd" / "csrc"
    csrc.mkdir(parents=True)
    (csrc / "lmhead.hip").write_text("int f() { return 1; }  // first\n")
    (csrc / "common.h").write_text("#pragma once\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    h0 = bench.kernel_source_hash()
    (csrc / "lmhead.hip").write_text("// a new header comment\nint f() { return 1; }  /* second */\n")
    assert bench.kernel_source_hash() == h0
    (csrc / "lmhead.hip").write_text("int f() { return 2; }\n")
    assert bench.kernel_source_hash() != h0


def test_traffic_record_matches_layout_and_code():
    path = os.path.join(ROOT, "profiles", "lmhead_confidence_llada_pmc.json")
    with open(path) as f:
        rec = json.load(f)
    assert rec["w_layout"] in ("packed", "plain")
    if rec["kernel_source_hash"] == bench.kernel_source_hash():
        assert bench.measured_traffic("llada", rec["w_layout"]) == rec["hbm_bytes_per_launch"]
    other = "plain" if rec["w_layout"] == "packed" else "packed"
    assert bench.measured_traffic("llada", other) is None
    assert bench.measured_traffic("no_such_workload", "packed") is None


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=300, cwd=ROOT)
    assert r.returncode != 0
    assert "one GPU" in (r.stdout + r.stderr)
