"""The bench harness on the host: the one-GPU contract and the
comment-insensitive source digests that tie profiles to kernel sources."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_more_than_one_gpu_exits_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_code_text_ignores_comments_and_layout():
    a = "int f(int x) {\n  // add one\n  return x + 1; /* done */\n}\n"
    b = "int f(int x){return x+1;}"
    c = "int f(int x) { return x + 2; }"
    assert bench.code_text(a) == bench.code_text(b)
    assert bench.code_text(a) != bench.code_text(c)


def test_source_digests_are_stable_and_distinct():
    d1 = bench.source_digest("attention.hip")
    assert d1 == bench.source_digest("attention.hip")
    assert len({d1, bench.source_digest("assemble.hip"), bench.source_digest("select.hip"),
                bench.source_digest("gemm.hip")}) == 4
