"""Host-side pieces of the benchmark, without a GPU: the multi-GPU refusal, and
the digest that ties a committed counter summary to the kernel code it was
taken on."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, cwd=ROOT, timeout=120)
    assert r.returncode != 0
    assert "single" in (r.stdout + r.stderr).lower()


def test_digest_ignores_comments_and_whitespace(tmp_path, monkeypatch):
    csrc = tmp_path / "paper_2606_10650_amd" / "csrc"
    csrc.mkdir(parents=True)
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "KERNEL_SOURCES", {"k": ["a.hip"]})
    f = csrc / "a.hip"
    f.write_text("int x = 1;  // one\n/* block\n comment */ int y = 2;\n")
    d0 = bench.source_digest("k")
    f.write_text("int x = 1;\n\n   int y = 2;   // a different comment\n")
    assert bench.source_digest("k") == d0
    f.write_text("int x = 1; int y = 3;\n")
    assert bench.source_digest("k") != d0

