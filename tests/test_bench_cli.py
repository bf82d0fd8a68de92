"""bench.py's command line on the host: it measures one GPU only and says so
for any other count, and rejects unknown optional sections, before touching
the GPU or building anything."""

import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _run(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args],
                          capture_output=True, text=True, timeout=120, cwd=ROOT)


def test_more_than_one_gpu_is_refused_with_a_message():
    p = _run("--gpus", "2")
    assert p.returncode == 2
    assert "one GPU" in p.stderr and p.stdout == ""


def test_unknown_section_is_rejected():
    p = _run("--skip", "qat,nonsense")
    assert p.returncode == 2
    assert "nonsense" in p.stderr
