"""bench.py command-line contract that holds without a GPU."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr
    assert r.stdout == ""


def test_bench_tokens_only_with_decode_only():
    for extra in (["--tokens", "4"], ["--decode-only", "--tokens", "17"], ["--decode-only", "--tokens", "0"]):
        r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *extra],
                           capture_output=True, text=True, timeout=120, cwd=ROOT)
        assert r.returncode == 2, extra
        assert "--tokens M (1..16) only with --decode-only" in r.stderr
        assert r.stdout == ""
