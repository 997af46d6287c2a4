"""The benchmark's command-line contract, checked without a GPU: more than
one GPU is refused with a message, and the help lists every workload flag."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _run(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args],
                          capture_output=True, text=True, timeout=120, cwd=ROOT)


def test_more_than_one_gpu_is_refused():
    r = _run("--gpus", "2")
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_help_lists_the_options():
    r = _run("--help")
    assert r.returncode == 0
    for flag in ("--config", "--steps", "--warmup", "--batch-prefill-layers",
                 "--row-major-weights", "--router", "--switch-table", "--graph"):
        assert flag in r.stdout, flag
