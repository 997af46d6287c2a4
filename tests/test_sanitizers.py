"""CPU runs of the host-side code under AddressSanitizer and
UndefinedBehaviorSanitizer: the fp64 oracle (wfref.c, built with gcc's
sanitizers) through its pinning tests, and libwf's host code (argument
validation, workspace queries, the lazy catch-up bookkeeping; built by hipcc
with the sanitizers on the host pass only) through the C-ABI tests.  Each run
is a child pytest process with the matching sanitizer runtime preloaded; any
report fails it.  No GPU call is made."""
import glob
import importlib.util
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN_DIR = os.path.join(ROOT, "_build", "san")

ORACLE_TESTS = ["test_oracle_attention.py", "test_oracle_decoder.py",
                "test_oracle_lmhead.py", "test_oracle_prefill.py",
                "test_oracle_router.py", "test_oracle_tree.py", "test_golden.py"]
HOST_TESTS = ["test_abi.py", "test_switch_state.py", "test_random_cases.py"]
SAN_ENV = {"ASAN_OPTIONS": "detect_leaks=0:abort_on_error=1",
           "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1"}


def _run(tests, env_extra):
    env = dict(os.environ, **SAN_ENV, **env_extra)
    cmd = [sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
           "-m", "not gpu"] + [os.path.join(ROOT, "tests", t) for t in tests]
    r = subprocess.run(cmd, env=env, cwd=ROOT, capture_output=True, text=True,
                       timeout=600)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "runtime error" not in out and "AddressSanitizer" not in out, out[-4000:]
    assert " passed" in out


def test_oracle_under_sanitizers():
    gcc = shutil.which("gcc")
    if not gcc:
        pytest.skip("gcc missing")
    asan = subprocess.run([gcc, "-print-file-name=libasan.so"], capture_output=True,
                          text=True).stdout.strip()
    ubsan = subprocess.run([gcc, "-print-file-name=libubsan.so"], capture_output=True,
                           text=True).stdout.strip()
    if not (os.path.isabs(asan) and os.path.isabs(ubsan)):
        pytest.skip("gcc sanitizer runtimes missing")
    os.makedirs(SAN_DIR, exist_ok=True)
    from oracle import build as oracle_build
    lib = oracle_build.build(out=os.path.join(SAN_DIR, "libwfref.so"), sanitize=True)
    _run(ORACLE_TESTS, {"WFREF_LIB": lib, "LD_PRELOAD": f"{asan}:{ubsan}"})


def test_library_host_code_under_sanitizers():
    rts = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    if not rts or not shutil.which("/opt/rocm/bin/hipcc"):
        pytest.skip("hipcc or its sanitizer runtime missing")
    spec = importlib.util.spec_from_file_location(
        "_wf_build_san", os.path.join(ROOT, "paper_2606_07710_amd", "build.py"))
    b = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(b)
    lib = b.build(sanitize=True)
    _run(HOST_TESTS, {"WF_LIB": lib, "LD_PRELOAD": rts[-1]})
