"""CPU: the host C++ (argument validation, the host planner and its sizing, the scheduler)
under AddressSanitizer and UndefinedBehaviorSanitizer.  The library is rebuilt with its host
sources compiled by g++ with -fsanitize=address,undefined (UB aborts), and the host-side test
files run against it in a child interpreter with the ASan runtime preloaded.  No GPU call is
made: those files only validate, plan and schedule."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HOST_TESTS = ["tests/test_abi_cpu.py", "tests/test_plan_cpu.py", "tests/test_sched_parity.py"]


def _asan_runtime():
    gcc = shutil.which("gcc")
    if not gcc:
        return None
    path = subprocess.run([gcc, "-print-file-name=libasan.so"], capture_output=True, text=True).stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


@pytest.fixture(scope="module")
def sanitized_env():
    asan = _asan_runtime()
    if asan is None or shutil.which("g++") is None:
        pytest.skip("g++ with libasan is needed for the sanitizer build")
    from paper_2604_16395_amd.build import build_sanitized
    lib = build_sanitized()
    env = dict(os.environ)
    pre = env.get("LD_PRELOAD", "")
    env["LD_PRELOAD"] = asan + (":" + pre if pre else "")   # the ASan runtime first, the rest kept
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1"   # the interpreter itself is not instrumented
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    env["S2L_LIBRARY"] = lib
    env["PYTHONPATH"] = ROOT + (os.pathsep + env["PYTHONPATH"] if env.get("PYTHONPATH") else "")
    return env, lib


def test_the_sanitized_library_is_the_one_loaded(sanitized_env):
    env, lib = sanitized_env
    code = ("import paper_2604_16395_amd._lib as L; L.lib(); "
            "print(any(L.LIB_PATH in l for l in open('/proc/self/maps')), L.LIB_PATH)")
    p = subprocess.run([sys.executable, "-c", code], env=env, cwd=ROOT, capture_output=True, text=True, timeout=300)
    assert p.returncode == 0, p.stdout + p.stderr
    assert p.stdout.split() == ["True", lib]


def test_host_side_tests_pass_under_asan_and_ubsan(sanitized_env):
    env, _ = sanitized_env
    cmd = [sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider", "-m", "not gpu", *HOST_TESTS]
    p = subprocess.run(cmd, env=env, cwd=ROOT, capture_output=True, text=True, timeout=900)
    out = p.stdout + p.stderr
    assert p.returncode == 0, out[-4000:]
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
    assert " passed" in out
