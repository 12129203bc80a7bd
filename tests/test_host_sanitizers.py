"""The library's host C++ (the CPU decode attention and its thread pool, the
scheduler simulator, the error text) and the oracle, built with sanitizers and
run on generated inputs: one build with AddressSanitizer and
UndefinedBehaviorSanitizer, one with ThreadSanitizer. The driver
(host_sanitize_check.cpp) also checks the CPU attention against the oracle."""
import os
import shutil
import subprocess

import pytest

from paper_2411_01142_amd import _build as B

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SOURCES = [os.path.join(B.CSRC, f) for f in ("cpu_attention.cpp", "scheduler.cpp",
                                             "neo_error.cpp")]
DRIVER = os.path.join(HERE, "host_sanitize_check.cpp")
ORACLE = os.path.join(ROOT, "oracle", "neo_ref.c")

FLAVOURS = {
    "address_undefined": ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined"],
    "thread": ["-fsanitize=thread"],
}


@pytest.mark.parametrize("flavour", sorted(FLAVOURS))
def test_host_code_runs_clean_under_sanitizer(flavour, tmp_path):
    gcc, gxx = shutil.which("gcc"), shutil.which("g++")
    if not gcc or not gxx:
        pytest.skip("gcc/g++ not found")
    san = FLAVOURS[flavour]
    common = ["-O1", "-g", "-fno-omit-frame-pointer", *san]
    ref_obj = str(tmp_path / "neo_ref.o")
    subprocess.run([gcc, *common, "-std=c11", "-c", ORACLE, "-o", ref_obj], check=True,
                   capture_output=True, text=True)
    exe = str(tmp_path / f"host_check_{flavour}")
    res = subprocess.run([gxx, *common, "-std=c++17", "-pthread", "-I" + B.INCLUDE, "-I" + B.CSRC,
                          DRIVER, *SOURCES, ref_obj, "-o", exe, "-lm"],
                         capture_output=True, text=True)
    assert res.returncode == 0, res.stderr[-4000:]
    env = dict(os.environ)
    env["ASAN_OPTIONS"] = "detect_leaks=1:abort_on_error=0:halt_on_error=1"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    env["TSAN_OPTIONS"] = "halt_on_error=1:second_deadlock_stack=1"
    env.pop("NEO_CPU_ISA", None)
    run = subprocess.run([exe], capture_output=True, text=True, timeout=900, env=env)
    assert run.returncode == 0, (run.stdout + run.stderr)[-6000:]
    assert run.stdout.startswith("ok"), run.stdout
    assert "runtime error" not in run.stderr, run.stderr[-4000:]
    assert "WARNING: ThreadSanitizer" not in run.stderr, run.stderr[-4000:]
