"""The input generator (synth/synth.c) and the C++ oracle (oracle/kvec_oracle.cpp)
built with AddressSanitizer and UndefinedBehaviorSanitizer on the host, and
run over small shapes through every entry point (tests/c/sanitize_driver.cpp).
No recovery: any report ends the driver with a non-zero status.  Host code
only; nothing here touches a GPU."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
FLAGS = ["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
         "-fno-sanitize-recover=all"]


@pytest.mark.skipif(not (shutil.which("gcc") and shutil.which("g++")), reason="needs gcc and g++")
def test_generator_and_oracle_under_sanitizers(tmp_path):
    obj = str(tmp_path / "synth.o")
    exe = str(tmp_path / "drv")
    subprocess.check_call(["gcc", "-std=c11", *FLAGS, "-c", os.path.join(ROOT, "synth", "synth.c"),
                           "-o", obj])
    subprocess.check_call(["g++", "-std=c++17", *FLAGS, "-pthread",
                           os.path.join(ROOT, "oracle", "kvec_oracle.cpp"),
                           os.path.join(ROOT, "tests", "c", "sanitize_driver.cpp"), obj, "-lm",
                           "-o", exe])
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    assert r.stdout.strip() == "ok"
