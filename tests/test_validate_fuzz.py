"""The C ABI's host-side argument validation under the address and undefined-
behaviour sanitizers: tests/native/validate_fuzz.cpp is built with g++ together
with csrc/moe_validate.cpp (plain C++, no GPU) and run on 200000 random and edge
argument sets."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(ROOT, "paper_2606_21712_amd", "csrc")


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_validation_under_sanitizers(tmp_path):
    exe = str(tmp_path / "validate_fuzz")
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-I", CSRC, os.path.join(HERE, "native", "validate_fuzz.cpp"), os.path.join(CSRC, "moe_validate.cpp"),
           "-o", exe]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0", UBSAN_OPTIONS="halt_on_error=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, r.stderr[-2000:]
    assert "no failures" in r.stdout
