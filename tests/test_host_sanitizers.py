"""The host-only C++ of libikv (session keys, the QueryMemory store, the trigger and
span resolution) built with g++ under AddressSanitizer and UndefinedBehaviorSanitizer
and driven by a random call sequence (tests/native/session_driver.cpp). CPU only."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ is not installed")
def test_session_code_under_sanitizers(tmp_path):
    exe = str(tmp_path / "session_driver")
    csrc = os.path.join(ROOT, "paper_2606_09916_amd", "csrc")
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=all", "-I", os.path.join(ROOT, "include"), "-I", csrc,
           os.path.join(csrc, "ikv_session.cpp"), os.path.join(ROOT, "tests", "native", "session_driver.cpp"),
           "-o", exe, "-pthread"]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300,
                       env={**os.environ, "ASAN_OPTIONS": "detect_leaks=1:abort_on_error=0"})
    assert r.returncode == 0, r.stdout + r.stderr
    assert "session driver: ok" in r.stdout
