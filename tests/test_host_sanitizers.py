"""The host codec under AddressSanitizer and UndefinedBehaviorSanitizer (CPU).

tests/native/host_fuzz.cpp drives codebook building, encoding (into buffers of
exactly the reported size) and validation of intact and damaged containers of
all three formats; here it is compiled together with the library's host
source, with both sanitizers, and run. Any out-of-bounds access, leak or
undefined operation aborts it with a report."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = [os.path.join(ROOT, "tests", "native", "host_fuzz.cpp"),
       os.path.join(ROOT, "paper_2502_00922_amd", "csrc", "host_codec.cpp")]


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_host_codec_under_sanitizers(tmp_path):
    exe = str(tmp_path / "host_fuzz")
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=undefined", "-I", os.path.join(ROOT, "include"),
           "-I", os.path.join(ROOT, "paper_2502_00922_amd", "csrc"), *SRC, "-o", exe, "-pthread"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([exe, "80"], capture_output=True, text=True, env=env, timeout=600)
    assert r.returncode == 0, (r.stdout + r.stderr)[-4000:]
    assert "0 failures" in r.stdout
