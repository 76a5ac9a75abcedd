"""The library's host code and the oracle under AddressSanitizer and
UndefinedBehaviorSanitizer (host only: gcc / g++, no device code).

tests/host_sanitizer_driver.cpp encodes seeded tensors of every dtype with
wc_encode and with the oracle (byte-identical blobs required), decodes them
with the oracle, and feeds wc_open truncated and bit-flipped blobs.  Any
out-of-bounds access, use after free, leak or undefined behaviour in either
aborts the driver.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_host_code_under_address_and_undefined_sanitizers(tmp_path):
    gcc, gxx = shutil.which("gcc"), shutil.which("g++")
    if not gcc or not gxx:
        pytest.skip("no host C/C++ compiler")
    san = ["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=all"]
    obj = str(tmp_path / "oracle.o")
    exe = str(tmp_path / "driver")
    subprocess.run([gcc, *san, "-std=c99", "-c", os.path.join(ROOT, "oracle", "wc_oracle.c"),
                    "-o", obj], check=True, capture_output=True, text=True)
    subprocess.run([gxx, *san, "-std=c++20", "-pthread",
                    os.path.join(ROOT, "paper_2606_15789_amd", "csrc", "wc_host.cpp"),
                    os.path.join(ROOT, "tests", "host_sanitizer_driver.cpp"), obj, "-lm",
                    "-o", exe], check=True, capture_output=True, text=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([exe], env=env, capture_output=True, text=True, timeout=900)
    assert r.returncode == 0, (r.stdout[-2000:], r.stderr[-4000:])
    assert "0 failures" in r.stdout
