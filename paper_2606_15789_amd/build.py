"""Compile libwc.so (host C++ + HIP decode kernel for gfx950) in place."""

from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libwc.so")
SOURCES = [os.path.join(CSRC, "wc_host.cpp"), os.path.join(CSRC, "wc_decode.hip"),
           os.path.join(CSRC, "wc_encode.hip")]
HEADERS = [os.path.join(CSRC, "wc_internal.h"),
           os.path.join(os.path.dirname(HERE), "include", "wc.h")]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = os.environ.get("WC_OFFLOAD_ARCH", "gfx950")

FLAGS = ["-O3", "-std=c++20", "-fno-strict-aliasing", "-fPIC", "-shared",
         f"--offload-arch={ARCH}",
         # packed fp32 instructions stay off for every HIP object of this project
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wall", "-lpthread"]


def stale() -> bool:
    if not os.path.exists(LIB):
        return True
    t = os.path.getmtime(LIB)
    return any(os.path.getmtime(p) > t for p in SOURCES + HEADERS)


def build(verbose: bool = False) -> str:
    tmp = LIB + f".tmp{os.getpid()}"
    cmd = [HIPCC] + FLAGS + SOURCES + ["-o", tmp]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError("libwc build failed: " + " ".join(cmd))
    if verbose:
        out = "\n".join(l for l in (res.stdout + res.stderr).splitlines()
                        if "packed-fp32-ops" not in l)
        if out.strip():
            print(out)
    os.replace(tmp, LIB)
    return LIB


def ensure_built() -> str:
    """Build only when nothing is built yet (tests and benches call this)."""
    if not os.path.exists(LIB):
        build()
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
