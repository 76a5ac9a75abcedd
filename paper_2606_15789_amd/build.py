"""Compile libwc.so (host C++ + HIP decode kernel for gfx950) in place."""

from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libwc.so")
SOURCES = [os.path.join(CSRC, "wc_host.cpp"), os.path.join(CSRC, "wc_decode.hip"),
           os.path.join(CSRC, "wc_decode_wide.hip"), os.path.join(CSRC, "wc_gemm.hip"),
           os.path.join(CSRC, "wc_gemm_wide.hip"), os.path.join(CSRC, "wc_gemm_wide_bf16.hip"),
           os.path.join(CSRC, "wc_encode.hip"), os.path.join(CSRC, "wc_stream.hip")]
HEADERS = [os.path.join(CSRC, "wc_internal.h"), os.path.join(CSRC, "wc_decoder.h"),
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


# Fingerprints of the decode kernels' gfx950 code, written next to the library
# by every build: the hash of each kernel's assembly with comments and label
# numbers taken out.  Measurements taken on one kernel (counter runs) name the
# fingerprint they were taken on, so they can tell when that kernel changed,
# whatever else changed in its source file.
KERNELS = os.path.join(HERE, "libwc.kernels.json")
KERNEL_SOURCES = [os.path.join(CSRC, "wc_decode.hip"), os.path.join(CSRC, "wc_decode_wide.hip"),
                  os.path.join(CSRC, "wc_gemm.hip"), os.path.join(CSRC, "wc_gemm_wide.hip"),
                  os.path.join(CSRC, "wc_gemm_wide_bf16.hip"), os.path.join(CSRC, "wc_stream.hip")]


def kernel_fingerprints(asm: str) -> dict:
    import hashlib
    import re
    out = {}
    for m in re.finditer(r"^(_Z\w+):", asm, re.M):
        name = m.group(1)
        end = asm.find(".Lfunc_end", m.end())
        if end < 0:
            continue
        lines = []
        for line in asm[m.end():end].splitlines():
            line = line.split(";")[0].strip()
            if not line:
                continue
            lines.append(re.sub(r"\.LBB\d+_", ".LBB_", line))
        out[name] = hashlib.sha256("\n".join(lines).encode()).hexdigest()[:16]
    return out


# A plain-C client of the ABI (no Python), built next to the library.
EXAMPLE_SRC = os.path.join(CSRC, "wc_example.c")
EXAMPLE = os.path.join(HERE, "wc_example")


def build_example() -> str:
    rocm = os.path.dirname(os.path.dirname(os.path.realpath(HIPCC)))
    cmd = ["gcc", "-std=c99", "-O2", "-Wall", "-D__HIP_PLATFORM_AMD__",
           f"-I{rocm}/include", EXAMPLE_SRC, "-o", EXAMPLE + ".tmp", f"-L{HERE}", "-lwc",
           f"-L{rocm}/lib", "-lamdhip64", "-lm", "-Wl,-rpath,$ORIGIN", f"-Wl,-rpath,{rocm}/lib"]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError("C example build failed: " + " ".join(cmd))
    os.replace(EXAMPLE + ".tmp", EXAMPLE)
    return EXAMPLE


def build(verbose: bool = False) -> str:
    import json
    import tempfile
    tmp = LIB + f".tmp{os.getpid()}"
    cmd = [HIPCC] + FLAGS + SOURCES + ["-o", tmp]
    with tempfile.TemporaryDirectory() as td:
        jobs = []
        for src in KERNEL_SOURCES:
            asm = os.path.join(td, os.path.basename(src) + ".s")
            acmd = ([HIPCC] + [f for f in FLAGS if f not in ("-shared", "-lpthread")] +
                    ["--cuda-device-only", "-S", src, "-o", asm])
            jobs.append((asm, acmd, subprocess.Popen(acmd, stdout=subprocess.PIPE,
                                                     stderr=subprocess.PIPE, text=True)))
        res = subprocess.run(cmd, capture_output=True, text=True)
        if res.returncode != 0:
            sys.stderr.write(res.stdout + res.stderr)
            raise RuntimeError("libwc build failed: " + " ".join(cmd))
        prints = {}
        for asm, acmd, ap in jobs:
            aout, aerr = ap.communicate()
            if ap.returncode != 0:
                sys.stderr.write(aout + aerr)
                raise RuntimeError("kernel assembly failed: " + " ".join(acmd))
            with open(asm) as fh:
                prints.update(kernel_fingerprints(fh.read()))
    if verbose:
        out = "\n".join(l for l in (res.stdout + res.stderr).splitlines()
                        if "packed-fp32-ops" not in l)
        if out.strip():
            print(out)
    with open(KERNELS + ".tmp", "w") as fh:
        json.dump(prints, fh, indent=1, sort_keys=True)
    os.replace(KERNELS + ".tmp", KERNELS)
    os.replace(tmp, LIB)
    build_example()
    return LIB


def ensure_example() -> str:
    """The C example, built (host code only, seconds) when it is missing."""
    ensure_built()
    if not os.path.exists(EXAMPLE):
        build_example()
    return EXAMPLE


def ensure_built() -> str:
    """Build only when nothing is built yet (tests and benches call this)."""
    if not os.path.exists(LIB):
        build()
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
