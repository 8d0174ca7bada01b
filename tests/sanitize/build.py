"""Builds the host-only sanitizer variant of the C ABI:

    python tests/sanitize/build.py OUT.so

csrc/api.cpp with the launchers replaced by launch_stubs.cpp, compiled by the
host compiler with AddressSanitizer and UndefinedBehaviorSanitizer (no device
code, so no GPU sanitizer is involved).  tests/test_sanitize.py runs the ABI
tests against it."""

from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
CSRC = os.path.join(ROOT, "paper_2505_22918_amd", "csrc")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def command(out):
    return ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-fPIC", "-shared",
            "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
            "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROCM, "include"), "-I", os.path.join(ROOT, "include"),
            "-I", CSRC, os.path.join(CSRC, "api.cpp"), os.path.join(HERE, "launch_stubs.cpp"), "-o", out]


def build(out):
    res = subprocess.run(command(out), capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"sanitizer build failed:\n{res.stdout}{res.stderr}")
    return out


if __name__ == "__main__":
    print(build(sys.argv[1]))
