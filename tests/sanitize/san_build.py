"""Builds of the library's host code and of the oracle for AddressSanitizer and
UndefinedBehaviorSanitizer (CPU only, gcc).

``api.hip`` holds every check the C ABI makes before a launch: argument validation,
workspace layout, plan sizing and dispatch.  It is compiled here as C++ for the host
against ``hip/hip_runtime.h`` in this directory (a stand-in for the HIP runtime) and
linked with ``stubs.cpp``, whose kernel launchers do nothing.  The oracle is compiled
from its C source with the same sanitizers.  Loaded into an unsanitized Python, both
need the ASan runtime preloaded (``preload()`` names it).
"""
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
CSRC = os.path.join(ROOT, "paper_1906_07155_amd", "csrc")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
       "-fno-omit-frame-pointer", "-g", "-O1", "-fPIC", "-shared"]


def preload() -> str:
    """Path of gcc's ASan runtime."""
    return subprocess.check_output(["gcc", "-print-file-name=libasan.so"], text=True).strip()


def build_library(outdir: str) -> str:
    src = os.path.join(outdir, "api.cpp")
    shutil.copyfile(os.path.join(CSRC, "api.hip"), src)
    out = os.path.join(outdir, "libroi_extract_host.so")
    subprocess.check_call(["g++", "-std=c++17", *SAN, "-Wno-attributes",
                           "-I" + HERE, "-I" + CSRC, "-I" + os.path.join(ROOT, "include"),
                           src, os.path.join(HERE, "stubs.cpp"), "-Wl,--no-undefined", "-o", out])
    return out


def build_oracle(outdir: str) -> str:
    out = os.path.join(outdir, "liboracle_san.so")
    subprocess.check_call(["gcc", "-std=c99", "-ffp-contract=off", "-fno-fast-math",
                           "-fopenmp", *SAN, os.path.join(ROOT, "oracle", "roi_oracle.c"),
                           "-o", out, "-lm"])
    return out


if __name__ == "__main__":
    d = sys.argv[1] if len(sys.argv) > 1 else os.getcwd()
    print(build_library(d))
    print(build_oracle(d))
