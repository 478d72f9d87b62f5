"""Build the sanitizer driver of the C ABI: tm_api.cpp (the host side of the
library) and host_abi_driver.cpp compiled by g++ with AddressSanitizer and
UndefinedBehaviorSanitizer into one executable, which takes the device
kernels' launchers from the built libtm.so. Host code only: the kernels are
not instrumented.

    python tests/sanitize/build.py
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
PKG = os.path.join(ROOT, "paper_2506_03099_amd")
DRIVER = os.path.join(HERE, "host_abi_driver")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")

SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer"]
CXXFLAGS = ["-std=c++17", "-O1", "-g", "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROCM, "include"),
            "-I", os.path.join(ROOT, "include"), "-I", os.path.join(PKG, "csrc")]


def build(verbose: bool = False) -> str:
    if not os.path.exists(os.path.join(PKG, "libtm.so")):
        raise RuntimeError("libtm.so must be built first")
    objs = []
    for src in (os.path.join(PKG, "csrc", "tm_api.cpp"), os.path.join(HERE, "host_abi_driver.cpp")):
        obj = os.path.join(HERE, os.path.basename(src) + ".o")
        cmd = ["g++", *CXXFLAGS, *SAN, "-c", src, "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.run(cmd, check=True)
        objs.append(obj)
    cmd = ["g++", *SAN, *objs, "-L", PKG, "-ltm", "-L", os.path.join(ROCM, "lib"), "-lamdhip64",
           "-Wl,-rpath," + PKG, "-Wl,-rpath," + os.path.join(ROCM, "lib"), "-o", DRIVER]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    for obj in objs:
        os.remove(obj)
    return DRIVER


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
