"""Build libkl.so (the HIP library behind include/kl.h) for gfx950, and the
host library of the kernel-looping pass (looping/libklloop.so), in place."""
from __future__ import annotations

import os
import subprocess
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libkl.so")
SOURCES = [os.path.join(CSRC, f) for f in (
    "kl_step_d128.hip", "kl_step_d128_batched.hip", "kl_step_d64.hip", "kl_step_d64_batched.hip",
    "kl_device.hip", "kl_host.cpp")]
ARCH = "gfx950"

HIPCC_FLAGS = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    # no packed-fp32 instructions anywhere in the device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
]


def build(verbose: bool = False, jobs: int = 0) -> str:
    """Compile every translation unit (in parallel) and link libkl.so."""
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    objdir = os.path.join(HERE, "_build")
    os.makedirs(objdir, exist_ok=True)
    inc = ["-I", os.path.join(ROOT, "include"), "-I", CSRC]

    def compile_one(src):
        obj = os.path.join(objdir, os.path.basename(src) + ".o")
        cmd = [hipcc, *HIPCC_FLAGS, *inc, "-c", "-o", obj, src]
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.run(cmd, check=True)
        return obj

    jobs = jobs or min(len(SOURCES), os.cpu_count() or 1)
    with ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(compile_one, SOURCES))
    tmp = LIB + ".tmp"
    cmd = [hipcc, "-shared", "-fPIC", f"--offload-arch={ARCH}", "-o", tmp, *objs]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


LOOPING = os.path.join(HERE, "looping")
LOOPING_LIB = os.path.join(LOOPING, "libklloop.so")


def build_looping(verbose: bool = False) -> str:
    """Compile the kernel-looping pass (host C++17) into libklloop.so."""
    cxx = os.environ.get("CXX", "g++")
    tmp = LOOPING_LIB + ".tmp"
    cmd = [cxx, "-std=c++17", "-O2", "-fPIC", "-shared", "-Wall", "-Wextra", "-o", tmp,
           os.path.join(LOOPING, "kl_looping.cpp")]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LOOPING_LIB)
    return LOOPING_LIB


if __name__ == "__main__":
    print(build(verbose=True))
    print(build_looping(verbose=True))
