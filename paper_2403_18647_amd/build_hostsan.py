"""Build libsdsat_hostsan.so: the host runtime (csrc/api.cpp) compiled by the host C++ compiler with
AddressSanitizer and UndefinedBehaviorSanitizer, linked with the ordinary kernel objects that
build.py compiled.  Only host code is instrumented; the CPU tests drive its argument checks and
size queries through the C-ABI in a process that preloads the sanitizer runtime."""
from __future__ import annotations

import os
import shutil
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libsdsat_hostsan.so")
KERNEL_OBJECTS = ["gemm.o", "attention.o", "verify.o", "misc.o", "prefill.o", "prefill_gemm.o", "noalloc.o"]
ROCM = "/opt/rocm"


def build() -> str:
    cxx = shutil.which("g++")
    if not cxx:
        raise RuntimeError("g++ not found")
    san = ["-fsanitize=address,undefined", "-fno-omit-frame-pointer"]
    obj = os.path.join(BUILD, "api_hostsan.o")
    src = os.path.join(HERE, "csrc", "api.cpp")
    cmd = [cxx, "-std=c++17", "-O1", "-g", "-fPIC", "-w", *san, "-D__HIP_PLATFORM_AMD__", f"-I{ROCM}/include",
           "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("host sanitizer compile failed:\n" + r.stdout + r.stderr)
    objs = [obj] + [os.path.join(BUILD, o) for o in KERNEL_OBJECTS]
    tmp = LIB + ".tmp"
    cmd = [cxx, "-shared", *san, *objs, f"-L{ROCM}/lib", "-lamdhip64", f"-Wl,-rpath,{ROCM}/lib", "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("host sanitizer link failed:\n" + r.stdout + r.stderr)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build())
