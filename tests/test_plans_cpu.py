"""Host-side checks of the library's launch plans (tests/plan_check.cpp): workspace sizing of the
attention split partials and residual-GEMM partial tiles for every plan a call can make, and the
plan properties block-size invariance rests on (a fixed key partition and fixed contraction slices
whatever the block rows), and the prefill launches' refusal of arguments their kernels do not
handle.  Compiled with the host compiler against the built library; no device."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
PKG = os.path.join(ROOT, "paper_2403_18647_amd")
LIB = os.path.join(PKG, "libsdsat.so")
ROCM = "/opt/rocm"


@pytest.mark.skipif(not os.path.exists(LIB) or shutil.which("g++") is None, reason="library or g++ missing")
def test_launch_plans(tmp_path):
    exe = str(tmp_path / "plan_check")
    cmd = ["g++", "-std=c++17", "-O1", "-w", "-D__HIP_PLATFORM_AMD__", f"-I{ROCM}/include",
           f"-I{os.path.join(PKG, 'csrc')}", os.path.join(HERE, "plan_check.cpp"), LIB,
           f"-Wl,-rpath,{PKG}", f"-L{ROCM}/lib", "-lamdhip64", f"-Wl,-rpath,{ROCM}/lib", "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stdout + r.stderr
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0 and r.stdout.strip().endswith("ok (0 failed)"), r.stdout[-3000:] + r.stderr[-2000:]
