"""The C ABI used from a plain C99 program on the GPU (no Python, no torch):
device memory from the HIP runtime's C API, pushes into the ring and
predictions, checked against the oracle inside the program."""
import os
import subprocess

import pytest

import oracle
import paper_2608_23429_amd as cheb
from tests.gpu_util import say

pytestmark = pytest.mark.gpu

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def test_c_program_on_the_gpu(tmp_path):
    exe = os.path.join(tmp_path, "c_gpu_check")
    libdir = os.path.dirname(cheb.LIB_PATH)
    odir = os.path.dirname(oracle.lib()._name)
    rocm_lib = os.path.join(ROCM, "lib")
    subprocess.run(["gcc", "-std=c99", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
                    "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROOT, "oracle"),
                    "-I", os.path.join(ROCM, "include"), os.path.join(HERE, "c_gpu_check.c"),
                    "-o", exe, "-L", libdir, "-lcheb", "-L", odir, "-loracle",
                    "-L", rocm_lib, "-lamdhip64", f"-Wl,-rpath,{libdir}", f"-Wl,-rpath,{odir}",
                    f"-Wl,-rpath,{rocm_lib}", "-lm"], check=True)
    say("c program: 6 pushes into a 5-entry ring, 4 predictions")
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    say(r.stdout.strip())
    assert r.returncode == 0, r.stdout + r.stderr
    assert "c gpu ok" in r.stdout
