"""The boundary is a C ABI: include/cheb.h compiles as strict C99 and a plain
C program links libcheb.so and runs its host-only calls (no GPU needed)."""
import os
import subprocess

import paper_2608_23429_amd as cheb

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)


def test_header_is_c99_and_library_links(tmp_path):
    exe = os.path.join(tmp_path, "c_abi_check")
    libdir = os.path.dirname(cheb.LIB_PATH)
    subprocess.run(["gcc", "-std=c99", "-Wall", "-Wextra", "-Werror", "-pedantic",
                    "-I", os.path.join(ROOT, "include"), os.path.join(HERE, "c_abi_check.c"),
                    "-o", exe, "-L", libdir, "-lcheb", f"-Wl,-rpath,{libdir}", "-lm"],
                   check=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0, r.stderr
    assert "c abi ok" in r.stdout
