"""The library's host code (weights, ring bookkeeping, tables, residual
planning, argument checks) built with g++ under AddressSanitizer and
UndefinedBehaviorSanitizer, with the device launchers replaced by stubs,
and driven by the C ABI test program.  CPU only."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(ROOT, "paper_2608_23429_amd", "csrc")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
HOST_SOURCES = ["api.cpp", "cache.cpp", "table.cpp", "residual.cpp"]


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_host_code_under_asan_ubsan(tmp_path):
    san = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
           "-fno-omit-frame-pointer", "-g", "-O1"]
    inc = ["-I", os.path.join(ROOT, "include"), "-I", CSRC, "-I", os.path.join(ROCM, "include")]
    objs = []
    for src in HOST_SOURCES + ["host_stubs.cpp"]:
        path = os.path.join(HERE if src == "host_stubs.cpp" else CSRC, src)
        obj = os.path.join(tmp_path, src + ".o")
        subprocess.run(["g++", "-std=c++17", "-D__HIP_PLATFORM_AMD__", *san, *inc, "-c", path,
                        "-o", obj], check=True)
        objs.append(obj)
    cobj = os.path.join(tmp_path, "c_abi_check.o")
    subprocess.run(["gcc", "-std=c99", *san, "-I", os.path.join(ROOT, "include"), "-c",
                    os.path.join(HERE, "c_abi_check.c"), "-o", cobj], check=True)
    exe = os.path.join(tmp_path, "c_abi_check_san")
    libdir = os.path.join(ROCM, "lib")
    subprocess.run(["g++", *san, cobj, *objs, "-o", exe, "-L", libdir, "-lamdhip64",
                    f"-Wl,-rpath,{libdir}", "-lm"], check=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([exe, os.path.join(tmp_path, "table.txt")], capture_output=True, text=True,
                       env=env, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "c abi ok" in r.stdout


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_host_code_under_tsan(tmp_path):
    """Eight threads call the host entry points at once (weights, tables,
    launch shape, error messages, a ring handle each) in a ThreadSanitizer
    build: no data race is reported and every result is as single-threaded."""
    san = ["-fsanitize=thread", "-fno-omit-frame-pointer", "-g", "-O1"]
    inc = ["-I", os.path.join(ROOT, "include"), "-I", CSRC, "-I", os.path.join(ROCM, "include")]
    objs = []
    for src in HOST_SOURCES + ["host_stubs.cpp", "host_threads.cpp"]:
        path = os.path.join(HERE if src.startswith("host_") else CSRC, src)
        obj = os.path.join(tmp_path, src + ".o")
        subprocess.run(["g++", "-std=c++17", "-D__HIP_PLATFORM_AMD__", *san, *inc, "-c", path,
                        "-o", obj], check=True)
        objs.append(obj)
    exe = os.path.join(tmp_path, "host_threads_tsan")
    libdir = os.path.join(ROCM, "lib")
    subprocess.run(["g++", *san, *objs, "-o", exe, "-L", libdir, "-lamdhip64",
                    f"-Wl,-rpath,{libdir}", "-lm", "-pthread"], check=True)
    env = dict(os.environ, TSAN_OPTIONS="halt_on_error=1:second_deadlock_stack=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "threads ok" in r.stdout
    assert "WARNING: ThreadSanitizer" not in r.stderr, r.stderr


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_failed_push_leaves_no_half_written_entry(tmp_path):
    """A copy push into a full ring whose second segment-copy launch fails
    (host stubs that let a set number of launches succeed): the history no
    longer lists the entry being overwritten, predictions report NOTREADY,
    and the next push reuses the slot.  Under ASan and UBSan, CPU only."""
    san = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
           "-fno-omit-frame-pointer", "-g", "-O1"]
    inc = ["-I", os.path.join(ROOT, "include"), "-I", CSRC, "-I", os.path.join(ROCM, "include")]
    objs = []
    for src in HOST_SOURCES + ["host_stubs.cpp"]:
        path = os.path.join(HERE if src == "host_stubs.cpp" else CSRC, src)
        obj = os.path.join(tmp_path, src + ".o")
        subprocess.run(["g++", "-std=c++17", "-D__HIP_PLATFORM_AMD__", *san, *inc, "-c", path,
                        "-o", obj], check=True)
        objs.append(obj)
    cobj = os.path.join(tmp_path, "push_failure_check.o")
    subprocess.run(["gcc", "-std=c99", *san, "-I", os.path.join(ROOT, "include"), "-c",
                    os.path.join(HERE, "push_failure_check.c"), "-o", cobj], check=True)
    exe = os.path.join(tmp_path, "push_failure_check")
    libdir = os.path.join(ROCM, "lib")
    subprocess.run(["g++", *san, cobj, *objs, "-o", exe, "-L", libdir, "-lamdhip64",
                    f"-Wl,-rpath,{libdir}", "-lm"], check=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "push failure ok" in r.stdout
