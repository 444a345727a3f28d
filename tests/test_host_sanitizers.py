"""The C ABI's host code (layout builder, argument checks, launch planning)
built with the address and undefined-behaviour sanitizers and driven over
every layout kind, a sweep of shapes, the launch plans and every argument
error path (tests/sanitize/host_abi_check.cpp).  CPU only: the kernel
launchers are stubs the driver never reaches."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2112_00029_amd", "csrc")
SAN = os.path.join(ROOT, "tests", "sanitize")
ROCM = "/opt/rocm"

SOURCES = [os.path.join(CSRC, "layout.cpp"), os.path.join(CSRC, "capi.cpp"),
           os.path.join(SAN, "kernel_stubs.cpp"), os.path.join(SAN, "host_abi_check.cpp")]
FLAGS = ["-std=c++17", "-O1", "-g", "-fsanitize=address,undefined",
         "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer",
         "-D__HIP_PLATFORM_AMD__", f"-I{ROCM}/include", f"-I{ROOT}/include", f"-I{CSRC}", "-w"]


def test_host_abi_under_sanitizers(tmp_path):
    if shutil.which("g++") is None or not os.path.isdir(f"{ROCM}/include/hip"):
        pytest.skip("needs g++ and the HIP headers")
    objs = []
    procs = []
    for src in SOURCES:
        obj = str(tmp_path / (os.path.basename(src) + ".o"))
        objs.append(obj)
        procs.append(subprocess.Popen(["g++", *FLAGS, "-c", src, "-o", obj],
                                      stdout=subprocess.PIPE, stderr=subprocess.STDOUT))
    for p in procs:
        out = p.communicate()[0].decode()
        assert p.returncode == 0, out
    exe = str(tmp_path / "host_abi_check")
    r = subprocess.run(["g++", *FLAGS, *objs, f"-L{ROCM}/lib", "-lamdhip64",
                        f"-Wl,-rpath,{ROCM}/lib", "-o", exe], capture_output=True, text=True)
    assert r.returncode == 0, r.stdout + r.stderr
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    out = r.stdout + r.stderr
    print(out[-4000:])
    assert r.returncode == 0, out[-4000:]
    assert "0 failed expectations" in out
    assert "runtime error" not in out and "AddressSanitizer" not in out
