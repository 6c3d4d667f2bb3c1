"""The C ABI's CPU tests (tests/test_abi_cpu.py) once more, against a build of the library whose
host code -- argument checks, workspace layout, split planning, the layer driver, the
allocation-free step's checks, all of delta_api.cpp -- is compiled with AddressSanitizer: every
error path and size computation the CPU tests reach must be free of out-of-bounds accesses and
use-after-free.  The kernels are the release build's objects (host ASan says nothing about
device code); the library is built here with g++ from the committed sources and loaded through
the binding's DELTA_ATTN_LIB switch, with libasan preloaded into the child interpreter."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2510_09883_amd")
KERNEL_OBJS = ["attn_kernel.o", "fused_delta_kernel.o", "select_kernel.o", "append_kernel.o",
               "probe_kernel.o", "noalloc.o"]


def test_abi_cpu_tests_pass_with_host_address_sanitizer(tmp_path):
    gxx = shutil.which("g++")
    objs = [os.path.join(PKG, "_build", o) for o in KERNEL_OBJS]
    if gxx is None or not all(os.path.exists(o) for o in objs):
        pytest.skip("needs g++ and the release build's kernel objects (run the build first)")
    api_obj = str(tmp_path / "delta_api_asan.o")
    lib = str(tmp_path / "libdelta_attn_asan.so")
    subprocess.run([gxx, "-std=c++17", "-O1", "-g", "-fPIC", "-fsanitize=address",
                    "-fno-omit-frame-pointer", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
                    "-I", os.path.join(ROOT, "include"), "-c",
                    os.path.join(PKG, "csrc", "delta_api.cpp"), "-o", api_obj], check=True)
    subprocess.run([gxx, "-shared", "-fsanitize=address", *objs, api_obj, "-L/opt/rocm/lib",
                    "-lamdhip64", "-o", lib], check=True)
    libasan = subprocess.run([gxx, "-print-file-name=libasan.so"], capture_output=True,
                             text=True, check=True).stdout.strip()
    env = dict(os.environ, LD_PRELOAD=libasan, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               DELTA_ATTN_LIB=lib)
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_abi_cpu.py")],
                       env=env, capture_output=True, text=True, timeout=600, cwd=ROOT)
    assert r.returncode == 0, (r.stdout[-4000:] + r.stderr[-4000:])
    assert "AddressSanitizer" not in r.stderr
