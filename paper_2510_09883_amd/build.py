"""Build the gfx950 HIP library libdelta_attn.so in-tree (hipcc, no PyTorch extension machinery).

    python -m paper_2510_09883_amd.build            # or __graft_entry__.build()
    python -m paper_2510_09883_amd.build --debug    # libdelta_attn_debug.so: device-side checks
    python -m paper_2510_09883_amd.build -DNAME=1   # extra compiler flags (build options)
"""
from __future__ import annotations

import concurrent.futures
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libdelta_attn.so")
DEBUG_LIB = os.path.join(PKG, "libdelta_attn_debug.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

SOURCES = ["attn_kernel.hip", "fused_delta_kernel.hip", "select_kernel.hip", "append_kernel.hip",
           "probe_kernel.hip", "noalloc.hip", "delta_api.cpp"]
FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-mcode-object-version=5",
    # no packed fp32 VALU instructions: scalar/float2 code is compiled to unpacked ops
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(ROOT, "include"),
    "-fvisibility=hidden", "-Wall", "-Wno-unused-function",
]


def _compile(src: str, obj: str, extra):
    cmd = [HIPCC, *FLAGS, *extra, "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return r.stderr


def build(verbose: bool = False, extra=(), debug: bool = False) -> str:
    """Compile every source for gfx950 and link the shared library. Returns its path.  With
    debug, the kernels check their device-side preconditions (-DDELTA_DEBUG=1) and the library
    is libdelta_attn_debug.so."""
    out_dir = os.path.join(PKG, "_build", "debug") if debug else os.path.join(PKG, "_build")
    lib = DEBUG_LIB if debug else LIB
    extra = list(extra) + (["-DDELTA_DEBUG=1"] if debug else [])
    os.makedirs(out_dir, exist_ok=True)
    objs = [os.path.join(out_dir, s.rsplit(".", 1)[0] + ".o") for s in SOURCES]
    with concurrent.futures.ThreadPoolExecutor(max_workers=len(SOURCES)) as ex:
        logs = list(ex.map(lambda so: _compile(so[0], so[1], list(extra)), zip(SOURCES, objs)))
    tmp = lib + ".tmp"
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, lib)
    if verbose:
        for s, log in zip(SOURCES, logs):
            if log.strip():
                print(f"--- {s}\n{log}", file=sys.stderr)
    return lib


if __name__ == "__main__":
    args = sys.argv[1:]
    dbg = "--debug" in args
    print(build(verbose=True, extra=[a for a in args if a != "--debug"], debug=dbg))
