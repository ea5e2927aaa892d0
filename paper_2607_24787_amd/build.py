"""Build libspp.so (gfx950 HIP kernels + host runtime) in-tree.

    python -m paper_2607_24787_amd.build        # or build() from Python

The kernels are compiled by hipcc for gfx950 only; the host runtime and the
replacement policy are plain C++ against the HIP runtime API.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libspp.so")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")

HIPCC = os.path.join(ROCM, "bin", "hipcc")
# Packed fp32 arithmetic is disabled for all device code.
DEVICE_FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
                "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
HOST_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-Wall", "-Wextra", "-D__HIP_PLATFORM_AMD__",
              "-I" + os.path.join(ROCM, "include")]


def _run(cmd):
    print("+", " ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)


def build(verbose: bool = True, sanitize: str = "") -> str:
    """Build libspp.so in the package.  sanitize "address" or "undefined":
    instead, build the host runtime (g++ objects only; the HIP kernels are
    compiled as usual) with that sanitizer into _build/<sanitize>/libspp.so,
    for CPU test runs that load it through SPP_LIB_PATH (with the sanitizer's
    runtime preloaded for ASan).  Returns the library's path."""
    out_dir = BUILD if not sanitize else os.path.join(BUILD, sanitize)
    os.makedirs(out_dir, exist_ok=True)
    inc = ["-I" + INCLUDE, "-I" + CSRC]
    objs = []
    for src in ("spp_kernels.hip", "spp_static.hip"):
        obj = os.path.join(out_dir, src.replace(".hip", ".o"))
        _run([HIPCC, *DEVICE_FLAGS, *inc, "-c", os.path.join(CSRC, src), "-o", obj])
        objs.append(obj)
    san = ["-fsanitize=" + sanitize, "-fno-omit-frame-pointer", "-fno-sanitize-recover=all", "-g"] if sanitize else []
    for src in ("spp_runtime.cpp", "spp_policy.cpp"):
        obj = os.path.join(out_dir, src.replace(".cpp", ".o"))
        _run(["g++", *HOST_FLAGS, *san, *inc, "-c", os.path.join(CSRC, src), "-o", obj])
        objs.append(obj)
    lib = LIB if not sanitize else os.path.join(out_dir, "libspp.so")
    tmp = lib + ".tmp"
    _run(["g++", "-shared", *san, "-o", tmp, *objs, "-L" + os.path.join(ROCM, "lib"), "-lamdhip64",
          "-Wl,-rpath," + os.path.join(ROCM, "lib")])
    shutil.move(tmp, lib)
    return lib


if __name__ == "__main__":
    build(sanitize=sys.argv[1] if len(sys.argv) > 1 else "")
    sys.exit(0)
