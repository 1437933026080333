"""Builds libglide.so (the HIP kernels + C ABI) in-tree for gfx950.

Usage: ``python -m paper_2402_02082_amd.build`` or ``build()`` from Python.
"""

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libglide.so")
SOURCES = ["api.hip", "tree_attn.hip", "cape.hip", "verify.hip", "commit.hip", "rows_matmul.hip",
           "spec_sampling.hip"]

HIPCC_FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-shared",
    "-Wall",
    # keep the compiler from forming packed fp32 VALU ops
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def hipcc():
    path = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(path):
        raise RuntimeError("hipcc not found: the HIP library cannot be built")
    return path


LIB_ASAN = os.path.join(PKG, "libglide_asan.so")
# AddressSanitizer on the host code only (argument checks, planning, launch
# set-up); the GPU code is built as usual.
ASAN_FLAGS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fno-omit-frame-pointer", "-g"]


def build(verbose=False, asan=False):
    """Compile every source into paper_2402_02082_amd/libglide.so (always
    rebuilds); with asan=True into libglide_asan.so, host code instrumented
    with AddressSanitizer (load it with GLIDE_LIBRARY and the sanitizer
    runtime preloaded)."""
    lib = LIB_ASAN if asan else LIB
    tmp = lib + ".tmp"
    cmd = [hipcc(), *HIPCC_FLAGS, *(ASAN_FLAGS if asan else []), "-I", INCLUDE, "-I", CSRC,
           *[os.path.join(CSRC, s) for s in SOURCES], "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    err = "\n".join(l for l in res.stderr.splitlines() if noise not in l)
    if res.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + err)
    if verbose and err.strip():
        print(err, file=sys.stderr)
    os.replace(tmp, lib)
    return lib


if __name__ == "__main__":
    print(build(verbose=True, asan="--asan" in sys.argv[1:]))
