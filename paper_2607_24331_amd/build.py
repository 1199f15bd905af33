"""Build libdckv.so in-tree for gfx950.

    python paper_2607_24331_amd/build.py

Host C++ (the C ABI and plan bookkeeping) is compiled with g++, kernels with
hipcc for gfx950, and everything is linked by hipcc into
paper_2607_24331_amd/libdckv.so.  Always rebuilds every object.
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
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libdckv.so")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
ARCH = "gfx950"

HOST_SOURCES = ["plan.cpp", "offline.cpp"]
HIP_SOURCES = ["append.hip", "decode.hip", "decode_mfma.hip", "dense.hip", "gram.hip", "rope.hip", "noalloc.hip", "decode_pass.hip"]

HIPCC_FLAGS = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    # keep the compiler from forming packed fp32 VALU instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
]
# Per-source extras.  The append GEMM keeps its MFMA accumulators in
# ordinary VGPRs: with the default AGPR form the register allocator rotated
# accumulators through AGPR copies inside the k loop, each copy waiting for
# an in-flight MFMA.
HIPCC_EXTRA = {"append.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"]}
HOST_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-D__HIP_PLATFORM_AMD__", "-Wall", "-Wextra"]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}\n{r.stdout}")
    out = "\n".join(l for l in r.stdout.splitlines() if "packed-fp32-ops" not in l
                    and "is not a recognized feature" not in l)
    if verbose and out.strip():
        print(out)


# Host code checked by AddressSanitizer and UndefinedBehaviorSanitizer (the
# kernels are built as usual); load it with DCKV_LIBRARY and the sanitizer
# runtime preloaded, e.g.
#   DCKV_LIBRARY=paper_2607_24331_amd/libdckv_sanitized.so \
#   LD_PRELOAD=$(g++ -print-file-name=libasan.so) ASAN_OPTIONS=detect_leaks=0 \
#   python -m pytest tests/test_lib_host.py tests/test_lib_offline_host.py
SANITIZE_FLAGS = ["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
                  "-fno-sanitize-recover=all"]
SANITIZED_LIB = os.path.join(PKG, "libdckv_sanitized.so")


def build(verbose: bool = False, sanitize: bool = False) -> str:
    hipcc = shutil.which("hipcc") or os.path.join(ROCM, "bin", "hipcc")
    os.makedirs(BUILD, exist_ok=True)
    objs = []
    for src in HOST_SOURCES:
        obj = os.path.join(BUILD, src + (".san.o" if sanitize else ".o"))
        flags = HOST_FLAGS + (SANITIZE_FLAGS if sanitize else [])
        _run(["g++", *flags, "-I", INCLUDE, "-I", CSRC, "-I", os.path.join(ROCM, "include"),
              "-c", os.path.join(CSRC, src), "-o", obj], verbose)
        objs.append(obj)
    for src in HIP_SOURCES:
        obj = os.path.join(BUILD, src + ".o")
        _run([hipcc, *HIPCC_FLAGS, *HIPCC_EXTRA.get(src, []), "-I", INCLUDE, "-I", CSRC, "-c",
              os.path.join(CSRC, src), "-o", obj], verbose)
        objs.append(obj)
    lib = SANITIZED_LIB if sanitize else LIB
    tmp = lib + ".tmp"
    if sanitize:   # g++ links the sanitizer runtimes its host objects were built for
        _run(["g++", "-shared", "-fPIC", *SANITIZE_FLAGS, "-o", tmp, *objs,
              "-L", os.path.join(ROCM, "lib"), "-lamdhip64", f"-Wl,-rpath,{os.path.join(ROCM, 'lib')}"],
             verbose)
    else:
        _run([hipcc, "-shared", "-fPIC", f"--offload-arch={ARCH}", "-o", tmp, *objs], verbose)
    os.replace(tmp, lib)
    return lib


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv, sanitize="--sanitize" in sys.argv))
