"""Build libbf1.so in-tree for gfx950.

    python -m paper_2608_20427_amd.build          # or __graft_entry__.build()

The device code is compiled by hipcc for gfx950 only; the C-ABI shim is plain
host C++ (g++ against the HIP runtime headers).  Packed FP32 VALU forms are
disabled in device code on purpose.
"""

import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libbf1.so")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
ARCH = "gfx950"

HIP_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
]
HOST_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-Wall", "-Wextra",
              f"-I{ROCM}/include", "-D__HIP_PLATFORM_AMD__"]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in r.stdout.splitlines() if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"build step failed ({r.returncode}): {' '.join(cmd)}\n{out}")
    if verbose and out.strip():
        print(out, flush=True)


def build(verbose=False, extra_hip_flags=()):
    hipcc = shutil.which("hipcc") or os.path.join(ROCM, "bin", "hipcc")
    gxx = shutil.which("g++") or "g++"
    os.makedirs(BUILD, exist_ok=True)
    k_obj = os.path.join(BUILD, "bf1_kernels.o")
    b_obj = os.path.join(BUILD, "bf1_bwd.o")
    d_obj = os.path.join(BUILD, "bf1_decode.o")
    a_obj = os.path.join(BUILD, "bf1_api.o")
    _run([hipcc, *HIP_FLAGS, *extra_hip_flags, "-c", os.path.join(CSRC, "bf1_kernels.hip"),
          "-o", k_obj], verbose)
    _run([hipcc, *HIP_FLAGS, *extra_hip_flags, "-c", os.path.join(CSRC, "bf1_bwd.hip"),
          "-o", b_obj], verbose)
    _run([hipcc, *HIP_FLAGS, *extra_hip_flags, "-c", os.path.join(CSRC, "bf1_decode.hip"),
          "-o", d_obj], verbose)
    _run([gxx, *HOST_FLAGS, "-c", os.path.join(CSRC, "bf1_api.cpp"), "-o", a_obj], verbose)
    tmp = LIB + ".tmp"
    _run([hipcc, f"--offload-arch={ARCH}", "-shared", "-fPIC", k_obj, b_obj, d_obj, a_obj, "-o", tmp,
          f"-L{ROCM}/lib", "-lamdhip64", f"-Wl,-rpath,{ROCM}/lib"], verbose)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
