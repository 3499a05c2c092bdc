"""Build libsemkv.so (the C-ABI library of gfx950 HIP kernels) in-tree with hipcc.

Quantizer and ranker objects are compiled with -ffp-contract=off and IEEE
division/square root so their codes are bit-for-bit reproducible; all HIP code
is compiled with packed-fp32 instructions disabled.
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libsemkv.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

COMMON = ["-O3", "-std=c++17", "--offload-arch=gfx950", "-fPIC", "-fno-fast-math",
          "-fhip-fp32-correctly-rounded-divide-sqrt", "-fno-gpu-flush-denormals-to-zero",
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-Wall", "-Wno-unused-function",
          "-I", os.path.join(ROOT, "include"), "-I", CSRC]
SOURCES = {
    "semkv_api.hip": ["-ffp-contract=off"],
    "rank.hip": ["-ffp-contract=off"],
    "quant.hip": ["-ffp-contract=off"],
    "decode.hip": ["-fconstexpr-steps=33554432"],   # the compile-time checks of the 7-level tables
    "score.hip": ["-ffp-contract=off"],
}


def build(verbose: bool = False) -> str:
    """Compile every source and link libsemkv.so (always recompiles)."""
    os.makedirs(BUILD, exist_ok=True)
    objs = []
    for src, extra in SOURCES.items():
        obj = os.path.join(BUILD, src.replace(".hip", ".o"))
        cmd = [HIPCC, "-c", os.path.join(CSRC, src), "-o", obj] + COMMON + extra
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.check_call(cmd)
        objs.append(obj)
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [HIPCC, "-shared", "-fPIC", "--offload-arch=gfx950", "-o", tmp] + objs
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    build(verbose="-v" in sys.argv)
    print(LIB)
