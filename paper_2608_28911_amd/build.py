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
    """Compile every source (in parallel) and link libsemkv.so (always recompiles)."""
    from concurrent.futures import ThreadPoolExecutor
    os.makedirs(BUILD, exist_ok=True)
    cmds, objs = [], []
    for src, extra in SOURCES.items():
        obj = os.path.join(BUILD, src.replace(".hip", ".o"))
        cmds.append([HIPCC, "-c", os.path.join(CSRC, src), "-o", obj] + COMMON + extra)
        objs.append(obj)
    for cmd in cmds if verbose else ():
        print(" ".join(cmd), flush=True)
    with ThreadPoolExecutor(max_workers=min(len(cmds), os.cpu_count() or 1)) as ex:
        for f in [ex.submit(subprocess.check_call, cmd) for cmd in cmds]:
            f.result()
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
