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
LIB_TIMELINE = os.path.join(HERE, "libsemkv_timeline.so")
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


REMARKS = "-Rpass-analysis=kernel-resource-usage"


def parse_remarks(text):
    """The compiler's kernel-resource-usage remarks in `text` as
    ({kernel: {field: value}}, [the other lines])."""
    usage, name, rest = {}, None, []
    for line in text.splitlines():
        if REMARKS not in line or "remark:" not in line:
            rest.append(line)
            continue
        field = line.split("remark:", 1)[1].replace("[" + REMARKS + "]", "").strip()
        key, _, val = field.partition(":")
        if key == "Function Name":
            name = val.strip()
            usage[name] = {}
        elif name is not None:
            usage[name][key.strip()] = val.strip()
    return usage, rest


def spilling(usage):
    """Kernels of `usage` that need private scratch memory."""
    return sorted(k for k, u in usage.items() if u.get("ScratchSize [bytes/lane]", "0") != "0")


def _compile(cmd):
    """Run one hipcc compile; return its kernels' resource remarks and pass
    every other line of its output on."""
    r = subprocess.run(cmd, capture_output=True, text=True)
    usage, rest = parse_remarks(r.stdout + r.stderr)
    if rest:
        print("\n".join(rest), file=sys.stderr, flush=True)
    if r.returncode:
        raise subprocess.CalledProcessError(r.returncode, cmd)
    return usage


def build(verbose: bool = False, timeline: bool = False, fine: bool = False) -> str:
    """Compile every source (in parallel) and link libsemkv.so (always recompiles).

    Fails when any kernel needs private scratch memory (register spills): every
    kernel here is written to fit the register file, and a spill would put
    per-lane stack traffic on the hot path.  The compiler's per-kernel figures
    (registers, LDS, scratch, occupancy) are written to resource_usage.txt
    beside the objects.

    timeline=True builds the tracing variant libsemkv_timeline.so instead: the
    decode kernel with its phase stamps compiled in (-DSEMKV_TIMELINE,
    include/semkv_timeline.h), objects under _build/timeline; fine=True adds
    the stamps inside the prologue and the first record (-DSEMKV_TIMELINE_FINE),
    which delay what they measure."""
    from concurrent.futures import ThreadPoolExecutor
    bdir = os.path.join(BUILD, "timeline") if timeline else BUILD
    lib_out = LIB_TIMELINE if timeline else LIB
    os.makedirs(bdir, exist_ok=True)
    cmds, objs = [], []
    for src, extra in SOURCES.items():
        obj = os.path.join(bdir, src.replace(".hip", ".o"))
        flag = (["-DSEMKV_TIMELINE"] + (["-DSEMKV_TIMELINE_FINE"] if fine else [])
                if timeline and src == "decode.hip" else [])
        cmds.append([HIPCC, "-c", os.path.join(CSRC, src), "-o", obj] + COMMON + extra + flag +
                    [REMARKS, "-fno-caret-diagnostics"])
        objs.append(obj)
    for cmd in cmds if verbose else ():
        print(" ".join(cmd), flush=True)
    with ThreadPoolExecutor(max_workers=min(len(cmds), os.cpu_count() or 1)) as ex:
        usage = {}
        for f in [ex.submit(_compile, cmd) for cmd in cmds]:
            usage.update(f.result())
    with open(os.path.join(bdir, "resource_usage.txt"), "w") as fh:
        for k in sorted(usage):
            fh.write("%s %s\n" % (k, " ".join("%s=%s" % (f.replace(" ", ""), v) for f, v in usage[k].items())))
    spills = spilling(usage)
    if not usage:
        raise RuntimeError("no resource remarks from the compiler")
    if spills and not timeline:
        raise RuntimeError("kernels with private scratch (register spills): %s" % spills)
    if spills:      # the tracing build's stamps take registers: its timings of these kernels are off
        print("tracing build: kernels with register spills: %s" % spills, file=sys.stderr)
    tmp = lib_out + ".tmp%d" % os.getpid()
    cmd = [HIPCC, "-shared", "-fPIC", "--offload-arch=gfx950", "-o", tmp] + objs
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd)
    os.replace(tmp, lib_out)
    return lib_out


if __name__ == "__main__":
    fine = "--timeline-fine" in sys.argv
    print(build(verbose="-v" in sys.argv, timeline=fine or "--timeline" in sys.argv, fine=fine))
