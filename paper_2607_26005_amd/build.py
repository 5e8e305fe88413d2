"""Builds the HIP library libpictura.so for gfx950 (in-tree)."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(os.path.dirname(HERE), "include")
LIB = os.path.join(HERE, "libpictura.so")
SOURCES = ["pictura_binner.hip", "pictura_render.hip", "pictura_abi.hip"]
# (source, object name, extra flags): the render source is compiled three
# times.  One object holds only the production class/depth kernels, one the
# production instance and one-sample colour kernels, both scheduled by LLVM's
# iterative ILP strategy (1.4 % faster on the class/depth kernel, and 1.6 %
# and 2.5 % on the tile-shape-specialised instance and colour kernels, than
# the next best setting, in A/B runs with identical images); the antialiased
# kernel spills and slows under it, so it keeps the default scheduler.
UNITS = [(src, src.replace(".hip", ".o"), []) for src in SOURCES] + [
    ("pictura_render.hip", "pictura_render_plain.o",
     ["-DPICTURA_RENDER_PLAIN", "-mllvm", "-amdgpu-sched-strategy=iterative-ilp"]),
    ("pictura_render.hip", "pictura_render_side.o",
     ["-DPICTURA_RENDER_SIDE", "-mllvm", "-amdgpu-sched-strategy=iterative-ilp"]),
]

# fp32 rules need IEEE arithmetic: no contraction, correctly rounded division,
# denormals kept.  Packed fp32 instructions are disabled.
HIPCC_FLAGS = [
    "-O3", "-std=c++17", "--offload-arch=gfx950", "-fPIC",
    "-ffp-contract=off", "-fno-fast-math", "-fhip-fp32-correctly-rounded-divide-sqrt",
    "-fno-gpu-flush-denormals-to-zero",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
]


def build(verbose: bool = False) -> str:
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    objs = []
    procs = []
    for src, oname, extra in UNITS:
        obj = os.path.join(CSRC, oname)
        cmd = [hipcc, *HIPCC_FLAGS, *extra, "-I", INCLUDE, "-c", os.path.join(CSRC, src), "-o", obj]
        if verbose:
            print(" ".join(cmd))
        procs.append(subprocess.Popen(cmd))
        objs.append(obj)
    for p in procs:
        if p.wait() != 0:
            raise RuntimeError("hipcc failed")
    tmp = LIB + ".tmp"
    subprocess.check_call([hipcc, "--offload-arch=gfx950", "-shared", "-fPIC", "-Wl,--no-undefined", "-o", tmp, *objs])
    os.replace(tmp, LIB)
    for o in objs:
        os.remove(o)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
