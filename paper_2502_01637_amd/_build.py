"""Compile libscone.so for gfx950 with hipcc (in-tree, no JIT cache)."""
import os
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libscone.so")
SOURCES = ["runtime.hip", "table_build.hip", "lookup.hip", "gather.hip", "embed.hip", "decode.hip",
           "gather_split.hip", "discover.hip", "fgram_model.hip", "pipeline.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"


def command(out):
    return ([HIPCC, "--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC", "-shared",
             "-Wall", "-Wno-unused-result",
             # no packed fp32 instructions anywhere in device code
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-I", os.path.join(ROOT, "include"), "-I", CSRC, "-o", out]
            + [os.path.join(CSRC, s) for s in SOURCES])


EXAMPLE_SRC = os.path.join(PKG, "examples", "scone_embed.c")
EXAMPLE = os.path.join(PKG, "examples", "scone_embed")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def example_command(out):
    """The plain-C example: C99 with gcc, the HIP runtime and libscone.so only."""
    return ["gcc", "-std=c99", "-O2", "-Wall", "-D__HIP_PLATFORM_AMD__",
            "-I", os.path.join(ROCM, "include"), "-I", os.path.join(ROOT, "include"),
            EXAMPLE_SRC, "-o", out, "-L", PKG, "-lscone", "-L", os.path.join(ROCM, "lib"),
            "-lamdhip64", "-Wl,-rpath,$ORIGIN/..", "-Wl,-rpath," + os.path.join(ROCM, "lib")]


def build(verbose: bool = False) -> str:
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = command(tmp)
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd)
    os.replace(tmp, LIB)
    tmp = EXAMPLE + ".tmp%d" % os.getpid()
    cmd = example_command(tmp)
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd)
    os.replace(tmp, EXAMPLE)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
