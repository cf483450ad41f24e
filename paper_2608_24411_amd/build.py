"""Build libresispec.so and the benchmark's read probe libresispec_probe.so (gfx950) in-tree
with hipcc."""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SRCS = [os.path.join(HERE, "csrc", "resispec.hip"), os.path.join(HERE, "csrc", "draft.hip")]
LIB = os.path.join(HERE, "libresispec.so")
# the benchmark's read-bandwidth probe, a library of its own
PROBE_SRCS = [os.path.join(HERE, "csrc", "probe.hip")]
PROBE_LIB = os.path.join(HERE, "libresispec_probe.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-Wall", "-Wno-unused-function",
    # packed fp32 instructions stay off: ordinary fp32 code only
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def _compile(srcs, lib, verbose):
    tmp = lib + ".tmp%d" % os.getpid()
    cmd = [HIPCC] + FLAGS + ["-I", os.path.join(ROOT, "include"), "-o", tmp] + srcs
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, lib)


def build(verbose: bool = False) -> str:
    _compile(SRCS, LIB, verbose)
    _compile(PROBE_SRCS, PROBE_LIB, verbose)
    return LIB


if __name__ == "__main__":
    build(verbose="-v" in sys.argv)
