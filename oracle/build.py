"""Compile the fp64 CPU oracle (plain C, gcc) into oracle/liboracle.so, and on request an
AddressSanitizer + UndefinedBehaviorSanitizer build (clang, the runtime of ROCm's LLVM)
into oracle/liboracle_san.so.

Test infrastructure: the oracle checks the GPU library; it is never part of it.
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "resispec_oracle.c")
LIB = os.path.join(HERE, "liboracle.so")
SAN_LIB = os.path.join(HERE, "liboracle_san.so")
CLANG = os.environ.get("CLANG", "/opt/rocm/llvm/bin/clang")
SAN_FLAGS = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
             "-fno-omit-frame-pointer", "-g"]


def build(verbose: bool = False, sanitize: bool = False) -> str:
    lib = SAN_LIB if sanitize else LIB
    tmp = lib + ".tmp%d" % os.getpid()
    if sanitize:
        cmd = [CLANG, "-O1", "-std=c99", "-fPIC", "-shared", "-Wall", "-Wextra",
               "-ffp-contract=off"] + SAN_FLAGS + ["-o", tmp, SRC, "-lm"]
    else:
        cmd = ["gcc", "-O2", "-std=c99", "-fPIC", "-shared", "-Wall", "-Wextra",
               "-fno-fast-math", "-ffp-contract=off", "-o", tmp, SRC, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, lib)
    return lib


if __name__ == "__main__":
    build(verbose="-v" in sys.argv, sanitize="--sanitize" in sys.argv)
