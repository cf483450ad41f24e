"""Build libresispec.so and the benchmark's read probe libresispec_probe.so (gfx950) in-tree
with hipcc."""
import os
import re
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


def _spills(report):
    """Functions whose registers spill to scratch memory, from the compiler's resource
    remarks: [(name, vgpr_spills, scratch_bytes_per_lane)]."""
    bad, name, scratch = [], None, 0
    for line in report.splitlines():
        m = re.search(r"Function Name: (\S+)", line)
        if m:
            name, scratch = m.group(1), 0
            continue
        m = re.search(r"ScratchSize \[bytes/lane\]: (\d+)", line)
        if m:
            scratch = int(m.group(1))
            continue
        m = re.search(r"VGPRs Spill: (\d+)", line)
        if m and name and (int(m.group(1)) > 0 or scratch > 0):
            bad.append((name, int(m.group(1)), scratch))
    return bad


def _compile(srcs, lib, verbose, extra=()):
    tmp = lib + ".tmp%d" % os.getpid()
    cmd = ([HIPCC] + FLAGS + list(extra) + ["-Rpass-analysis=kernel-resource-usage", "-I",
                                            os.path.join(ROOT, "include"), "-o", tmp] + srcs)
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    other = [l for l in r.stderr.splitlines()
             if "kernel-resource-usage" not in l and "packed-fp32-ops" not in l and l.strip()]
    if r.returncode != 0:
        sys.stderr.write("\n".join(other) + "\n")
        raise subprocess.CalledProcessError(r.returncode, cmd)
    if verbose and other:
        print("\n".join(other), flush=True)
    # A register spilled inside a branch that only some lanes take is stored for those
    # lanes alone; a value that other lanes still hold would come back from stale
    # scratch.  Every kernel is built to fit its registers, and the build checks it.
    bad = _spills(r.stderr)
    if bad:
        os.remove(tmp)
        raise RuntimeError("registers spill to scratch in: " +
                           ", ".join("%s (%d VGPRs, %d B/lane)" % b for b in bad))
    os.replace(tmp, lib)


# Host-side AddressSanitizer + UndefinedBehaviorSanitizer build of the same sources: the
# argument checks, host validator and size queries run instrumented (every -fsanitize
# flag is for the host pass only; the device code is built as usual).  Used by the
# sanitizer run of the CPU tests, never by the GPU path.
SAN_LIB = os.path.join(HERE, "libresispec_san.so")
SAN_FLAGS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
             "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer",
             "-Xarch_host", "-g"]


def build(verbose: bool = False) -> str:
    _compile(SRCS, LIB, verbose)
    _compile(PROBE_SRCS, PROBE_LIB, verbose)
    return LIB


def build_sanitized(verbose: bool = False) -> str:
    _compile(SRCS, SAN_LIB, verbose, extra=SAN_FLAGS)
    return SAN_LIB


if __name__ == "__main__":
    if "--sanitize" in sys.argv:
        build_sanitized(verbose="-v" in sys.argv)
    else:
        build(verbose="-v" in sys.argv)
