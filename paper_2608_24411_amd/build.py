"""Build libresispec.so and the benchmark's read probe libresispec_probe.so (gfx950) in-tree
with hipcc."""
import os
import re
import subprocess
import sys
import tempfile

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


def _spills(report, scratch_users=None):
    """Functions whose registers spill to scratch memory, from the compiler's resource
    remarks: [(name, vgpr_spills, scratch_bytes_per_lane)].  Any VGPR spill counts.  A
    private segment without VGPR spills counts when the function's device assembly
    accesses scratch memory (scratch_users: the names of such functions), or whenever the
    assembly was not looked at (scratch_users None).  The register allocator sometimes
    reserves a frame that no instruction uses."""
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
        if m and name:
            used = scratch > 0 and (scratch_users is None or name in scratch_users)
            if int(m.group(1)) > 0 or used:
                bad.append((name, int(m.group(1)), scratch))
    return bad


_SCRATCH_OP = re.compile(r"^\s+(scratch_(load|store)|buffer_(load|store)|buffer_atomic)\w*\b")


def _scratch_users(asm_text):
    """Names of the functions of a device assembly listing whose instructions access
    scratch (private) memory."""
    users, name = set(), None
    for line in asm_text.splitlines():
        m = re.match(r"^([A-Za-z_][\w.$]*):", line)
        if m and not m.group(1).startswith(".L"):
            name = m.group(1)
            continue
        if name and _SCRATCH_OP.match(line):
            users.add(name)
    return users


def _compile(srcs, lib, verbose, extra=()):
    tmp = lib + ".tmp%d" % os.getpid()
    # -save-temps keeps the device assembly (in a scratch directory) for the scratch check
    cmd = ([HIPCC] + FLAGS + list(extra) + ["-Rpass-analysis=kernel-resource-usage", "-save-temps",
                                            "-I", os.path.join(ROOT, "include"), "-o", tmp] + srcs)
    if verbose:
        print(" ".join(cmd), flush=True)
    with tempfile.TemporaryDirectory() as work:
        r = subprocess.run(cmd, capture_output=True, text=True, cwd=work)
        asm = [os.path.join(work, f) for f in os.listdir(work)
               if f.endswith(".s") and "amdgcn" in f and "gfx950" in f]
        users = set()
        for path in asm:
            with open(path) as fh:
                users |= _scratch_users(fh.read())
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
    bad = _spills(r.stderr, users if asm else None)
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
