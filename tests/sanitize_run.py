"""Run CPU tests with the oracle and the library's host code built with AddressSanitizer
and UndefinedBehaviorSanitizer (clang's runtimes from ROCm's LLVM, preloaded into the
interpreter; leak detection off, since the interpreter itself keeps allocations alive).

    python tests/sanitize_run.py                # the whole CPU suite
    python tests/sanitize_run.py tests/test_abi.py -k validate   # any pytest arguments

The instrumented libraries are oracle/liboracle_san.so and
paper_2608_24411_amd/libresispec_san.so (rebuilt when their sources are newer); the
loaders take them from RESISPEC_ORACLE_LIBRARY and RESISPEC_LIBRARY.  The device code in
the instrumented library is built as usual and never runs here: the CPU tests call only
the host paths (argument checks, the host validator, size queries, status strings)."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

CLANG = os.environ.get("CLANG", "/opt/rocm/llvm/bin/clang")


def _stale(lib, srcs):
    return not os.path.exists(lib) or any(os.path.getmtime(s) > os.path.getmtime(lib) for s in srcs)


def instrumented_env():
    """Build the instrumented libraries if needed; the environment that runs with them."""
    from oracle import build as ob
    from paper_2608_24411_amd import build as lb
    if _stale(ob.SAN_LIB, [ob.SRC, os.path.join(ROOT, "oracle", "resispec_oracle.h")]):
        ob.build(sanitize=True)
    srcs = lb.SRCS + [os.path.join(lb.HERE, "csrc", "common.h"),
                      os.path.join(ROOT, "include", "resispec.h")]
    if _stale(lb.SAN_LIB, srcs):
        lb.build_sanitized()
    runtime = subprocess.run([CLANG, "-print-file-name=libclang_rt.asan-x86_64.so"],
                             capture_output=True, text=True, check=True).stdout.strip()
    env = dict(os.environ)
    env.update(LD_PRELOAD=runtime, RESISPEC_LIBRARY=lb.SAN_LIB, RESISPEC_ORACLE_LIBRARY=ob.SAN_LIB,
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=0:halt_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    return env


def run(args):
    env = instrumented_env()
    cmd = [sys.executable, "-m", "pytest", "-p", "no:cacheprovider", "-q", "-x"]
    cmd += list(args) if args else ["tests", "-m", "not gpu", "--deselect",
                                    "tests/test_sanitize.py::test_cpu_suite_under_sanitizers"]
    return subprocess.run(cmd, env=env, cwd=ROOT, capture_output=True, text=True)


if __name__ == "__main__":
    r = run(sys.argv[1:])
    sys.stdout.write(r.stdout)
    sys.stderr.write(r.stderr)
    sys.exit(r.returncode)
