"""The oracle and the library's host code under AddressSanitizer and
UndefinedBehaviorSanitizer (tests/sanitize_run.py): the CPU suite, which drives the
oracle and the library's host entry points, runs clean in a subprocess with the
instrumented builds."""
import os
import sys

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))

import sanitize_run  # noqa: E402


def test_cpu_suite_under_sanitizers():
    r = sanitize_run.run([])     # every CPU test but this one
    out = r.stdout + r.stderr
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
    assert r.returncode == 0, out[-4000:]
    assert " passed" in r.stdout, out[-2000:]
