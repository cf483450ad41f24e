"""Host logic of bench.py: the profile that supplies roofline.traffic stays matched to the
kernels only while their code is unchanged (comments and white space aside)."""
import json

import pytest

import bench


@pytest.fixture
def sources(tmp_path, monkeypatch):
    a, b = tmp_path / "k.hip", tmp_path / "k.h"
    monkeypatch.setattr(bench, "KERNEL_SRCS", [str(a), str(b)])
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    return a, b


def test_kernel_hash_ignores_comments_only(sources):
    a, b = sources
    a.write_text("int f(int x) {  // the row\n    return x + 1; /* one\n more */ }\n")
    b.write_text("#define K 4\n")
    h0 = bench.kernel_source_hash()
    a.write_text("// another comment\nint f(int x) {\n  return x + 1;\n}\n")
    assert bench.kernel_source_hash() == h0
    a.write_text("int f(int x) { return x + 2; }\n")
    assert bench.kernel_source_hash() != h0
    a.write_text("int f(int x) { return x + 1; }\n")
    b.write_text("#define K 5\n")
    assert bench.kernel_source_hash() != h0


def test_measured_traffic_needs_a_matching_profile(sources, tmp_path):
    a, b = sources
    a.write_text("int f();\n")
    b.write_text("\n")
    wl, mode = "wide-b128-n33-v128256-bf16", "resispec"
    assert bench.measured_traffic(wl, mode) is None   # no profile
    prof = tmp_path / "profiles"
    prof.mkdir()
    rec = {"kernel_source_sha256": bench.kernel_source_hash(), "hbm_bytes_per_launch": 1.5e9}
    path = prof / ("traffic_rs_decide_kernel_%s_%s.json" % (wl, mode))
    path.write_text(json.dumps(rec))
    assert bench.measured_traffic(wl, mode) == 1.5e9
    a.write_text("int f(); int g();\n")                # the kernel changed since the counters
    assert bench.measured_traffic(wl, mode) is None
