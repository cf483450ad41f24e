"""The C ABI on the host: the library loads, exports every symbol the header declares,
and its host-only entry points and argument checks behave as documented.  No device
compute is launched here (every call below returns before any launch)."""
import ctypes
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER_DIR = os.path.join(ROOT, "include")


def _declared_functions():
    names = set()
    for fn in os.listdir(HEADER_DIR):
        if not fn.endswith(".h"):
            continue
        text = open(os.path.join(HEADER_DIR, fn)).read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        for m in re.finditer(r"^[A-Za-z_][\w \t\*]*?\b(resispec_\w+)\s*\(", text, flags=re.M):
            names.add(m.group(1))
    return names


@pytest.fixture(scope="module")
def native():
    from paper_2608_24411_amd import native
    return native


def test_library_exports_every_declared_symbol(native):
    declared = _declared_functions()
    assert declared, "no declarations found"
    assert declared == set(native.EXPORTS)
    for name in declared:
        assert hasattr(native.lib, name), name
        assert hasattr(native, name), name     # binding has the same names


def test_abi_version_and_status_strings(native):
    assert native.resispec_abi_version() == 3
    for code in range(5):
        s = native.resispec_status_string(code)
        assert s.startswith("RS_")
    assert "unknown" in native.resispec_status_string(99)


def test_workspace_bytes(native):
    assert native.resispec_workspace_bytes(0, 5) == 0
    assert native.resispec_workspace_bytes(5, 0) == 0
    for B, N in ((1, 1), (128, 33), (1024, 26), (3, 7)):
        w = native.resispec_workspace_bytes(B, N)
        assert w >= 3 * 4 * B * N
        assert w % 256 == 0


def test_validate_tree_host(native):
    parent = np.array([[-1, 0, 0, 1, 1], [-1, 0, 1, 2, 3]], dtype=np.int32)
    tok = np.array([[0, 1, 2, 3, 4], [0, 5, 6, 7, 8]], dtype=np.int32)
    assert native.resispec_validate_tree_host(parent, tok, 16) == (native.RS_OK, -1)
    bad = parent.copy()
    bad[1, 3] = 3
    assert native.resispec_validate_tree_host(bad, tok, 16) == (native.RS_ERR_INVALID_ARG, 8)
    bad = parent.copy()
    bad[0, 0] = 0
    assert native.resispec_validate_tree_host(bad, tok, 16) == (native.RS_ERR_INVALID_ARG, 0)
    badtok = tok.copy()
    badtok[1, 4] = 16
    assert native.resispec_validate_tree_host(parent, badtok, 16) == (native.RS_ERR_INVALID_ARG, 9)
    star = np.zeros((1, 66), dtype=np.int32)
    star[0, 0] = -1
    assert native.resispec_validate_tree_host(star, np.zeros((1, 66), np.int32), 4)[0] == \
        native.RS_ERR_INVALID_ARG
    assert native.resispec_validate_tree_host(star[:, :65], np.zeros((1, 65), np.int32), 4)[0] == \
        native.RS_OK


def _prm(native, mode=0, dtype=0, T=1.0):
    return native.RsParams(mode, dtype, T, 0, 1)


def test_argument_errors_return_before_launch(native):
    lib = native.lib
    fake = ctypes.c_void_p(0x1000)   # never dereferenced: every call below fails validation
    i32p = ctypes.c_void_p(0x2000)
    ok = _prm(native)
    # flat verify
    assert lib.resispec_verify(fake, fake, i32p, fake, fake, 4, 100, 2, None, i32p, i32p, None,
                               None) == native.RS_ERR_INVALID_ARG
    for bad in (_prm(native, mode=7), _prm(native, dtype=5), _prm(native, T=0.0),
                _prm(native, T=-1.0), _prm(native, T=float("inf"))):
        assert lib.resispec_verify(fake, fake, i32p, fake, fake, 4, 100, 2, ctypes.byref(bad),
                                   i32p, i32p, None, None) == native.RS_ERR_INVALID_ARG
    assert lib.resispec_verify(None, fake, i32p, fake, fake, 4, 100, 2, ctypes.byref(ok), i32p,
                               i32p, None, None) == native.RS_ERR_INVALID_ARG
    assert lib.resispec_verify(fake, fake, i32p, fake, fake, 4, 0, 2, ctypes.byref(ok), i32p,
                               i32p, None, None) == native.RS_ERR_INVALID_ARG
    assert lib.resispec_verify(fake, fake, i32p, fake, fake, 4, 100, 65, ctypes.byref(ok), i32p,
                               i32p, None, None) == native.RS_ERR_UNSUPPORTED
    assert lib.resispec_verify(fake, fake, i32p, fake, fake, 4, (1 << 22) + 1, 2, ctypes.byref(ok),
                               i32p, i32p, None, None) == native.RS_ERR_UNSUPPORTED
    # B = 0 is a no-op
    assert lib.resispec_verify(None, None, None, None, None, 0, 100, 2, ctypes.byref(ok), None,
                               None, None, None) == native.RS_OK
    # tree verify
    args = [fake, fake, i32p, i32p, fake, fake]
    assert lib.resispec_verify_tree(*args, 4, 5, 100, 2, ctypes.byref(ok), i32p, i32p, None,
                                    None, 0, None) == native.RS_ERR_WORKSPACE
    ws = native.resispec_workspace_bytes(4, 5)
    assert lib.resispec_verify_tree(*args, 4, 5, 100, 2, ctypes.byref(ok), i32p, i32p, None,
                                    ctypes.c_void_p(0x10000), ws - 1, None) == native.RS_ERR_WORKSPACE
    assert lib.resispec_verify_tree(*args, 4, 0, 100, 2, ctypes.byref(ok), i32p, i32p, None,
                                    fake, ws, None) == native.RS_ERR_INVALID_ARG
    assert lib.resispec_verify_tree(*args, 4, 5, 100, -1, ctypes.byref(ok), i32p, i32p, None,
                                    fake, ws, None) == native.RS_ERR_INVALID_ARG
    assert lib.resispec_verify_tree(fake, None, i32p, i32p, fake, fake, 4, 5, 100, 2,
                                    ctypes.byref(ok), i32p, i32p, None, fake, ws,
                                    None) == native.RS_ERR_INVALID_ARG
    # deferred draws: the larger workspace, checked by every entry point of the schedule
    dws = native.resispec_deferred_workspace_bytes(4, 5)
    assert dws >= ws + 4 * 5 * 2 * 128 * 8
    wsp = ctypes.c_void_p(0x10000)
    assert lib.resispec_verify_tree_deferred(*args, 4, 5, 100, 2, ctypes.byref(ok), i32p, i32p,
                                             None, wsp, dws - 1, None) == native.RS_ERR_WORKSPACE
    assert lib.resispec_verify_tree_deferred(*args, 4, 5, 100, 2, ctypes.byref(ok), i32p, i32p,
                                             None, ctypes.c_void_p(0x10008), dws,
                                             None) == native.RS_ERR_WORKSPACE   # misaligned
    assert lib.resispec_decide_nodes(*args, 4, 5, 100, ctypes.byref(ok), wsp, ws,
                                     None) == native.RS_ERR_WORKSPACE
    assert lib.resispec_walk_draw(*args, 4, 5, 100, 2, ctypes.byref(ok), wsp, dws - 1, i32p, i32p,
                                  None, None) == native.RS_ERR_WORKSPACE
    assert lib.resispec_walk_draw(*args, 4, 5, 100, -1, ctypes.byref(ok), wsp, dws, i32p, i32p,
                                  None, None) == native.RS_ERR_INVALID_ARG
    assert lib.resispec_decide_nodes(*args, 4, 5, 100, ctypes.byref(_prm(native, T=0.0)), wsp,
                                     dws, None) == native.RS_ERR_INVALID_ARG
    assert lib.resispec_verify_tree_deferred(*args, 0, 5, 100, 2, ctypes.byref(ok), None, None,
                                             None, None, 0, None) == native.RS_OK   # B = 0
    assert native.resispec_deferred_workspace_bytes(0, 5) == 0
    assert native.resispec_deferred_workspace_bytes(5, 0) == 0
    assert lib.resispec_verify_tree(None, None, None, None, None, None, 0, 5, 100, 2,
                                    ctypes.byref(ok), None, None, None, None, 0,
                                    None) == native.RS_OK
    assert lib.resispec_verify_tree_debug(*args, 4, 5, 100, 2, ctypes.byref(ok), i32p, i32p, None,
                                          None, 0, None, None, None, None,
                                          None) == native.RS_ERR_INVALID_ARG
    # path schedule: same argument rules, no workspace
    assert lib.resispec_verify_tree_path(*args, 4, 0, 100, 2, ctypes.byref(ok), i32p, i32p, None,
                                         None) == native.RS_ERR_INVALID_ARG
    assert lib.resispec_verify_tree_path(*args, 4, 5, 100, -1, ctypes.byref(ok), i32p, i32p, None,
                                         None) == native.RS_ERR_INVALID_ARG
    assert lib.resispec_verify_tree_path(*args, 4, 5, (1 << 22) + 1, 2, ctypes.byref(ok), i32p,
                                         i32p, None, None) == native.RS_ERR_UNSUPPORTED
    assert lib.resispec_verify_tree_path(fake, fake, i32p, i32p, fake, fake, 4, 5, 100, 2,
                                         ctypes.byref(_prm(native, T=0.0)), i32p, i32p, None,
                                         None) == native.RS_ERR_INVALID_ARG
    assert lib.resispec_verify_tree_path(None, None, None, None, None, None, 0, 5, 100, 2,
                                         ctypes.byref(ok), None, None, None, None) == native.RS_OK
    # path schedule with row groups: group size and workspace are checked before launch
    pg = lib.resispec_verify_tree_path_group
    pws = native.resispec_path_workspace_bytes(4, 100)
    assert pws > 0 and native.resispec_path_workspace_bytes(0, 100) == 0
    assert native.resispec_path_workspace_bytes(4, 0) == 0
    # two cache rows per sequence, padded to 1024 elements, after the group states
    assert native.resispec_path_workspace_bytes(4, 1025) - pws == 4 * 2 * 1024 * 4
    wsp = ctypes.c_void_p(0x10000)
    for g in (-1, 17):
        assert pg(*args, 4, 5, 100, 2, ctypes.byref(ok), i32p, i32p, None, g, wsp, pws,
                  None) == native.RS_ERR_INVALID_ARG
    assert pg(*args, 4, 5, 100, 2, ctypes.byref(ok), i32p, i32p, None, 2, None, 0,
              None) == native.RS_ERR_WORKSPACE                     # members need a workspace
    assert pg(*args, 4, 5, 100, 2, ctypes.byref(ok), i32p, i32p, None, 0, wsp, pws - 1,
              None) == native.RS_ERR_WORKSPACE                     # too small
    assert pg(*args, 4, 5, 100, 2, ctypes.byref(ok), i32p, i32p, None, 0,
              ctypes.c_void_p(0x10008), pws, None) == native.RS_ERR_WORKSPACE   # misaligned
    assert pg(*args, 4, 0, 100, 2, ctypes.byref(ok), i32p, i32p, None, 0, wsp, pws,
              None) == native.RS_ERR_INVALID_ARG
    assert pg(None, None, None, None, None, None, 0, 5, 100, 2, ctypes.byref(ok), None, None,
              None, 0, None, 0, None) == native.RS_OK
    # all-nodes schedule with row groups
    tg = lib.resispec_verify_tree_group
    tws = native.resispec_tree_group_workspace_bytes(4, 5)
    assert tws > native.resispec_workspace_bytes(4, 5)
    assert native.resispec_tree_group_workspace_bytes(0, 5) == 0
    for g in (-1, 17):
        assert tg(*args, 4, 5, 100, 2, ctypes.byref(ok), i32p, i32p, None, g, wsp, tws,
                  None) == native.RS_ERR_INVALID_ARG
    assert tg(*args, 4, 5, 100, 2, ctypes.byref(ok), i32p, i32p, None, 0, None, 0,
              None) == native.RS_ERR_WORKSPACE
    assert tg(*args, 4, 5, 100, 2, ctypes.byref(ok), i32p, i32p, None, 0, wsp, tws - 1,
              None) == native.RS_ERR_WORKSPACE
    assert tg(None, None, None, None, None, None, 0, 5, 100, 2, ctypes.byref(ok), None, None,
              None, 0, None, 0, None) == native.RS_OK
    assert lib.resispec_tree_group_size(0, 5, 100, ctypes.byref(ok)) == -1
    assert lib.resispec_path_group_size(0, 100, ctypes.byref(ok)) == -1
    assert lib.resispec_path_group_size(4, 100, ctypes.byref(_prm(native, dtype=5))) == -1
    # draft step
    f32p = fake
    assert lib.resispec_draft_candidates(fake, i32p, 4, 5, 100, ctypes.byref(ok), 1, 0, None, f32p,
                                         f32p, None, None) == native.RS_ERR_INVALID_ARG
    assert lib.resispec_draft_candidates(fake, i32p, 4, 0, 100, ctypes.byref(ok), 1, 0, i32p,
                                         f32p, f32p, None, None) == native.RS_ERR_INVALID_ARG
    assert lib.resispec_draft_candidates(fake, i32p, 4, 5, (1 << 22) + 1, ctypes.byref(ok), 1, 0,
                                         i32p, f32p, f32p, None, None) == native.RS_ERR_UNSUPPORTED
    assert lib.resispec_draft_candidates(fake, i32p, 4, 5, 100, ctypes.byref(_prm(native, dtype=9)),
                                         1, 0, i32p, f32p, f32p, None,
                                         None) == native.RS_ERR_INVALID_ARG
    assert lib.resispec_draft_candidates(None, None, 0, 5, 100, ctypes.byref(ok), 1, 0, None, None,
                                         None, None, None) == native.RS_OK


def test_product_path_has_no_oracle_dependency():
    """The package and its native sources never reference the oracle."""
    pkg = os.path.join(ROOT, "paper_2608_24411_amd")
    for dirpath, _, files in os.walk(pkg):
        for fn in files:
            if fn.endswith((".py", ".hip", ".cpp", ".h")):
                text = open(os.path.join(dirpath, fn)).read()
                assert "oracle" not in text.lower(), os.path.join(dirpath, fn)


def test_read_probe_library_rejects_bad_arguments():
    """The benchmark's read probe (a library of its own) loads and checks its arguments
    before any launch."""
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2608_24411_amd", "libresispec_probe.so"))
    fn = lib.resispec_probe_read
    fn.restype = ctypes.c_int
    fn.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                   ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p]
    p = ctypes.c_void_p(4096)   # never dereferenced: every call below fails its checks
    q = 1 << 15                 # the chunk quantum (32 KiB)
    assert fn(None, 4 * q, q, 0, 1, p, None) == 1          # null source
    assert fn(p, 4 * q, q, 0, 1, None, None) == 1          # null sink
    assert fn(p, 0, q, 0, 1, p, None) == 1                 # empty buffer
    assert fn(p, 4 * q, q + 16, 0, 1, p, None) == 1        # chunk not a multiple of 32 KiB
    assert fn(p, 5 * q, 2 * q, 0, 1, p, None) == 1         # chunk does not divide the buffer
    assert fn(p, 4 * q, q, 2, 1, p, None) == 1             # unknown load policy
    assert fn(p, 4 * q, q, 0, 3, p, None) == 1             # unknown pass count


def test_build_rejects_register_spills():
    """The build's check of the compiler's resource remarks finds spilling functions."""
    from paper_2608_24411_amd import build
    report = "\n".join([
        "x.hip:1:1: remark: Function Name: k_ok [-Rpass-analysis=kernel-resource-usage]",
        "x.hip:1:1: remark:     VGPRs: 120 [-Rpass-analysis=kernel-resource-usage]",
        "x.hip:1:1: remark:     ScratchSize [bytes/lane]: 0 [-Rpass-analysis=kernel-resource-usage]",
        "x.hip:1:1: remark:     SGPRs Spill: 30 [-Rpass-analysis=kernel-resource-usage]",
        "x.hip:1:1: remark:     VGPRs Spill: 0 [-Rpass-analysis=kernel-resource-usage]",
        "x.hip:9:1: remark: Function Name: k_bad [-Rpass-analysis=kernel-resource-usage]",
        "x.hip:9:1: remark:     ScratchSize [bytes/lane]: 204 [-Rpass-analysis=kernel-resource-usage]",
        "x.hip:9:1: remark:     VGPRs Spill: 50 [-Rpass-analysis=kernel-resource-usage]",
        "x.hip:12:1: remark: Function Name: k_stack [-Rpass-analysis=kernel-resource-usage]",
        "x.hip:12:1: remark:     ScratchSize [bytes/lane]: 16 [-Rpass-analysis=kernel-resource-usage]",
        "x.hip:12:1: remark:     VGPRs Spill: 0 [-Rpass-analysis=kernel-resource-usage]",
    ])
    assert build._spills(report) == [("k_bad", 50, 204), ("k_stack", 0, 16)]
    # with the device assembly: a frame that no instruction uses is not a spill
    asm = "\n".join([
        "k_ok:", "\ts_load_dwordx4 s[4:7], s[0:1], 0x0", "\tglobal_load_dwordx4 v[0:3], v4, s[4:5]",
        "k_stack:", "\tv_mov_b32_e32 v1, 0", ".LBB2_1:", "\ts_endpgm",
        "k_bad:", "\tscratch_store_dword off, v7, s33 offset:4", "\tbuffer_load_dword v3, off, s[0:3], 0",
    ])
    users = build._scratch_users(asm)
    assert users == {"k_bad"}
    assert build._spills(report, users) == [("k_bad", 50, 204)]


def test_plain_c_caller(tmp_path):
    """The header is plain C: a C99 program built with gcc -Werror -pedantic against it and
    linked to the library calls its host-side functions and argument checks."""
    import shutil
    import subprocess
    from paper_2608_24411_amd import native
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("gcc not found")
    libdir = os.path.dirname(native.LIB_PATH)
    exe = str(tmp_path / "c_consumer")
    subprocess.run([gcc, "-std=c99", "-Wall", "-Wextra", "-Werror", "-pedantic", "-I", HEADER_DIR,
                    os.path.join(ROOT, "tests", "c_consumer.c"), "-o", exe, "-L", libdir,
                    "-lresispec", "-Wl,-rpath," + libdir], check=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0 and r.stdout.strip() == "ok", r.stdout + r.stderr
