"""All-nodes verification with row groups (resispec_verify_tree_group): several
workgroups share every node row.  Tokens, lengths and statuses must equal the ordinary
all-nodes schedule's bit for bit (same chunks, slots and summation order), and the
oracle's walk on unflagged sequences."""
import numpy as np
import pytest
import torch

from paper_2608_24411_amd import synth
from parity_util import compare_walk, gpu_tree, host_tree, oracle_walk

pytestmark = pytest.mark.gpu
MODES = ("resispec", "specinfer")


def _log(*a):
    print(*a, flush=True)


def group_tree(native, w, mode, group, max_depth=None, bonus=True, workspace=None):
    md = w["max_depth"] if max_depth is None else max_depth
    t, l, s = native.resispec_verify_tree_group(
        w["target"], w["draft"], w["node_token"], w["parent"], w["u_accept"], w["u_resample"],
        temperature=w["temperature"], max_depth=md, mode=mode,
        without_replacement=w["without_replacement"], bonus=bonus, group_size=group,
        workspace=workspace)
    torch.cuda.synchronize()
    return {"tokens": t, "accepted_len": l, "status": s}


def same(a, b):
    for k in ("tokens", "accepted_len", "status"):
        if not torch.equal(a[k], b[k]):
            x, y = a[k].cpu().numpy(), b[k].cpu().numpy()
            rows = sorted(set(int(i) for i in np.argwhere(x != y)[:, 0]))
            for r in rows[:5]:
                _log("mismatch", k, "seq", r, x[r].tolist(), y[r].tolist())
            raise AssertionError("%s differs on %d sequences" % (k, len(rows)))


# few rows: B * N * group <= the device's resident workgroups
CASES = [(1, dict(B=2)), (2, dict(B=1)), (3, dict(B=1)), (4, dict(B=2)),
         (1, dict(B=1, V=32003)), (2, dict(B=1, V=100003, dtype="f32")),
         (3, dict(B=1, V=65537, dtype="bf16")), (4, dict(B=1, V=4099))]


@pytest.mark.parametrize("cfg,over", CASES, ids=[f"cfg{c}-{o}" for c, o in CASES])
@pytest.mark.parametrize("mode", MODES)
def test_row_groups_equal_all_nodes(gpu_lib, cfg, over, mode):
    w = synth.make_workload(cfg, device="cuda", **over)
    ref = gpu_tree(gpu_lib, w, mode)
    rows = w["B"] * w["N"]
    for g in (2, 3, 0):
        if g and rows * g > 256:
            continue
        _log("row groups", cfg, over, mode, g)
        same(group_tree(gpu_lib, w, mode, g), ref)
    h = host_tree(w)
    compare_walk(ref, oracle_walk(h, w, mode), h, w, mode)


def test_row_groups_fallback_and_faults(gpu_lib):
    """The exact-maximum pass (maxima exchanged between members) and faults, groups of 3."""
    w = synth.make_workload(2, device="cuda", B=2, V=40000)
    w["target"][:, 3, 39990] = 200.0
    w["target"][1, 0, 39000] = 150.0
    for mode in MODES:
        same(group_tree(gpu_lib, w, mode, 3), gpu_tree(gpu_lib, w, mode))
    f = synth.make_workload(1, device="cuda", B=3, V=3001)
    f["u_accept"][0, 1:5] = 0.999
    f["node_token"][1, 2] = 3001
    f["parent"][2, 7] = 9
    for mode in MODES:
        for bonus in (True, False):
            _log("row group faults", mode, bonus)
            same(group_tree(gpu_lib, f, mode, 3, bonus=bonus), gpu_tree(gpu_lib, f, mode, bonus=bonus))


def test_row_groups_unsupported_and_automatic(gpu_lib):
    """More members than a row has slots, or more workgroups than the device holds at
    once: an error before anything runs.  The automatic size falls back to the ordinary
    row kernel for large batches, with the same results."""
    w = synth.make_workload(4, device="cuda", B=1, V=512)    # one slot per row
    with pytest.raises(Exception):
        group_tree(gpu_lib, w, "resispec", 2)
    big = synth.make_workload(1, device="cuda", B=40, V=8192)   # 840 rows
    with pytest.raises(Exception):
        group_tree(gpu_lib, big, "resispec", 2)
    assert gpu_lib.resispec_tree_group_size(40, 21, 8192, dtype="f32") == 1
    same(group_tree(gpu_lib, big, "resispec", 0), gpu_tree(gpu_lib, big, "resispec"))


def test_row_groups_barrier_time_limit(gpu_lib):
    """Zero-tick barrier limit (testing hook): every workgroup ends; rows report status 8
    or finish with the reference result, and the default limit restores normal results."""
    w = synth.make_workload(2, device="cuda", B=1, V=40000)
    ref = gpu_tree(gpu_lib, w, "resispec")
    try:
        gpu_lib.resispec_debug_set_group_waits(barrier=0)
        g = group_tree(gpu_lib, w, "resispec", 4)
    finally:
        gpu_lib.resispec_debug_set_group_waits()
    st = g["status"].cpu().numpy()
    _log("statuses with a zero time limit", st.tolist())
    assert set(st.tolist()) <= {0, 8}
    done = st == 0
    assert np.array_equal(g["tokens"].cpu().numpy()[done], ref["tokens"].cpu().numpy()[done])
    same(group_tree(gpu_lib, w, "resispec", 4), ref)


def test_row_groups_full_batch_of_one(gpu_lib):
    """One tree of the benchmarked shape (33 rows of V = 128,256 bf16), automatic size,
    twice on one workspace."""
    w = synth.make_workload(2, device="cuda", B=1)
    ws = torch.empty(gpu_lib.resispec_tree_group_workspace_bytes(1, w["N"]), dtype=torch.uint8,
                     device="cuda")
    g = gpu_lib.resispec_tree_group_size(1, w["N"], w["V"], dtype="bf16")
    _log("automatic group for one tree:", g)
    assert g >= 2
    for mode in MODES:
        ref = gpu_tree(gpu_lib, w, mode)
        for _ in range(2):
            same(group_tree(gpu_lib, w, mode, 0, workspace=ws), ref)


def test_row_groups_formation_fallback(gpu_lib):
    """Zero-tick formation limit (testing hook): rows whose group is given up are verified
    by one workgroup alone, with the same outcomes; the default limit restores grouping."""
    w = synth.make_workload(4, device="cuda", B=2, V=40000)
    for mode in MODES:
        ref = gpu_tree(gpu_lib, w, mode)
        try:
            gpu_lib.resispec_debug_set_group_waits(formation=0)
            for g in (2, 4, 0):
                _log("row group with a zero formation limit", mode, g)
                same(group_tree(gpu_lib, w, mode, g), ref)
        finally:
            gpu_lib.resispec_debug_set_group_waits()
        same(group_tree(gpu_lib, w, mode, 4), ref)


def test_row_groups_automatic_size(gpu_lib):
    """The automatic size keeps to one workgroup per CU, eight members per row, 40 KiB of
    a row's logits per member and rows of at least 160 KiB (256 CUs): one tree of 33 rows
    of V = 128,256 bf16 takes 6 (250 KiB rows), one of 26 rows of V = 151,936 bf16 takes
    7, 21 rows of V = 32,000 fp32 (125 KiB) none, and 60 rows of V = 128,256 fp32 four
    (256 / 60)."""
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    _log("CUs:", cus)
    if cus != 256:
        pytest.skip("the expected sizes assume 256 CUs")
    assert gpu_lib.resispec_tree_group_size(1, 33, 128256, dtype="bf16") == 6
    assert gpu_lib.resispec_tree_group_size(1, 26, 151936, dtype="bf16") == 7
    assert gpu_lib.resispec_tree_group_size(1, 21, 32000, dtype="f32") == 1
    assert gpu_lib.resispec_tree_group_size(1, 60, 128256, dtype="f32") == 4
    assert gpu_lib.resispec_tree_group_size(2, 60, 128256, dtype="f32") == 2
    assert gpu_lib.resispec_tree_group_size(4, 33, 128256, dtype="bf16") == 1
