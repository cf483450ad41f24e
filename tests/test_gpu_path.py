"""Path-only schedule (resispec_verify_tree_path): one workgroup per sequence verifies
only the nodes its walk reaches.  Its tokens, lengths and statuses must equal the
all-nodes schedule's bit for bit (the per-node outcome is the same function of the
node's rows and uniforms), and the oracle's walk on unflagged sequences."""
import numpy as np
import pytest
import torch

from paper_2608_24411_amd import synth
from parity_util import compare_walk, gpu_tree, host_tree, oracle_nodes, oracle_walk

pytestmark = pytest.mark.gpu
MODES = ("resispec", "specinfer")


def _log(*a):
    print(*a, flush=True)


def path_tree(native, w, mode, max_depth=None, bonus=True):
    md = w["max_depth"] if max_depth is None else max_depth
    t, l, s = native.resispec_verify_tree_path(
        w["target"], w["draft"], w["node_token"], w["parent"], w["u_accept"], w["u_resample"],
        temperature=w["temperature"], max_depth=md, mode=mode,
        without_replacement=w["without_replacement"], bonus=bonus)
    torch.cuda.synchronize()
    return {"tokens": t, "accepted_len": l, "status": s}


def same(a, b):
    for k in ("tokens", "accepted_len", "status"):
        if not torch.equal(a[k], b[k]):
            x, y = a[k].cpu().numpy(), b[k].cpu().numpy()
            rows = sorted(set(int(i) for i in np.argwhere(x != y)[:, 0]))
            for r in rows[:5]:
                _log("mismatch", k, "seq", r, "path", x[r].tolist(), "reference", y[r].tolist(),
                     "| status", a["status"][r].item(), b["status"][r].item())
            raise AssertionError("%s differs on %d sequences" % (k, len(rows)))


CASES = [(1, dict(B=8)), (2, dict(B=4)), (3, dict(B=3)), (4, dict(B=8)),
         (1, dict(B=4, V=32003)), (2, dict(B=2, V=100003, dtype="f32")),
         (3, dict(B=2, V=65537, dtype="bf16")), (4, dict(B=3, V=4099)),
         # 21 sequences: groups placed one XCD each, the grid padded to 24 groups
         (4, dict(B=21, V=20000))]


@pytest.mark.parametrize("cfg,over", CASES, ids=[f"cfg{c}-{o}" for c, o in CASES])
@pytest.mark.parametrize("mode", MODES)
def test_path_equals_all_nodes_and_oracle(gpu_lib, cfg, over, mode):
    _log("path parity", cfg, over, mode)
    w = synth.make_workload(cfg, device="cuda", **over)
    p = path_tree(gpu_lib, w, mode)
    same(p, gpu_tree(gpu_lib, w, mode))
    h = host_tree(w)
    compare_walk(p, oracle_walk(h, w, mode), h, w, mode)


@pytest.mark.parametrize("cfg", [2, 4])
def test_path_full_size(gpu_lib, cfg):
    """Full configurations: the path schedule equals the all-nodes schedule."""
    _log("path full size", cfg)
    w = synth.make_workload(cfg, device="cuda")
    for mode in MODES:
        p = path_tree(gpu_lib, w, mode)
        same(p, gpu_tree(gpu_lib, w, mode))
        assert (p["status"].cpu().numpy() == 0).all()


def test_path_edges(gpu_lib):
    """Faults met on the walk, bonus off, a short max_depth, root-only trees, B = 0."""
    w = synth.make_workload(1, device="cuda", B=6, V=3001)
    w["u_accept"][2, 1:5] = 0.999
    w["node_token"][3, 2] = 3001
    w["parent"][4, 7] = 9
    w["u_resample"][5, :] = 1.0
    h = host_tree(w)
    for mode in MODES:
        for bonus in (True, False):
            p = path_tree(gpu_lib, w, mode, bonus=bonus)
            same(p, gpu_tree(gpu_lib, w, mode, bonus=bonus))
            compare_walk(p, oracle_walk(h, w, mode, bonus=bonus), h, w, mode, bonus=bonus)
        short = path_tree(gpu_lib, w, mode, max_depth=1)
        same(short, gpu_tree(gpu_lib, w, mode, max_depth=1))
        assert p["status"].cpu().numpy()[4] == 4
    w1 = synth.make_workload(1, device="cuda", B=5, V=777)
    for k in ("target", "draft", "node_token", "parent", "u_accept", "u_resample"):
        w1[k] = w1[k][:, :1].contiguous()
    w1["max_depth"] = 0
    p = path_tree(gpu_lib, w1, "resispec")
    same(p, gpu_tree(gpu_lib, w1, "resispec"))
    assert (p["accepted_len"].cpu() == 0).all()
    e = {k: (v[:0] if isinstance(v, torch.Tensor) else v) for k, v in w.items()}
    t, l, s = gpu_lib.resispec_verify_tree_path(e["target"], e["draft"], e["node_token"],
                                                e["parent"], e["u_accept"], e["u_resample"],
                                                temperature=1.0, max_depth=5)
    torch.cuda.synchronize()
    assert t.numel() == 0


def test_path_side_stream(gpu_lib):
    w = synth.make_workload(3, device="cuda", B=4, V=20000)
    ref = path_tree(gpu_lib, w, "resispec")
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        t, l, st = gpu_lib.resispec_verify_tree_path(
            w["target"], w["draft"], w["node_token"], w["parent"], w["u_accept"],
            w["u_resample"], temperature=w["temperature"], max_depth=w["max_depth"],
            stream=s)
    s.synchronize()
    assert torch.equal(t, ref["tokens"]) and torch.equal(l, ref["accepted_len"])


# ---- row groups: several workgroups per sequence (resispec_verify_tree_path_group)

def group_tree(native, w, mode, group, max_depth=None, bonus=True, workspace=None):
    md = w["max_depth"] if max_depth is None else max_depth
    t, l, s = native.resispec_verify_tree_path_group(
        w["target"], w["draft"], w["node_token"], w["parent"], w["u_accept"], w["u_resample"],
        temperature=w["temperature"], max_depth=md, mode=mode,
        without_replacement=w["without_replacement"], bonus=bonus, group_size=group,
        workspace=workspace)
    torch.cuda.synchronize()
    return {"tokens": t, "accepted_len": l, "status": s}


@pytest.mark.parametrize("cfg,over", CASES, ids=[f"cfg{c}-{o}" for c, o in CASES])
@pytest.mark.parametrize("mode", MODES)
def test_path_groups_equal_path(gpu_lib, cfg, over, mode):
    """Every group size gives the one-workgroup path's results bit for bit (ragged
    vocabularies and the unaligned kernels included), and the oracle's walk."""
    w = synth.make_workload(cfg, device="cuda", **over)
    ref = path_tree(gpu_lib, w, mode)
    for g in (2, 3, 5, 0):
        _log("path group", cfg, over, mode, g)
        same(group_tree(gpu_lib, w, mode, g), ref)
    h = host_tree(w)
    compare_walk(ref, oracle_walk(h, w, mode), h, w, mode)


def _chain_workload(V, dtype, worep, seed):
    """Trees whose walked nodes reject many candidates in a row: a root with 12 children
    and two nodes with 6, candidates taken where the draft over-weights the target
    (Gumbel-top-k of d - t), accept uniforms in [0.97, 1), and in sequence b the target
    row masked (-inf) at its first 3 + b candidates, which are then rejected whatever the
    residual: the later ResiSpec rejection passes (the ones that read the workspace's
    residual) run."""
    g = torch.Generator().manual_seed(seed)
    par = [-1] + [0] * 12 + [1] * 6 + [13] * 6
    B, N = 6, len(par)
    t = 2.0 * torch.randn((B, N, V), generator=g)
    d = 0.3 * t + 2.0 * torch.randn((B, N, V), generator=g)
    if dtype == "bf16":
        t, d = t.to(torch.bfloat16), d.to(torch.bfloat16)
    parent = torch.tensor(par, dtype=torch.int32).repeat(B, 1)
    tok = torch.zeros((B, N), dtype=torch.int32)
    kids_of = {n: [m for m in range(N) if par[m] == n] for n in range(N)}
    for b in range(B):
        for n, kids in kids_of.items():
            if kids:
                gum = -torch.log(-torch.log(torch.rand(V, generator=g).clamp_(min=1e-20)))
                pick = torch.topk(d[b, n].float() - t[b, n].float() + gum, len(kids)).indices
                tok[b, torch.as_tensor(kids)] = pick.to(torch.int32)
                t[b, n, pick[:3 + b]] = float("-inf")
    ua = 0.97 + 0.03 * torch.rand((B, N), generator=g)
    return dict(target=t.cuda(), draft=d.cuda(), node_token=tok.cuda(), parent=parent.cuda(),
                u_accept=ua.clamp_(max=0.9999).cuda(),
                u_resample=torch.rand((B, N), generator=g).cuda(), temperature=1.0,
                without_replacement=worep, max_depth=3), kids_of


@pytest.mark.parametrize("worep", [False, True])
@pytest.mark.parametrize("V,dtype", [(10007, "f32"), (12288, "bf16"), (12289, "bf16")])
def test_path_residual_cache(gpu_lib, worep, V, dtype):
    """The workspace's residual rows: the later ResiSpec rejection passes read the
    residual and draft masses the earlier passes stored instead of re-deriving them from
    the logits.  One workgroup with the workspace, groups of 2 and 3 and the automatic
    size give the results of the path without a workspace and of the all-nodes
    schedule, bit for bit, and the oracle's walk; the walked roots reject at least three
    candidates in a row, so the stored rows are read."""
    w, kids_of = _chain_workload(V, dtype, worep, V + 3 * worep)
    h = host_tree(w)
    for mode in MODES:
        _log("residual cache", V, dtype, "worep", worep, mode)
        ref = path_tree(gpu_lib, w, mode)
        same(ref, gpu_tree(gpu_lib, w, mode))
        ws = torch.empty(gpu_lib.resispec_path_workspace_bytes(6, V), dtype=torch.uint8, device="cuda")
        for g in (1, 2, 3, 0):
            same(group_tree(gpu_lib, w, mode, g, workspace=ws), ref)
        orc = oracle_walk(h, w, mode)
        compare_walk(ref, orc, h, w, mode)
        # rejections at the walked roots (every walk starts there)
        nodes = oracle_nodes(h, w, mode, rows=np.arange(6) * len(kids_of))
        child = nodes["child"]
        rej = [12 if c < 0 else c - kids_of[0][0] for c in child]
        _log("  root rejections", rej)
        assert all(r >= 3 + b for b, r in enumerate(rej)), rej


def test_path_groups_full_size(gpu_lib):
    """The benchmarked configuration with the automatic group size, twice in a row on
    one workspace (its counters are reset by every call)."""
    w = synth.make_workload(2, device="cuda")
    B = w["B"]
    ws = torch.empty(gpu_lib.resispec_path_workspace_bytes(B, w["V"]), dtype=torch.uint8, device="cuda")
    g = gpu_lib.resispec_path_group_size(B, w["V"], dtype="bf16")
    _log("path group full size, automatic group", g)
    assert g >= 1
    for mode in MODES:
        ref = gpu_tree(gpu_lib, w, mode)
        for _ in range(2):
            p = group_tree(gpu_lib, w, mode, 0, workspace=ws)
            same(p, ref)
        assert (p["status"].cpu().numpy() == 0).all()


def test_path_groups_fallback_and_faults(gpu_lib):
    """The exact-maximum pass (maxima exchanged between members) and faults met on the
    walk, with a group of 4."""
    w = synth.make_workload(2, device="cuda", B=3, V=40000)
    w["target"][:, 3, 39990] = 200.0
    w["target"][1, 0, 39000] = 150.0
    for mode in MODES:
        _log("path group fallback", mode)
        same(group_tree(gpu_lib, w, mode, 4), gpu_tree(gpu_lib, w, mode))
    ws = dict(w)
    ws["draft"] = (w["draft"].float() - 60.0).to(w["draft"].dtype)
    for mode in MODES:
        same(group_tree(gpu_lib, ws, mode, 4), gpu_tree(gpu_lib, ws, mode))
    f = synth.make_workload(1, device="cuda", B=6, V=3001)
    f["u_accept"][2, 1:5] = 0.999
    f["node_token"][3, 2] = 3001
    f["parent"][4, 7] = 9
    f["u_resample"][5, :] = 1.0
    for mode in MODES:
        for bonus in (True, False):
            _log("path group faults", mode, bonus)
            same(group_tree(gpu_lib, f, mode, 3, bonus=bonus), path_tree(gpu_lib, f, mode, bonus=bonus))
        same(group_tree(gpu_lib, f, mode, 2, max_depth=1), path_tree(gpu_lib, f, mode, max_depth=1))


def test_path_groups_unsupported(gpu_lib):
    """More members than a row has slots, or than the device holds at once: an error
    before anything runs."""
    w = synth.make_workload(4, device="cuda", B=3, V=512)    # one slot per row
    with pytest.raises(Exception):
        group_tree(gpu_lib, w, "resispec", 2)
    big = synth.make_workload(1, device="cuda", B=400, V=8192)   # 16 slots, 400 x 16 > device
    with pytest.raises(Exception):
        group_tree(gpu_lib, big, "resispec", 16)
    # automatic: falls back to one workgroup per sequence
    same(group_tree(gpu_lib, w, "resispec", 0), path_tree(gpu_lib, w, "resispec"))


def test_path_groups_barrier_time_limit(gpu_lib):
    """Forced from the host (testing hook): with a barrier time limit of zero ticks the
    members of a row group do not wait for each other.  Every workgroup still ends; a
    sequence either reports RS_SEQ_GROUP_TIMEOUT (8) with its outputs at -1, or finishes
    with the reference result (a barrier passes only once every member has published its
    totals).  The default limit restores normal results."""
    w = synth.make_workload(2, device="cuda", B=4, V=40000)
    ref = path_tree(gpu_lib, w, "resispec")
    try:
        gpu_lib.resispec_debug_set_group_waits(barrier=0)
        g = group_tree(gpu_lib, w, "resispec", 4)
    finally:
        gpu_lib.resispec_debug_set_group_waits()
    st = g["status"].cpu().numpy()
    _log("statuses with a zero time limit", st.tolist())
    assert set(st.tolist()) <= {0, 8}
    late = st == 8
    assert (g["accepted_len"].cpu().numpy()[late] == -1).all()
    assert (g["tokens"].cpu().numpy()[late] == -1).all()
    done = ~late
    assert np.array_equal(g["tokens"].cpu().numpy()[done], ref["tokens"].cpu().numpy()[done])
    assert np.array_equal(g["accepted_len"].cpu().numpy()[done],
                          ref["accepted_len"].cpu().numpy()[done])
    same(group_tree(gpu_lib, w, "resispec", 4), ref)


def test_path_groups_formation_fallback(gpu_lib):
    """Forced from the host (testing hook): with a formation limit of zero ticks nearly
    every group is given up and its sequence done by one workgroup alone; formed or not,
    every sequence gets the one-workgroup path's results, in every mode, and the default
    limit restores normal grouping."""
    w = synth.make_workload(2, device="cuda", B=6, V=40000)
    for mode in MODES:
        ref = path_tree(gpu_lib, w, mode)
        try:
            gpu_lib.resispec_debug_set_group_waits(formation=0)
            for g in (2, 4, 0):
                _log("path group with a zero formation limit", mode, g)
                same(group_tree(gpu_lib, w, mode, g), ref)
        finally:
            gpu_lib.resispec_debug_set_group_waits()
        same(group_tree(gpu_lib, w, mode, 4), ref)
