"""GPU tests of the all-nodes schedule with deferred draws (resispec_verify_tree_deferred,
and its two launches resispec_decide_nodes and resispec_walk_draw), through the C ABI.

A row that rejects its one candidate keeps its pass-1 slot totals instead of drawing, and a
leaf's row (which serves only its bonus draw) is not read; the walk draws where it ends.
Checked here:
  - tokens, accepted lengths and statuses equal the all-nodes schedule's bit for bit, and
    the walks agree with the oracle's sequential walk (exact outside the 1e-6 window,
    admissible inside it);
  - after the first launch every node that did not defer has the all-nodes schedule's
    outcome, and only rows with at most one child defer;
  - after the second launch every node the walks drew for has the all-nodes outcome."""
import numpy as np
import pytest
import torch

from paper_2608_24411_amd import synth
from parity_util import compare_walk, gpu_tree, host_tree, oracle_walk

pytestmark = pytest.mark.gpu
MODES = ("resispec", "specinfer")
DEFERRED = 9


def _log(*a):
    print(*a, flush=True)


def _args(w):
    return (w["target"], w["draft"], w["node_token"], w["parent"], w["u_accept"], w["u_resample"])


def _deferred(lib, w, mode, bonus=True, max_depth=None):
    """Both launches, with the node outcomes after each, and the one-call entry point."""
    md = w["max_depth"] if max_depth is None else max_depth
    B, N = w["node_token"].shape
    kw = dict(temperature=w["temperature"], mode=mode,
              without_replacement=w["without_replacement"], bonus=bonus)
    ws = torch.empty(max(1, lib.resispec_deferred_workspace_bytes(B, N)), dtype=torch.uint8,
                     device="cuda")
    lib.resispec_decide_nodes(*_args(w), ws, **kw)
    decided = tuple(t.cpu().numpy() for t in lib.resispec_node_outcomes(ws, B, N))
    t, l, s = lib.resispec_walk_draw(*_args(w), ws, max_depth=md, **kw)
    torch.cuda.synchronize()
    final = tuple(x.cpu().numpy() for x in lib.resispec_node_outcomes(ws, B, N))
    t1, l1, s1 = lib.resispec_verify_tree_deferred(*_args(w), max_depth=md, **kw)
    torch.cuda.synchronize()
    assert torch.equal(t1, t) and torch.equal(l1, l) and torch.equal(s1, s)
    return dict(tokens=t, accepted_len=l, status=s, decided=decided, final=final)


def _terminals(rc, max_depth):
    """(b, n) of the node where each walk over the all-nodes outcomes ends and draws: it
    follows accepted children and stops at the first node that accepts none (a walk that
    would pass max_depth stops without a draw)."""
    out = set()
    for b in range(rc.shape[0]):
        n, length = 0, 0
        while rc[b, n] >= 0:
            if length >= max_depth:
                n = -1
                break
            n, length = rc[b, n], length + 1
        if n >= 0:
            out.add((b, int(n)))
    return out


def _against_all_nodes(lib, w, mode, bonus=True, max_depth=None, leaves_defer=True):
    """The deferred schedule against the all-nodes schedule on the same inputs.
    leaves_defer: every leaf without a fault must defer (not for rows that take the
    exact-maximum pass, which draw at once)."""
    ref = gpu_tree(lib, w, mode, debug=True, bonus=bonus, max_depth=max_depth)
    d = _deferred(lib, w, mode, bonus=bonus, max_depth=max_depth)
    for k in ("tokens", "accepted_len", "status"):
        assert torch.equal(d[k], ref[k]), k
    rc, rk, rs = (ref[k].cpu().numpy() for k in ("node_child", "node_token", "node_status"))
    dc, dk, ds = d["decided"]
    par = w["parent"].cpu().numpy()
    B, N = par.shape
    kids = np.zeros((B, N), dtype=np.int64)
    for b in range(B):
        for m in range(1, N):
            if 0 <= par[b, m] < m:
                kids[b, par[b, m]] += 1
    defer = ds == DEFERRED
    keep = ~defer
    assert np.array_equal(dc[keep], rc[keep]) and np.array_equal(dk[keep], rk[keep])
    assert np.array_equal(ds[keep], rs[keep])
    # only rows with at most one candidate defer, and only those that accept nothing; the
    # all-nodes schedule drew for them (or met a fault of the draw)
    assert (kids[defer] <= 1).all()
    assert (rc[defer] == -1).all()
    assert np.isin(rs[defer], (0, 3, 5)).all()
    if bonus and leaves_defer:
        assert (defer | (kids > 0) | (rs != 0)).all()   # every healthy leaf deferred
    # after the walks: the nodes drawn for are exactly the deferred nodes where walks end,
    # and they now have the all-nodes outcome; the others are still deferred
    fc, fk, fs = d["final"]
    done = fs != DEFERRED
    assert done[keep].all()
    assert np.array_equal(fc[done], rc[done]) and np.array_equal(fk[done], rk[done])
    assert np.array_equal(fs[done], rs[done])
    md = w["max_depth"] if max_depth is None else max_depth
    drawn = {(int(b), int(n)) for b, n in zip(*np.nonzero(done & defer))}
    assert drawn == {(b, n) for b, n in _terminals(rc, md) if defer[b, n]}
    return d, ref, int(defer.sum()), len(drawn)


TREE_CASES = [
    (1, dict(B=8)),
    (2, dict(B=3)),
    (3, dict(B=3)),
    (4, dict(B=6)),
    (1, dict(B=4, V=32003)),
    (2, dict(B=2, V=100003, dtype="f32")),
    (3, dict(B=2, V=65537, dtype="bf16")),
    (4, dict(B=3, V=4099)),
]


@pytest.mark.parametrize("cfg,over", TREE_CASES, ids=[f"cfg{c}-{o}" for c, o in TREE_CASES])
@pytest.mark.parametrize("mode", MODES)
def test_deferred_reduced(gpu_lib, cfg, over, mode):
    _log("deferred", cfg, over, mode)
    w = synth.make_workload(cfg, device="cuda", **over)
    d, ref, n_def, n_drawn = _against_all_nodes(gpu_lib, w, mode)
    h = host_tree(w)
    compare_walk(d, oracle_walk(h, w, mode), h, w, mode)
    _log("  deferred rows", n_def, "drawn by the walks", n_drawn, compare_walk.last)


@pytest.mark.parametrize("mode", MODES)
def test_deferred_benchmark_shape(gpu_lib, mode):
    """The benchmarked 128 x 33 bf16 batch at V = 128,256: every node's first-launch outcome
    and every walk against the all-nodes schedule."""
    w = synth.make_workload(2, device="cuda")
    d, ref, n_def, n_drawn = _against_all_nodes(gpu_lib, w, mode)
    _log("benchmark shape", mode, "deferred rows", n_def, "drawn by the walks", n_drawn)
    assert n_def > 1000 and n_drawn > 0


def test_deferred_edges(gpu_lib):
    """Faults met by the walks (bad tree, bad token, out-of-range uniforms at every draw),
    bonus off, max_depth too small, root-only trees, B = 0."""
    w = synth.make_workload(1, device="cuda", B=6, V=3001)
    w["u_accept"][2, 1:5] = 0.999   # push node 2's walk towards a resample
    w["node_token"][3, 2] = 3001    # out of range id on a child of the root
    w["parent"][4, 7] = 9           # not topological
    w["u_resample"][5, :] = 1.0     # out of range uniform on every draw
    h = host_tree(w)
    for mode in MODES:
        for bonus in (True, False):
            d, _, _, _ = _against_all_nodes(gpu_lib, w, mode, bonus=bonus)
            compare_walk(d, oracle_walk(h, w, mode, bonus=bonus), h, w, mode, bonus=bonus)
        for md in (0, 1, 2):
            d, _, _, _ = _against_all_nodes(gpu_lib, w, mode, max_depth=md)
            compare_walk(d, oracle_walk(h, w, mode, max_depth=md), h, w, mode)
    w1 = synth.make_workload(1, device="cuda", B=5, V=777)
    for k in ("target", "draft", "node_token", "parent", "u_accept", "u_resample"):
        w1[k] = w1[k][:, :1].contiguous()
    w1["max_depth"] = 0
    for mode in MODES:
        d, _, n_def, n_drawn = _against_all_nodes(gpu_lib, w1, mode)
        assert n_def == 5 and n_drawn == 5   # every root is a leaf that the walk ends at
        assert (d["accepted_len"].cpu() == 0).all()
    e = {k: (v[:0] if isinstance(v, torch.Tensor) else v) for k, v in w.items()}
    t, l, s = gpu_lib.resispec_verify_tree_deferred(*_args(e), temperature=1.0, max_depth=5)
    torch.cuda.synchronize()
    assert t.numel() == 0


def test_deferred_reference_fallback(gpu_lib):
    """Rows that take the exact-maximum pass draw at once instead of deferring; the walks
    are the same."""
    w = synth.make_workload(2, device="cuda", B=3, V=40000)
    w["target"][:, 3, 39990] = 200.0
    w["target"][1, 0, 39000] = 150.0
    w["target"][:, 9, 39995] = 180.0   # single-child rows
    w["target"][:, 30, 39001] = 170.0  # leaves
    h = host_tree(w)
    for mode in MODES:
        d, _, _, _ = _against_all_nodes(gpu_lib, w, mode, leaves_defer=False)
        compare_walk(d, oracle_walk(h, w, mode), h, w, mode)


@pytest.mark.parametrize("worep", [False, True])
def test_deferred_chains_and_wide_nodes(gpu_lib, worep):
    """Trees mixing nodes of 1 to 12 children, with and without replacement; candidates
    taken where the draft over-weights the target, so single-child rows reject often."""
    g = torch.Generator().manual_seed(31 + worep)
    par = [-1, 0, 0, 0, 1, 4, 5, 6, 2, 2, 3] + [8] * 12 + [10, 23, 24]
    B, N, V = 5, len(par), 12288
    t = (2.0 * torch.randn((B, N, V), generator=g)).to(torch.bfloat16)
    d = (0.3 * t.float() + 2.0 * torch.randn((B, N, V), generator=g)).to(torch.bfloat16)
    parent = torch.tensor(par, dtype=torch.int32).repeat(B, 1)
    tok = torch.zeros((B, N), dtype=torch.int32)
    kids_of = {n: [m for m in range(N) if par[m] == n] for n in range(N)}
    for b in range(B):
        for n, kids in kids_of.items():
            if kids:
                gum = -torch.log(-torch.log(torch.rand(V, generator=g).clamp_(min=1e-20)))
                pick = torch.topk(d[b, n].float() - t[b, n].float() + gum, len(kids)).indices
                tok[b, torch.as_tensor(kids)] = pick.to(torch.int32)
    w = dict(target=t.cuda(), draft=d.cuda(), node_token=tok.cuda(), parent=parent.cuda(),
             u_accept=torch.rand((B, N), generator=g).cuda(),
             u_resample=torch.rand((B, N), generator=g).cuda(), temperature=1.0,
             without_replacement=worep, max_depth=6)
    h = host_tree(w)
    for mode in MODES:
        d, _, n_def, n_drawn = _against_all_nodes(gpu_lib, w, mode)
        compare_walk(d, oracle_walk(h, w, mode), h, w, mode)
        _log("chains", worep, mode, "deferred", n_def, "drawn", n_drawn)


def test_deferred_many_nodes(gpu_lib):
    """Trees of 700 nodes (more nodes than threads: rows described in shared memory):
    chains, a node of 64 children and a leaf-heavy tail."""
    N, V, B = 700, 4096, 2
    par = [-1] + list(range(0, 40)) + [40] * 64 + list(range(41, 41 + 595))
    par = par[:N]
    g = torch.Generator().manual_seed(700)
    t = torch.randn((B, N, V), generator=g)
    d = t + 1.2 * torch.randn((B, N, V), generator=g)
    parent = torch.tensor(par, dtype=torch.int32).repeat(B, 1)
    tok = torch.randint(0, V, (B, N), generator=g, dtype=torch.int32)
    w = dict(target=t.cuda(), draft=d.cuda(), node_token=tok.cuda(), parent=parent.cuda(),
             u_accept=(0.02 * torch.rand((B, N), generator=g)).cuda(),
             u_resample=torch.rand((B, N), generator=g).cuda(), temperature=1.0,
             without_replacement=False, max_depth=N)
    h = host_tree(w)
    for mode in MODES:
        d, _, n_def, n_drawn = _against_all_nodes(gpu_lib, w, mode)
        compare_walk(d, oracle_walk(h, w, mode), h, w, mode)
        _log("700 nodes", mode, "deferred", n_def, "drawn", n_drawn,
             "lengths", d["accepted_len"].cpu().tolist())


def test_deferred_determinism_and_stream(gpu_lib):
    w = synth.make_workload(3, device="cuda", B=4, V=20000)
    a = _deferred(gpu_lib, w, "resispec")
    b = _deferred(gpu_lib, w, "resispec")
    assert torch.equal(a["tokens"], b["tokens"]) and torch.equal(a["accepted_len"], b["accepted_len"])
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        t, l, st = gpu_lib.resispec_verify_tree_deferred(
            *_args(w), temperature=w["temperature"], max_depth=w["max_depth"], stream=s)
    s.synchronize()
    assert torch.equal(t, a["tokens"]) and torch.equal(l, a["accepted_len"])
