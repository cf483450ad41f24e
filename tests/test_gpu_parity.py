"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle on the same
seeded inputs.  Token ids, accepted lengths, statuses and per-node outcomes must be
bit-exact on every decision outside the 1e-6 flag window; drawn distributions agree
within 1e-5 absolute per entry and 1e-4 L1."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2608_24411_amd import synth
from parity_util import (STATUS_MAP, compare_node_outcomes, compare_nodes, compare_walk,
                         gpu_tree, host_tree, oracle_nodes, oracle_walk)

pytestmark = pytest.mark.gpu
MODES = ("resispec", "specinfer")


def _log(*a):
    print(*a, flush=True)


# ------------------------------------------------------------------ flat ----

def _flat_check(w, tok, length, st, mode):
    """Every flat row against the oracle: exact outside the flag window, admissible inside
    it.  Returns (exact, flagged)."""
    t, d = synth.to_host(w["target"]), synth.to_host(w["draft"])
    cand, ua, ur = (synth.to_host(w[k]) for k in ("cand_ids", "u_accept", "u_resample"))
    tok, length, st = tok.cpu().numpy(), length.cpu().numpy(), st.cpu().numpy()
    n_flag = 0
    for b in range(w["B"]):
        p = O.softmax(t[b], w["temperature"])
        q = O.softmax(d[b], w["temperature"])
        r = O.verify_node(p, q, cand[b], ua[b], ur[b], mode)
        same = (st[b] == STATUS_MAP[r["status"]] and tok[b] == (r["token"] if r["status"] == O.OK else -1)
                and length[b] == (1 if r["kind"] == O.KIND_ACCEPT else (0 if r["status"] == O.OK else -1)))
        if not r["flagged"]:
            assert same, (b, tok[b], length[b], st[b], r)
            continue
        n_flag += 1
        if same:
            continue
        # the accepted candidate is the first one carrying the returned token (a rejected
        # token has no residual mass left, so a later copy of it is rejected too)
        assert st[b] == 0, (b, st[b], r)
        idx = int(np.flatnonzero(cand[b] == tok[b])[0]) if length[b] == 1 else -1
        assert O.check_node_outcome(p, q, cand[b], ua[b], ur[b], idx, int(tok[b]), mode) != 0, (b, r)
    return w["B"] - n_flag, n_flag


@pytest.mark.parametrize("mode", MODES)
def test_flat_config0_full(gpu_lib, mode):
    """8 rows, V = 32000 fp32, k = 4 i.i.d. candidates: every row against the oracle."""
    w = synth.make_workload(0, device="cuda")
    tok, length, st = gpu_lib.resispec_verify(w["target"], w["draft"], w["cand_ids"],
                                              w["u_accept"], w["u_resample"],
                                              temperature=w["temperature"], mode=mode)
    torch.cuda.synchronize()
    n_exact, n_flag = _flat_check(w, tok, length, st, mode)
    _log("flat config 0", mode, "exact", n_exact, "flagged", n_flag)


@pytest.mark.parametrize("V,dtype", [(32003, "f32"), (50001, "bf16"), (7, "f32"), (1, "bf16")])
def test_flat_ragged_vocab(gpu_lib, V, dtype):
    """V not a multiple of the vector width (element-by-element path) and tiny V."""
    w = synth.make_workload(0, device="cuda", V=V, dtype=dtype, B=16)
    for mode in MODES:
        tok, length, st = gpu_lib.resispec_verify(w["target"], w["draft"], w["cand_ids"],
                                                  w["u_accept"], w["u_resample"],
                                                  temperature=w["temperature"], mode=mode)
        torch.cuda.synchronize()
        _flat_check(w, tok, length, st, mode)


def test_flat_k0_draws_from_target(gpu_lib):
    w = synth.make_workload(0, device="cuda", B=8)
    empty_i = torch.empty((8, 0), dtype=torch.int32, device="cuda")
    empty_f = torch.empty((8, 0), dtype=torch.float32, device="cuda")
    tok, length, st = gpu_lib.resispec_verify(w["target"], w["draft"], empty_i, empty_f,
                                              w["u_resample"], temperature=1.0)
    torch.cuda.synchronize()
    t = synth.to_host(w["target"])
    ur = synth.to_host(w["u_resample"])
    empty = np.empty(0, np.int32)
    for b in range(8):
        p = O.softmax(t[b], 1.0)
        ref, margin, _ = O.invcdf(p, float(ur[b]))
        assert length[b].item() == 0 and st[b].item() == 0
        if margin >= 1e-6:
            assert tok[b].item() == ref
        else:
            assert O.check_node_outcome(p, None, empty, np.empty(0, np.float32), float(ur[b]), -1,
                                        tok[b].item()) != 0


# ------------------------------------------------------------------ trees ---

TREE_CASES = [
    # cfg, overrides: reduced batches that still span many tiles; full V
    (1, dict(B=8)),
    (2, dict(B=3)),
    (3, dict(B=3)),
    (4, dict(B=6)),
    # ragged V (element path) and fp32/bf16 swaps of the same recipes
    (1, dict(B=4, V=32003)),
    (2, dict(B=2, V=100003, dtype="f32")),
    (3, dict(B=2, V=65537, dtype="bf16")),
    (4, dict(B=3, V=4099)),
]


@pytest.mark.parametrize("cfg,over", TREE_CASES, ids=[f"cfg{c}-{o}" for c, o in TREE_CASES])
@pytest.mark.parametrize("mode", MODES)
def test_tree_parity_reduced(gpu_lib, cfg, over, mode):
    _log("tree parity", cfg, over, mode)
    w = synth.make_workload(cfg, device="cuda", **over)
    h = host_tree(w)
    gpu = gpu_tree(gpu_lib, w, mode, debug=True, want_residual=True)
    orc = oracle_walk(h, w, mode)
    compare_walk(gpu, orc, h, w, mode)
    _log("  walks", compare_walk.last)
    B, N = h["parent"].shape
    # residual parity on every node that drew a token (up to 40 rows)
    nt = gpu["node_token"].cpu().numpy().reshape(-1)
    nc = gpu["node_child"].cpu().numpy().reshape(-1)
    drew = np.flatnonzero((nc < 0) & (nt >= 0))[:40]
    n_exact, n_flag, _ = compare_nodes(gpu, h, w, mode, residual_rows=drew)
    _log("  nodes", compare_nodes.last)
    # flagged decisions are checked for admissibility above; most of them are draws that
    # land on a token whose own mass is below the window (V = 128k Zipf tails)
    assert n_flag <= 0.15 * B * N
    # the plain entry point returns the same walk as the debug one
    plain = gpu_tree(gpu_lib, w, mode)
    assert torch.equal(plain["tokens"], gpu["tokens"])
    assert torch.equal(plain["accepted_len"], gpu["accepted_len"])


@pytest.mark.parametrize("T", [0.2, 0.5, 1.5, 3.0])
@pytest.mark.parametrize("mode", MODES)
def test_tree_parity_temperatures(gpu_lib, T, mode):
    """Temperatures away from the recipes' own (0.7-1.0): at T = 0.2 the exponents of a
    Zipf row span hundreds of binades and most elements underflow against the row's
    reference; at T = 3 the rows are nearly flat.  Ragged vocabularies, both dtypes,
    walk and node outcomes against the oracle."""
    for cfg, over in ((2, dict(B=2, V=40003)), (4, dict(B=3, V=30000, dtype="f32"))):
        _log("tree parity at T", T, cfg, over, mode)
        w = synth.make_workload(cfg, device="cuda", T=T, **over)
        h = host_tree(w)
        gpu = gpu_tree(gpu_lib, w, mode, debug=True)
        compare_walk(gpu, oracle_walk(h, w, mode), h, w, mode)
        B, N = h["parent"].shape
        n_exact, n_flag, _ = compare_nodes(gpu, h, w, mode)
        _log("  nodes", compare_nodes.last)
        assert n_flag <= 0.15 * B * N


_FULL = {}


@pytest.fixture(scope="module", autouse=True)
def _release_full_workloads():
    yield
    _FULL.clear()
    torch.cuda.empty_cache()


def _full_workload(cfg):
    """One full-size workload per configuration, with its host copy (the 1024 x 26
    serving batch is 8.1 GB per logits tensor on both sides)."""
    if cfg not in _FULL:
        _FULL.clear()
        torch.cuda.empty_cache()
        w = synth.make_workload(cfg, device="cuda")
        _FULL[cfg] = (w, host_tree(w))
    return _FULL[cfg]


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("cfg", [1, 2, 3, 4])
def test_tree_parity_full_size_walk(gpu_lib, cfg, mode):
    """Full configurations in the launch shape the benchmark times: the walk of every
    sequence against the oracle's sequential walk (exact outside the window, admissible
    inside it), for the all-nodes step, the path-only schedule and the all-nodes schedule
    with deferred draws."""
    _log("full-size walk parity", cfg, mode)
    w, h = _full_workload(cfg)
    plain = gpu_tree(gpu_lib, w, mode)
    orc = oracle_walk(h, w, mode)
    compare_walk(plain, orc, h, w, mode)
    _log("  all-nodes step", compare_walk.last)
    assert compare_walk.last["compared"] == w["B"]
    assert (plain["status"].cpu().numpy() == 0).all()
    pt, pl, ps = gpu_lib.resispec_verify_tree_path(
        w["target"], w["draft"], w["node_token"], w["parent"], w["u_accept"], w["u_resample"],
        temperature=w["temperature"], max_depth=w["max_depth"], mode=mode,
        without_replacement=w["without_replacement"])
    torch.cuda.synchronize()
    assert torch.equal(pt, plain["tokens"]) and torch.equal(pl, plain["accepted_len"])
    assert torch.equal(ps, plain["status"])
    # the all-nodes schedule with deferred draws
    dt, dl, ds = gpu_lib.resispec_verify_tree_deferred(
        w["target"], w["draft"], w["node_token"], w["parent"], w["u_accept"], w["u_resample"],
        temperature=w["temperature"], max_depth=w["max_depth"], mode=mode,
        without_replacement=w["without_replacement"])
    torch.cuda.synchronize()
    assert torch.equal(dt, plain["tokens"]) and torch.equal(dl, plain["accepted_len"])
    assert torch.equal(ds, plain["status"])


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("cfg", [2, 3, 4])
def test_tree_parity_full_size_nodes(gpu_lib, cfg, mode):
    """Full configurations: every node row's own outcome (the all-nodes step verifies all
    of them) against the oracle's evaluation of that node."""
    _log("full-size node parity", cfg, mode)
    w, h = _full_workload(cfg)
    gpu = gpu_tree(gpu_lib, w, mode, debug=True)
    compare_nodes(gpu, h, w, mode)
    _log("  nodes", compare_nodes.last)
    B, N = h["parent"].shape
    assert compare_nodes.last["compared"] == B * N
    assert compare_nodes.last["flagged"] <= 0.15 * B * N
    plain = gpu_tree(gpu_lib, w, mode)
    assert torch.equal(plain["tokens"], gpu["tokens"])


def test_tree_edges(gpu_lib):
    """Root-only trees (bonus draw), bonus off, faults: bad tree, bad token, uniform 1.0,
    max_depth too small, and B = 0."""
    w = synth.make_workload(1, device="cuda", B=6, V=3001)
    w["u_accept"][2, 1:5] = 0.999   # push node 2's walk towards a resample
    w["node_token"][3, 2] = 3001    # out of range id on a child of the root
    w["parent"][4, 7] = 9           # not topological
    w["u_resample"][5, :] = 1.0     # out of range uniform on every draw
    h = host_tree(w)
    for mode in MODES:
        for bonus in (True, False):
            gpu = gpu_tree(gpu_lib, w, mode, debug=True, bonus=bonus)
            orc = oracle_walk(h, w, mode, bonus=bonus)
            compare_walk(gpu, orc, h, w, mode, bonus=bonus)
            compare_nodes(gpu, h, w, mode, bonus=bonus)
        st = gpu_tree(gpu_lib, w, mode)["status"].cpu().numpy()
        assert st[4] == 4
        short = gpu_tree(gpu_lib, w, mode, max_depth=1)
        compare_walk(short, oracle_walk(h, w, mode, max_depth=1), h, w, mode)
    # root only
    w1 = synth.make_workload(1, device="cuda", B=5, V=777)
    for k in ("target", "draft", "node_token", "parent", "u_accept", "u_resample"):
        w1[k] = w1[k][:, :1].contiguous()
    w1["max_depth"] = 0
    h1 = host_tree(w1)
    gpu = gpu_tree(gpu_lib, w1, "resispec", debug=True)
    compare_walk(gpu, oracle_walk(h1, w1, "resispec"), h1, w1, "resispec")
    assert (gpu["accepted_len"].cpu() == 0).all()
    # empty batch
    e = {k: (v[:0] if isinstance(v, torch.Tensor) else v) for k, v in w.items()}
    t, l, s = gpu_lib.resispec_verify_tree(e["target"], e["draft"], e["node_token"], e["parent"],
                                           e["u_accept"], e["u_resample"], temperature=1.0,
                                           max_depth=5)
    torch.cuda.synchronize()
    assert t.numel() == 0


@pytest.mark.parametrize("cfg,over", [(2, dict(B=3, V=20000)), (4, dict(B=3, V=30000)),
                                      (3, dict(B=2, V=30001))])
def test_masked_logits(gpu_lib, cfg, over):
    """Rows with -inf entries (masked vocabulary, as after top-k filtering) at every
    temperature of the recipes; candidate tokens keep finite logits."""
    w = synth.make_workload(cfg, device="cuda", **over)
    g = torch.Generator(device="cuda").manual_seed(7)
    for key in ("target", "draft"):
        mask = torch.rand(w[key].shape, generator=g, device="cuda") < 0.3
        B, N = w["node_token"].shape
        keep = torch.zeros_like(mask)
        for b in range(B):   # keep every candidate's own entries finite
            par = w["parent"][b].cpu().numpy()
            tok = w["node_token"][b].cpu().numpy()
            for m in range(1, N):
                keep[b, par[m], tok[m]] = True
        w[key] = w[key].masked_fill(mask & ~keep, float("-inf"))
    h = host_tree(w)
    for mode in MODES:
        gpu = gpu_tree(gpu_lib, w, mode, debug=True)
        compare_walk(gpu, oracle_walk(h, w, mode), h, w, mode)
        compare_nodes(gpu, h, w, mode)
        assert (gpu["status"].cpu().numpy() == 0).all()


def test_reference_fallback(gpu_lib):
    """Rows whose exponent reference (taken from the first chunks) does not fit: a +200
    logit placed late in target rows (the sums overflow), and draft rows shifted by -60
    (their sums underflow; a constant shift leaves the softmax unchanged).  Both take the
    exact-maximum path and must still agree with the oracle."""
    w = synth.make_workload(2, device="cuda", B=3, V=40000)
    w["target"][:, 3, 39990] = 200.0
    w["target"][1, 0, 39000] = 150.0
    h = host_tree(w)
    for mode in MODES:
        gpu = gpu_tree(gpu_lib, w, mode, debug=True)
        compare_walk(gpu, oracle_walk(h, w, mode), h, w, mode)
        compare_nodes(gpu, h, w, mode)
    ws = dict(w)
    ws["draft"] = (w["draft"].float() - 60.0).to(w["draft"].dtype)
    hs = host_tree(ws)
    for mode in MODES:
        a = gpu_tree(gpu_lib, ws, mode, debug=True)
        compare_walk(a, oracle_walk(hs, ws, mode), hs, ws, mode)
        compare_nodes(a, hs, ws, mode)


def test_max_children(gpu_lib):
    """A node with RS_MAX_CANDIDATES children, and one with one more (device status 7)."""
    for n_kids, expect_status in ((64, 0), (65, 7)):
        N, V, B = n_kids + 1, 2048, 2
        g = torch.Generator().manual_seed(n_kids)
        t = torch.randn((B, N, V), generator=g)
        d = t + 1.5 * torch.randn((B, N, V), generator=g)
        par = torch.zeros((B, N), dtype=torch.int32)
        par[:, 0] = -1
        tok = torch.randint(0, V, (B, N), generator=g, dtype=torch.int32)
        ua = torch.rand((B, N), generator=g)
        ur = torch.rand((B, N), generator=g)
        w = dict(target=t.cuda(), draft=d.cuda(), node_token=tok.cuda(), parent=par.cuda(),
                 u_accept=ua.cuda(), u_resample=ur.cuda(), temperature=1.0,
                 without_replacement=False, max_depth=1)
        for mode in MODES:
            gpu = gpu_tree(gpu_lib, w, mode)
            if expect_status:
                assert (gpu["status"].cpu().numpy() == expect_status).all()
            else:
                h = host_tree(w)
                compare_walk(gpu, oracle_walk(h, w, mode), h, w, mode)


@pytest.mark.parametrize("worep", [False, True])
@pytest.mark.parametrize("V,dtype", [(10007, "f32"), (12288, "bf16")])
def test_long_rejection_chains(gpu_lib, worep, V, dtype):
    """Nodes that reject several candidates in a row: a root with 12 children and two
    nodes with 6, candidates taken where the draft over-weights the target (Gumbel-top-k
    of d - t; with replacement the second candidate repeats the first).  Exercises the
    later steps of both residual updates, with and without replacement, and checks the
    drawn distributions entry by entry."""
    g = torch.Generator().manual_seed(V + 7 * worep)
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
            if not kids:
                continue
            gum = -torch.log(-torch.log(torch.rand(V, generator=g).clamp_(min=1e-20)))
            pick = torch.topk(d[b, n].float() - t[b, n].float() + gum, len(kids)).indices
            if not worep and len(kids) > 2:
                pick[1] = pick[0]
            tok[b, torch.as_tensor(kids)] = pick.to(torch.int32)
    w = dict(target=t.cuda(), draft=d.cuda(), node_token=tok.cuda(), parent=parent.cuda(),
             u_accept=torch.rand((B, N), generator=g).cuda(),
             u_resample=torch.rand((B, N), generator=g).cuda(), temperature=1.0,
             without_replacement=worep, max_depth=3)
    h = host_tree(w)
    internal = [n for n in range(N) if kids_of[n]]
    for mode in MODES:
        _log("long chains", V, dtype, "worep", worep, mode)
        gpu = gpu_tree(gpu_lib, w, mode, debug=True, want_residual=True)
        compare_walk(gpu, oracle_walk(h, w, mode), h, w, mode)
        drew = [r for r in range(B * N) if gpu["node_child"].reshape(-1)[r].item() < 0]
        n_exact, n_flag, orc = compare_nodes(gpu, h, w, mode, residual_rows=drew)
        _log("  nodes", compare_nodes.last)
        assert n_flag <= 0.15 * B * N
        # the chains are long: internal nodes reject candidates before they accept (the
        # proxy-shaped residual accepts within two or three), and with the standard
        # residual most of them reject every candidate and draw
        child = orc["child"].reshape(B, N)
        rejected = np.array([len(kids_of[n]) if child[b, n] < 0 else child[b, n] - kids_of[n][0]
                             for b in range(B) for n in internal])
        assert np.mean(rejected >= 1) > 0.8, rejected
        if mode == "specinfer":
            assert np.mean(rejected == np.array([len(kids_of[n]) for b in range(B)
                                                 for n in internal])) > 0.5, rejected


def test_determinism(gpu_lib):
    w = synth.make_workload(2, device="cuda", B=16)
    for mode in MODES:
        a = gpu_tree(gpu_lib, w, mode, debug=True)
        b = gpu_tree(gpu_lib, w, mode, debug=True)
        for k in ("tokens", "accepted_len", "node_child", "node_token"):
            assert torch.equal(a[k], b[k])


def test_stream_ordering(gpu_lib):
    """Results on a side stream equal those on the default stream."""
    w = synth.make_workload(3, device="cuda", B=4, V=20000)
    ref = gpu_tree(gpu_lib, w, "resispec")
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        t, l, st = gpu_lib.resispec_verify_tree(
            w["target"], w["draft"], w["node_token"], w["parent"], w["u_accept"], w["u_resample"],
            temperature=w["temperature"], max_depth=w["max_depth"], stream=s)
    s.synchronize()
    assert torch.equal(t, ref["tokens"]) and torch.equal(l, ref["accepted_len"])


def test_max_vocab(gpu_lib):
    """V = RS_MAX_VOCAB (2^22): slots of many chunks, draws that re-read a slot from
    memory instead of registers; both schedules and the draft step."""
    V = 1 << 22
    g = torch.Generator(device="cuda").manual_seed(22)
    par = torch.tensor([[-1, 0, 0, 1]], dtype=torch.int32, device="cuda").repeat(2, 1)
    B, N = par.shape
    t = (2.0 * torch.randn((B, N, V), generator=g, device="cuda")).to(torch.bfloat16)
    d = (t.float() + torch.randn((B, N, V), generator=g, device="cuda")).to(torch.bfloat16)
    tok, ua, ur, st = gpu_lib.resispec_draft_candidates(d, par, temperature=1.0, seed=4)
    w = dict(target=t, draft=d, node_token=tok, parent=par, u_accept=ua, u_resample=ur,
             temperature=1.0, without_replacement=False, max_depth=2)
    h = host_tree(w)
    for mode in MODES:
        gpu = gpu_tree(gpu_lib, w, mode, debug=True)
        compare_walk(gpu, oracle_walk(h, w, mode), h, w, mode)
        compare_nodes(gpu, h, w, mode)
        t2, l2, s2 = gpu_lib.resispec_verify_tree_path(
            t, d, tok, par, ua, ur, temperature=1.0, max_depth=2, mode=mode)
        torch.cuda.synchronize()
        assert torch.equal(t2, gpu["tokens"]) and torch.equal(l2, gpu["accepted_len"])


@pytest.mark.parametrize("mode", MODES)
def test_large_trees(gpu_lib, mode):
    """Trees of more nodes than a workgroup has threads (700): the row is described
    directly in shared memory and the candidates' logits gathered by one wave.  Sequence 0
    has a root with 64 children (the limit) and a random tree below; sequence 1 the same
    with 65 children under node 2 (that node reports RS_SEQ_TOO_MANY_CHILDREN, 7);
    sequence 2 a parent that is not topological (every node and the walk report
    RS_SEQ_BAD_TREE, 4).  All-nodes step and path schedule (one workgroup and row groups)
    against the oracle and each other."""
    B, N, V = 3, 700, 3000
    rng = np.random.default_rng(700)
    par = np.empty((B, N), np.int32)
    for b in range(B):
        par[b, 0] = -1
        par[b, 1:65] = 0
        for n in range(65, N):   # below the root's children, at most 64 children each
            while True:
                p = int(rng.integers(1, n))
                if (par[b, :n] == p).sum() < 64:
                    break
            par[b, n] = p
    # sequence 1: node 2 takes 65 children (moved from elsewhere, keeping the order)
    kids2 = np.flatnonzero(par[1] == 2)
    extra = [n for n in range(200, N) if par[1, n] != 2][:65 - kids2.size]
    par[1, extra] = 2
    assert (par[1] == 2).sum() == 65
    par[2, 500] = 600
    g = torch.Generator().manual_seed(5)
    t = 1.5 * torch.randn((B, N, V), generator=g)
    d = t + torch.randn((B, N, V), generator=g)
    tok = torch.zeros((B, N), dtype=torch.int32)
    for b in range(B):   # children drawn from the parent's draft row
        q = torch.softmax(d[b], dim=-1)
        for n in range(1, N):
            tok[b, n] = int(torch.multinomial(q[par[b, n]], 1, generator=g))
    w = dict(target=t.cuda(), draft=d.cuda(), node_token=tok.cuda(),
             parent=torch.as_tensor(par).cuda(), u_accept=torch.rand((B, N), generator=g).cuda(),
             u_resample=torch.rand((B, N), generator=g).cuda(), temperature=1.0,
             without_replacement=False, max_depth=N)
    h = host_tree(w)
    gpu = gpu_tree(gpu_lib, w, mode, debug=True)
    gc = gpu["node_child"].cpu().numpy().reshape(-1)
    gk = gpu["node_token"].cpu().numpy().reshape(-1)
    gs = gpu["node_status"].cpu().numpy().reshape(-1)
    # the over-full node, then every other row against the oracle
    r7 = 1 * N + 2
    assert gs[r7] == 7 and gc[r7] == -1 and gk[r7] == -1
    assert (gs[2 * N:3 * N] == 4).all()
    rows = np.setdiff1d(np.arange(B * N), [r7])
    orc = oracle_nodes(h, w, mode, rows=rows)
    summary = compare_node_outcomes(gc[rows], gk[rows], gs[rows], orc, h, w, mode, rows=rows)
    _log("large trees", mode, summary)
    # walks: sequence 0 against the oracle; sequence 1 too unless it reaches node 2
    orc_w = oracle_walk(h, w, mode)
    st = gpu["status"].cpu().numpy()
    assert st[2] == 4 and orc_w["status"][2] == O.BAD_TREE
    excl = np.array([False, st[1] == 7, False])
    compare_walk(gpu, orc_w, h, w, mode, exclude=excl)
    # the path schedule returns the same, alone and with row groups
    plain = gpu_tree(gpu_lib, w, mode)
    for group in (1, 2, 4):
        pt, pl, ps = gpu_lib.resispec_verify_tree_path_group(
            w["target"], w["draft"], w["node_token"], w["parent"], w["u_accept"],
            w["u_resample"], temperature=1.0, max_depth=N, mode=mode, group_size=group)
        torch.cuda.synchronize()
        assert torch.equal(pt, plain["tokens"]) and torch.equal(pl, plain["accepted_len"])
        assert torch.equal(ps, plain["status"])
