"""Pins of the oracle's tree walk (Preliminary, multi-candidate tree-structured
verification): descend into the accepted child, stop at a resample, bonus draw
at an accepted leaf, children verified in ascending node index."""
import numpy as np
import pytest
import scipy.special
import scipy.stats

import oracle as O

# depth-2 tree: root 0 -> {1, 2}; node 1 -> {3, 4}; nodes 2, 3, 4 are leaves
PARENT = np.array([-1, 0, 0, 1, 1], dtype=np.int32)


def _chisq(counts, expected):
    keep = expected >= 5
    obs, ex = counts[keep].astype(np.float64), expected[keep]
    if (~keep).any():
        obs = np.append(obs, counts[~keep].sum())
        ex = np.append(ex, expected[~keep].sum())
    ex = ex * (obs.sum() / ex.sum())
    return scipy.stats.chisquare(obs, ex)[1]


@pytest.mark.parametrize("mode", ["specinfer", "resispec"])
def test_tree_walk_monte_carlo(mode):
    rng = np.random.default_rng(51 + (mode == "resispec"))
    V, T, B = 4, 1.0, 200_000
    tl = rng.normal(scale=1.2, size=(5, V)).astype(np.float32)
    dl = (tl + rng.normal(scale=1.5, size=(5, V))).astype(np.float32)
    p = [scipy.special.softmax(tl[i].astype(np.float64) / T) for i in range(5)]
    q = [scipy.special.softmax(dl[i].astype(np.float64) / T) for i in range(5)]
    target = np.broadcast_to(tl, (B, 5, V)).copy()
    draft = np.broadcast_to(dl, (B, 5, V)).copy()
    tok = np.zeros((B, 5), dtype=np.int32)
    tok[:, 1:3] = rng.choice(V, size=(B, 2), p=q[0])
    tok[:, 3:5] = rng.choice(V, size=(B, 2), p=q[1])
    par = np.broadcast_to(PARENT, (B, 5)).copy()
    ua = rng.random((B, 5)).astype(np.float32)
    ur = rng.random((B, 5)).astype(np.float32)
    out = O.verify_tree_walk(target, draft, tok, par, ua, ur, temperature=T, max_depth=2, mode=mode)
    assert (out["status"] == O.OK).all()
    L = out["accepted_len"]
    toks = out["tokens"]
    assert ((L >= 0) & (L <= 2)).all()
    # exactly accepted_len + 1 tokens, the rest -1
    for length in range(3):
        sel = L == length
        assert (toks[sel, : length + 1] >= 0).all()
        assert (toks[sel, length + 1:] == -1).all()

    # first token: the root's node output (p for Eq. 2, enumerated for Algorithm 1)
    first = p[0] if mode == "specinfer" else O.enumerate_output(p[0], q[0], 2, mode)
    assert _chisq(np.bincount(toks[:, 0], minlength=V), first * B) > 1e-3

    # second token given which child was accepted (only where the two children differ)
    differ = tok[:, 1] != tok[:, 2]
    via1 = differ & (L >= 1) & (toks[:, 0] == tok[:, 1])
    via2 = differ & (L >= 1) & (toks[:, 0] == tok[:, 2])
    assert via1.sum() > 10_000 and via2.sum() > 10_000
    after1 = p[1] if mode == "specinfer" else O.enumerate_output(p[1], q[1], 2, mode)
    assert _chisq(np.bincount(toks[via1, 1], minlength=V), after1 * via1.sum()) > 1e-3
    # node 2 is a leaf: bonus draw from its own target row
    assert _chisq(np.bincount(toks[via2, 1], minlength=V), p[2] * via2.sum()) > 1e-3
    assert (L[via2] == 1).all()


def test_walk_matches_independent_node_outcomes():
    """Per-node outcomes do not depend on the path taken: the walk equals following
    the independently evaluated outcomes from the root."""
    rng = np.random.default_rng(61)
    B, N, V = 64, 5, 16
    target = rng.normal(size=(B, N, V)).astype(np.float32)
    draft = (target + rng.normal(size=(B, N, V))).astype(np.float32)
    tok = rng.integers(0, V, size=(B, N)).astype(np.int32)
    par = np.broadcast_to(PARENT, (B, N)).copy()
    ua = rng.random((B, N)).astype(np.float32)
    ur = rng.random((B, N)).astype(np.float32)
    for mode in ("resispec", "specinfer"):
        walk = O.verify_tree_walk(target, draft, tok, par, ua, ur, temperature=0.8, max_depth=2,
                                  mode=mode)
        rows = np.arange(B * N)
        nodes = O.verify_tree_nodes(target, draft, tok, par, ua, ur, rows, temperature=0.8,
                                    mode=mode)
        for b in range(B):
            n, seq = 0, []
            while True:
                r = b * N + n
                c = nodes["child"][r]
                if c >= 0:
                    seq.append(tok[b, c])
                    n = c
                    continue
                seq.append(nodes["token"][r])
                break
            assert walk["accepted_len"][b] == len(seq) - 1
            assert list(walk["tokens"][b, : len(seq)]) == seq


def test_tree_faults():
    rng = np.random.default_rng(62)
    B, N, V = 3, 5, 8
    target = rng.normal(size=(B, N, V)).astype(np.float32)
    draft = rng.normal(size=(B, N, V)).astype(np.float32)
    tok = rng.integers(0, V, size=(B, N)).astype(np.int32)
    par = np.broadcast_to(PARENT, (B, N)).copy()
    par[1, 3] = 3              # not topological
    ua = np.zeros((B, N), dtype=np.float32)   # u = 0 accepts every candidate with R(x) > 0
    ur = rng.random((B, N)).astype(np.float32)
    out = O.verify_tree_walk(target, draft, tok, par, ua, ur, temperature=1.0, max_depth=2)
    assert out["status"][1] == O.BAD_TREE and out["accepted_len"][1] == -1
    assert (out["tokens"][1] == -1).all()
    assert out["status"][0] == O.OK and out["accepted_len"][0] == 2
    short = O.verify_tree_walk(target, draft, tok, np.broadcast_to(PARENT, (B, N)).copy(), ua, ur,
                               temperature=1.0, max_depth=1)
    assert (short["status"] == O.DEPTH_EXCEEDED).all()
    nob = O.verify_tree_walk(target, draft, tok, np.broadcast_to(PARENT, (B, N)).copy(), ua, ur,
                             temperature=1.0, max_depth=2, bonus=False)
    assert (nob["accepted_len"] == 2).all() and (nob["tokens"][:, 2] == -1).all()
