"""Pins of the oracle's outcome check (the validity test of decisions inside the flag
window).  A claimed node outcome is admissible when every decision on its path is the
oracle's own, except that an accept test with |u - ratio| < 1e-6, or a draw whose
u * total lies within 1e-6 * total of a cumulative-sum boundary, may go either way.

The hand cases use the worked example of the golden file (p = (.2, .4, .4),
q = (.5, .4, .1), candidate 0 rejected): its first ratio is 0.4, its ResiSpec residual
is (0, 8/13, 5/13) and its standard residual is (0, 0, 1).
"""
import numpy as np
import pytest

import oracle as O

P = np.array([0.2, 0.4, 0.4])
Q = np.array([0.5, 0.4, 0.1])


def _check(mode, ua, ur, idx, tok, cand=(0,), worep=False):
    return O.check_node_outcome(P, Q, np.array(cand, np.int32), np.array(ua, np.float32), ur,
                                idx, tok, mode=mode, without_replacement=worep)


def test_accept_test_far_from_the_window():
    # u = 0.1 < 0.4: accepted outside the window; the rejection path is not admissible
    assert _check("resispec", [0.1], 0.5, 0, 0) == 1
    assert _check("resispec", [0.1], 0.5, -1, 1) == 0
    # u = 0.7 >= 0.4: rejected; residual (0, 8/13, 5/13), t = 0.5 -> token 1
    assert _check("resispec", [0.7], 0.5, -1, 1) == 1
    assert _check("resispec", [0.7], 0.5, -1, 2) == 0
    assert _check("resispec", [0.7], 0.5, 0, 0) == 0
    # standard residual (0, 0, 1): every draw is token 2
    assert _check("specinfer", [0.7], 0.5, -1, 2) == 1
    assert _check("specinfer", [0.7], 0.5, -1, 1) == 0
    # an accepted claim must name the candidate's own token
    assert _check("resispec", [0.1], 0.5, 0, 1) == 0


def test_accept_test_inside_the_window():
    u = float(np.float32(0.4))          # |u - 0.4| < 1e-8
    assert abs(u - 0.4) < 1e-6
    oracle_accepts = u < 0.4
    acc = _check("resispec", [u], 0.5, 0, 0)
    rej = _check("resispec", [u], 0.5, -1, 1)
    assert {acc, rej} == {1, 2}
    assert (acc == 1) == oracle_accepts
    # still only the tokens the residual admits
    assert _check("resispec", [u], 0.5, -1, 2) == 0


def test_draw_inside_the_window():
    ur = float(np.float32(8.0 / 13.0))   # t within 1e-7 of the boundary between tokens 1, 2
    assert abs(ur - 8.0 / 13.0) < 1e-7
    v1 = _check("resispec", [0.7], ur, -1, 1)
    v2 = _check("resispec", [0.7], ur, -1, 2)
    assert {v1, v2} == {1, 2}
    assert _check("resispec", [0.7], ur, -1, 0) == 0   # zero mass, far from t
    # a draw just inside the window at the start of the row admits the zero-mass token 0
    # only through the window
    assert _check("resispec", [0.7], 1e-7, -1, 1) == 1
    assert _check("resispec", [0.7], 1e-7, -1, 0) == 2
    assert _check("resispec", [0.7], 1e-4, -1, 0) == 0


def test_faults_on_the_claimed_path_are_not_admissible():
    # a bad candidate id, and a uniform outside [0, 1)
    assert _check("resispec", [0.7, 0.1], 0.5, 1, 5, cand=(0, 5)) == 0
    assert _check("resispec", [1.0], 0.5, -1, 1) == 0
    assert _check("resispec", [0.7], 1.0, -1, 1) == 0


def _rand_node(rng, V, k):
    p = rng.dirichlet(np.full(V, 0.5))
    q = rng.dirichlet(np.full(V, 0.5))
    cand = rng.choice(V, size=k, p=q).astype(np.int32)
    ua = rng.random(k).astype(np.float32)
    ur = float(np.float32(rng.random()))
    return p, q, cand, ua, ur


@pytest.mark.parametrize("mode", ["resispec", "specinfer"])
def test_the_oracles_own_outcome_is_admissible_and_others_are_not(mode):
    """On random nodes the oracle's own outcome always has verdict 1; every other outcome
    has verdict 0 unless the node has a decision inside the window."""
    rng = np.random.default_rng(5)
    others = 0
    for _ in range(400):
        V, k = int(rng.integers(2, 12)), int(rng.integers(0, 4))
        p, q, cand, ua, ur = _rand_node(rng, V, k)
        worep = bool(rng.integers(0, 2))
        if worep and k > 1:
            cand = rng.choice(V, size=min(k, V), replace=False, p=q).astype(np.int32)
            k = cand.size
            ua = ua[:k]
        r = O.verify_node(p, q, cand, ua, ur, mode, worep)
        if r["status"] != O.OK:
            continue
        assert O.check_node_outcome(p, q, cand, ua, ur, r["accepted_index"], r["token"], mode,
                                    worep) == 1
        if r["flagged"]:
            continue
        for idx in range(-1, k):
            for tok in range(V):
                if (idx, tok) == (r["accepted_index"], r["token"]):
                    continue
                if idx >= 0 and tok != cand[idx]:
                    continue
                assert O.check_node_outcome(p, q, cand, ua, ur, idx, tok, mode, worep) == 0
                others += 1
    assert others > 1000


@pytest.mark.parametrize("mode", ["resispec", "specinfer"])
def test_tree_node_claims(mode):
    """Per-node claims of a small tree batch: the oracle's own node outcomes are
    admissible, a wrong child, a wrong token or a wrong fault is not."""
    rng = np.random.default_rng(9)
    B, N, V = 4, 7, 64
    parent = np.array([[-1, 0, 0, 1, 1, 2, 3]] * B, np.int32)
    t = rng.normal(size=(B, N, V)).astype(np.float32)
    d = (t + rng.normal(size=(B, N, V))).astype(np.float32)
    tok = rng.integers(0, V, size=(B, N)).astype(np.int32)
    ua = rng.random((B, N)).astype(np.float32)
    ur = rng.random((B, N)).astype(np.float32)
    tok[3, 3] = V + 2                      # node 1 of sequence 3 tests a bad token first
    rows = np.arange(B * N)
    ref = O.verify_tree_nodes(t, d, tok, parent, ua, ur, rows, temperature=1.0, mode=mode)
    args = (t, d, tok, parent, ua, ur, rows)
    v = O.check_tree_nodes(*args, ref["child"], ref["token"], ref["status"], temperature=1.0,
                           mode=mode)
    assert (v == 1).all()
    assert (ref["status"] == O.BAD_TOKEN).sum() >= 1
    keep = ~ref["flagged"].astype(bool) & (ref["status"] == O.OK)
    # a wrong token on a drawing node, a child that is not a child, a wrong fault
    wrong_tok = np.where(ref["token"] >= 0, (ref["token"] + 1) % V, ref["token"])
    v = O.check_tree_nodes(*args, ref["child"], wrong_tok, ref["status"], temperature=1.0,
                           mode=mode)
    assert (v[keep & (ref["token"] >= 0)] == 0).all()
    bad_child = np.where(ref["child"] >= 0, 0, ref["child"])   # the root is nobody's child
    v = O.check_tree_nodes(*args, bad_child, ref["token"], ref["status"], temperature=1.0,
                           mode=mode)
    assert (v[ref["child"] >= 0] == 0).all()
    wrong_st = np.where(ref["status"] != O.OK, O.ZERO_DRAFT, ref["status"])
    v = O.check_tree_nodes(*args, ref["child"], ref["token"], wrong_st, temperature=1.0,
                           mode=mode)
    assert (v[ref["status"] != O.OK] == 0).all()
