"""Pins of the draft-step oracle (CPU): Philox4x32-10 against its published known-answer
vectors, the uniform mapping, and the candidate sampler against brute force and exact
distributions (inverse CDF in vocabulary order; without replacement, sequential draws
from the renormalised draft)."""
import json
import os

import numpy as np
import pytest
from scipy import stats

import oracle as O

HERE = os.path.dirname(os.path.abspath(__file__))


def test_philox_known_answers():
    with open(os.path.join(HERE, "golden", "philox4x32_10_kat.json")) as f:
        kat = json.load(f)
    for v in kat["vectors"]:
        c = [int(x, 16) for x in v["counter"]]
        k = [int(x, 16) for x in v["key"]]
        e = [int(x, 16) for x in v["out"]]
        assert [int(x) for x in O.philox4x32_10(c, k)] == e


def test_u01_mapping():
    assert O.u01(0) == 0.0
    assert O.u01(0xFFFFFFFF) == np.float32(1.0 - 2.0 ** -24)
    assert O.u01(0x80000000) == 0.5
    assert O.u01(0x000000FF) == 0.0          # the low 8 bits are dropped
    assert O.u01(0x00000100) == np.float32(2.0 ** -24)


def test_node_uniform_layout():
    seed, offset = 0x0123456789ABCDEF, 0xFEDCBA9876543210
    for b, n in ((0, 0), (3, 7), (1023, 25)):
        w = O.philox4x32_10([n, b, offset & 0xFFFFFFFF, offset >> 32],
                            [seed & 0xFFFFFFFF, seed >> 32])
        ua, ur, uc = O.node_uniforms(seed, offset, b, n)
        assert (ua, ur, uc) == (O.u01(w[0]), O.u01(w[1]), O.u01(w[2]))


def _softmax(l, T):
    x = (l.astype(np.float64) - l.max()) / T
    e = np.exp(x)
    return e / e.sum()


def _invcdf(D, u):
    t = u * D.sum()
    c = 0.0
    for j, v in enumerate(D):
        c += v
        if c > t:
            return j
    return int(np.flatnonzero(D > 0)[-1])


@pytest.mark.parametrize("worep", [False, True])
def test_sampler_brute_force(worep):
    rng = np.random.default_rng(5 + worep)
    for _ in range(50):
        V = int(rng.integers(2, 40))
        k = int(rng.integers(1, min(V, 8) + 1))
        l = rng.normal(0, 2, V).astype(np.float32)
        T = float(rng.choice([0.5, 1.0, 1.7]))
        uc = rng.random(k).astype(np.float32)
        tok, mg, st = O.sample_candidates(l, k, uc, temperature=T, without_replacement=worep)
        assert st == O.OK
        D = _softmax(l, T)
        for i in range(k):
            x = _invcdf(D, float(uc[i]))
            if mg[i] >= 1e-9:      # rounding-level margins may fall either way
                assert tok[i] == x
            x = int(tok[i])
            if worep and i + 1 < k:
                D = D.copy()
                D[x] = 0.0
                D /= D.sum()
        if worep:
            assert len(set(tok.tolist())) == k


def test_sampler_distributions():
    """Frequencies of Philox-driven draws against the exact laws: i.i.d. draws follow D;
    the first two draws without replacement follow D(x) D(y) / (1 - D(x))."""
    V, T = 6, 1.0
    l = np.array([1.0, 0.2, -0.5, 2.0, 0.0, -1.5], dtype=np.float32)
    D = _softmax(l, T)
    n = 40000
    seed = 2608
    iid = np.zeros(V)
    pairs = np.zeros((V, V))
    for trial in range(n):
        uc = np.array([O.node_uniforms(seed, trial, 0, i)[2] for i in (1, 2)], dtype=np.float32)
        t1, _, _ = O.sample_candidates(l, 1, uc[:1], temperature=T)
        iid[t1[0]] += 1
        t2, _, _ = O.sample_candidates(l, 2, uc, temperature=T, without_replacement=True)
        pairs[t2[0], t2[1]] += 1
    assert stats.chisquare(iid, n * D).pvalue > 1e-3
    exact = np.array([[D[x] * D[y] / (1 - D[x]) if x != y else 0.0 for y in range(V)]
                      for x in range(V)])
    m = exact > 0
    assert pairs[~m].sum() == 0
    assert stats.chisquare(pairs[m], n * exact[m]).pvalue > 1e-3


def test_draft_tree_consistency():
    rng = np.random.default_rng(11)
    B, V = 3, 50
    parent = np.array([[-1, 0, 0, 0, 1, 1, 4], [-1, 0, 1, 2, 3, 4, 5], [-1, 0, 0, 2, 2, 2, 3]],
                      dtype=np.int32)
    N = parent.shape[1]
    draft = rng.normal(0, 1.5, (B, N, V)).astype(np.float32)
    for worep in (False, True):
        out = O.draft_tree(draft, parent, temperature=0.8, without_replacement=worep, seed=9,
                           offset=4)
        assert out["status"] == O.OK
        for b in range(B):
            assert out["node_token"][b, 0] == -1
            for n in range(N):
                ua, ur, uc = O.node_uniforms(9, 4, b, n)
                assert out["u_accept"][b, n] == np.float32(ua)
                assert out["u_resample"][b, n] == np.float32(ur)
                kids = np.flatnonzero(parent[b] == n)
                if kids.size == 0:
                    continue
                ucs = np.array([O.node_uniforms(9, 4, b, m)[2] for m in kids], dtype=np.float32)
                tok, _, _ = O.sample_candidates(draft[b, n], kids.size, ucs, temperature=0.8,
                                                without_replacement=worep)
                assert (out["node_token"][b, kids] == tok).all()
    bad = parent.copy()
    bad[1, 3] = 5
    assert O.draft_tree(draft, bad, temperature=1.0)["status"] == O.BAD_TREE


def test_check_candidates_pins():
    """The admissibility check of claimed draws.  Logits ln(1), ln(2), ln(3), ln(4) at
    T = 1 give D = (1, 2, 3, 4) / 10, whose cumulative sums are .1, .3, .6, 1."""
    row = np.log(np.array([1.0, 2.0, 3.0, 4.0], np.float32)).astype(np.float32)
    D = _softmax(row, 1.0)
    assert np.allclose(D, [0.1, 0.2, 0.3, 0.4], atol=1e-7)
    chk = lambda claimed, uc, worep=False: O.check_candidates(
        row, np.array(claimed, np.int32), np.array(uc, np.float32), temperature=1.0,
        without_replacement=worep)
    assert chk([1], [0.2]) == 1           # .2 lies in [.1, .3)
    assert chk([2], [0.2]) == 0
    assert chk([3, 3], [0.9, 0.65]) == 1  # i.i.d.: the same token twice
    # without replacement the second draw is from (1, 2, 3) / 6: .65 * 6 = 3.9 -> token 2
    assert chk([3, 2], [0.9, 0.65], worep=True) == 1
    assert chk([3, 3], [0.9, 0.65], worep=True) == 0
    # a uniform on a boundary (float32 of .3 is within 1e-8 of it): either side
    u = float(np.float32(0.3))
    assert {chk([1], [u]), chk([2], [u])} == {1, 2}
    assert chk([0], [u]) == 0
    # the claim is followed, not the oracle's own draw: after a windowed first draw the
    # second is judged against the draft without the claimed token
    first = 2 if chk([2], [u]) == 2 else 1
    other = 3 - first
    rest = np.array([0.1, 0.2, 0.3, 0.4])
    rest[first] = 0.0
    rest /= rest.sum()
    v = chk([first, other], [u, float(np.float32(rest[:other].sum() + rest[other] / 2))], worep=True)
    assert v == 2


def test_check_candidates_random_rows():
    """The oracle's own draws are always exact; changing one unflagged draw makes the
    claim inadmissible."""
    rng = np.random.default_rng(21)
    changed = 0
    for _ in range(300):
        V, k = int(rng.integers(2, 30)), int(rng.integers(1, 5))
        worep = bool(rng.integers(0, 2)) and k <= V
        row = rng.normal(size=V).astype(np.float32)
        uc = rng.random(k).astype(np.float32)
        tok, mg, st = O.sample_candidates(row, k, uc, temperature=1.0, without_replacement=worep)
        if st != O.OK:
            continue
        assert O.check_candidates(row, tok, uc, temperature=1.0, without_replacement=worep) == 1
        i = int(rng.integers(0, k))
        if mg[i] < 1e-6 or (i > 0 and (mg[:i] < 1e-6).any()):
            continue
        bad = tok.copy()
        bad[i] = (tok[i] + 1) % V
        assert O.check_candidates(row, bad, uc, temperature=1.0, without_replacement=worep) == 0
        changed += 1
    assert changed > 100
