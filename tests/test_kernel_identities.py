"""The algebra the GPU path relies on, checked against the oracle's step-by-step
evaluation (CPU only).

The kernel never materialises a residual row.  It evaluates:

* GetProxy in closed form (Algorithm 1, GetProxy steps 1-3).  With
  Z = D(x0) - R(x0), m_j = min(Z D_j, R_j) (j != x0), M = sum m, SR = sum_{j != x0} R_j
  and a = (Z - M) / (SR - M), the next residual is R'_j = ((1 - a) m_j + a R_j) / Z and
  R'_x0 = 0.  Since R is normalised, SR = 1 - R(x0).
* The standard recurrence (Eq. 1/2) after i rejections in collapsed form
  max(p - C_i q, 0) / Tot_i, with C_0 = 1, C_i = C_{i-1} + Tot_{i-1} s_i and Tot_i the
  sum of max(p - C_i q, 0).  s_i is the draft scale of step i: 1 for i.i.d. candidates,
  and 1 / (1 - removed draft mass) without replacement.
* min(c Q, R) as exp2(min(log2 R, log2 Q + log2 c)).
* One step of that closed form as min(a/Z R + (1 - a) c/Z Q, R/Z), c Q = Z D, which
  holds because 0 <= a <= 1 (the later rejection passes chain it).

Each identity is compared with the oracle's own functions, which take the paper's
steps one at a time.  These functions are pinned separately in test_oracle_pins.py.
"""
import numpy as np
import pytest

import oracle as O


def _pair(rng, V, alpha=0.3):
    p = rng.dirichlet(np.full(V, alpha))
    q = rng.dirichlet(np.full(V, alpha))
    return p, q


def _rejectable(p, q, rng):
    """A token where the draft over-estimates the target (a possible rejection)."""
    cand = np.flatnonzero(q > p)
    return int(rng.choice(cand))


@pytest.mark.parametrize("seed", range(20))
def test_getproxy_closed_form(seed):
    rng = np.random.default_rng(seed)
    V = int(rng.integers(3, 200))
    R, D = _pair(rng, V)
    x0 = _rejectable(R, D, rng)
    steps = O.get_proxy(R, D, x0)
    stepped, st = O.residual_update(R, steps["K"])
    assert st == O.OK
    Z = D[x0] - R[x0]
    m = np.minimum(Z * D, R)
    m[x0] = 0.0
    M = m.sum()
    SR = 1.0 - R[x0]
    assert abs(SR - (R.sum() - R[x0])) < 1e-14
    a = (Z - M) / (SR - M) if SR - M > 0 else 0.0
    closed = ((1.0 - a) * m + a * R) / Z
    closed[x0] = 0.0
    # the step-by-step form computes r as R - (R - r), which cancels when r << R; its
    # rounding is a few ulps of R_j (and K_j) per element, magnified by the
    # normalisation 1/Z, plus the same relative error in the normaliser itself
    eps = np.finfo(np.float64).eps
    RK = R + np.abs(steps["K"])
    tol = 1e-13 + 16 * eps * (RK + closed * RK.sum()) / Z
    assert (np.abs(closed - stepped) <= tol).all()
    assert abs(closed.sum() - 1.0) < 1e-12


@pytest.mark.parametrize("seed", range(20))
@pytest.mark.parametrize("worep", [False, True])
def test_standard_recurrence_collapses(seed, worep):
    rng = np.random.default_rng(1000 + seed)
    V = int(rng.integers(4, 300))
    p, q = _pair(rng, V)
    R, D = p.copy(), q.copy()
    C, s = 1.0, 1.0          # C_0 = s_0 = 1
    steps = 0
    for i in range(int(rng.integers(1, 7))):
        cand = np.flatnonzero(D > R)      # tokens whose test can fail: R(x) < D(x)
        if cand.size == 0:
            break
        x = int(rng.choice(cand))
        R, st = O.residual_update(R, D)  # one step of Eq. 2 with the current draft
        if st != O.OK:
            break
        w = np.maximum(p - C * q, 0.0)
        tot = w.sum()
        assert np.allclose(w / tot, R, rtol=0, atol=1e-12), i
        steps += 1
        if worep:
            s = s / (1.0 - D[x])          # s_{i+1} = s_i / (1 - D_i(x_i))
            D, st = O.draft_remove(D, x)
            assert st == O.OK
            live = D > 0
            assert np.allclose(D[live], q[live] * s, rtol=1e-12, atol=0)
        C = C + tot * s                   # C_{i+1} = C_i + Tot_i s_{i+1}
    assert steps >= 1


@pytest.mark.parametrize("seed", range(10))
def test_min_in_exponent_space(seed):
    rng = np.random.default_rng(2000 + seed)
    aR = rng.normal(-10, 5, size=1000)
    aQ = rng.normal(-10, 5, size=1000)
    c = float(np.exp(rng.normal(0, 3)))
    e = np.floor(np.log2(c))
    f = np.log2(c) - e
    lhs = np.minimum(c * np.exp2(aQ), np.exp2(aR))
    rhs = 2.0 ** f * np.exp2(np.minimum(aR - f, aQ + e))
    assert np.allclose(lhs, rhs, rtol=1e-13, atol=0)


@pytest.mark.parametrize("seed", range(20))
def test_getproxy_step_as_min_of_two_lines(seed):
    """Several rejections in a row: the oracle's GetProxy steps against the kernel's
    four-operation form of each step, min(k1 R + kc D, R / Z) with k1 = a / Z and
    kc = (1 - a); also 0 <= a <= 1 at every step, which the form needs."""
    rng = np.random.default_rng(3000 + seed)
    V = int(rng.integers(4, 300))
    R, D = _pair(rng, V)
    chained = R.copy()
    for step in range(int(rng.integers(2, 6))):
        cand = np.flatnonzero((D > R) & (R > 0))
        if cand.size == 0:
            break
        x0 = int(rng.choice(cand))
        stepped, st = O.residual_update(R, O.get_proxy(R, D, x0)["K"])
        assert st == O.OK
        Z = D[x0] - R[x0]
        m = np.minimum(Z * D, R)
        m[x0] = 0.0
        M = m.sum()
        SR = 1.0 - R[x0]
        a = (Z - M) / (SR - M) if SR - M > 0 else 0.0
        assert -1e-15 <= a <= 1.0 + 1e-15
        chained = np.minimum((a / Z) * chained + (1.0 - a) * D, chained / Z)
        chained[x0] = 0.0
        eps = np.finfo(np.float64).eps
        tol = 1e-12 + 64 * eps * (np.abs(stepped) + stepped.sum()) / Z
        assert (np.abs(chained - stepped) <= tol * 10 ** step).all()
        R = stepped
