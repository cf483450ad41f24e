"""Synthetic analogue of the paper's exactness study (its KL table): the output
distribution of one node, enumerated exactly over every candidate value and accept/
reject path (oracle.enumerate_output), against the target p, for both residual updates,
with and without replacement, on Zipf+noise rows (CPU).

The standard recurrence is exact (TV below 1e-12).  The literal Algorithm 1 with
GetProxy is not: its GetProxy depends on the rejected token, which the exactness
argument assumes it does not.  Its deviation is measured and kept within the range
recorded below, so that a change in it is noticed.  Run with -s to print the table."""
import numpy as np
import pytest

import oracle as O


def _rows(rng, V, a=1.1, sigma_t=1.0, sigma_d=1.5):
    rank = rng.permutation(V) + 1
    t = -a * np.log(rank) + sigma_t * rng.normal(size=V)
    d = t + sigma_d * rng.normal(size=V)
    p = np.exp(t - t.max())
    q = np.exp(d - d.max())
    return p / p.sum(), q / q.sum()


def _tv(a, b):
    return 0.5 * np.abs(a - b).sum()


def _kl(p, o):
    m = p > 0
    return float(np.sum(p[m] * np.log(p[m] / o[m])))


@pytest.mark.parametrize("worep", [False, True])
def test_exactness_table(worep):
    rows = []
    for V in (4, 6, 8):
        for k in (1, 2, 3):
            tv = {"resispec": [], "specinfer": []}
            kl = {"resispec": [], "specinfer": []}
            for seed in range(6):
                p, q = _rows(np.random.default_rng(1000 * V + 10 * k + seed), V)
                for mode in tv:
                    out = O.enumerate_output(p, q, k, mode=mode, without_replacement=worep)
                    assert abs(out.sum() - 1.0) < 1e-12
                    tv[mode].append(_tv(out, p))
                    kl[mode].append(_kl(p, out))
            rows.append((V, k, max(tv["specinfer"]), np.mean(tv["resispec"]),
                         max(tv["resispec"]), np.mean(kl["resispec"])))
            assert max(tv["specinfer"]) < 1e-12
            assert max(abs(x) for x in kl["specinfer"]) < 1e-12
            assert 1e-3 < np.mean(tv["resispec"]) < 0.5
    print("\nwithout replacement" if worep else "\ni.i.d. candidates")
    print("  V  k  max TV standard   mean TV ResiSpec   max TV ResiSpec   mean KL(p||out) ResiSpec")
    for V, k, ts, tr, trm, kr in rows:
        print("%3d %2d  %15.2e   %16.4f   %15.4f   %12.4f" % (V, k, ts, tr, trm, kr))
