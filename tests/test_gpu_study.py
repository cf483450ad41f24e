"""The synthetic analogues of the paper's studies (bench.py --study: acceptance by
candidate index, the paper's first figure; mean accepted length by tree shape, its
topology ablation; the marginal gain per extra candidate, its efficiency score), run on
the device at reduced trials and checked against the oracle on the same inputs:

- every trial's outcomes (the root's accepted candidate; every sequence's walk) equal
  the oracle's on the device's draws (exact outside the flag window, admissible inside);
- the study's reported figures are the ones these outcomes give;
- the first candidate's acceptance rate agrees with its closed form: a candidate drawn
  from q is accepted with probability min(1, p(x)/q(x)), so a row accepts its first
  candidate with probability sum_x min(p(x), q(x)) (Eq. 2 with i = 1), the same in
  both modes."""
import numpy as np
import pytest
import torch

import bench
import oracle as O
from paper_2608_24411_amd import synth
from parity_util import compare_node_outcomes, compare_walk, host_tree, oracle_nodes, oracle_walk

pytestmark = pytest.mark.gpu


def _log(*a):
    print(*a, flush=True)


def test_study_against_oracle(gpu_lib):
    B_root, B_tree, n_root, n_tree = 128, 24, 4, 2
    seen = {"root8": {}, "walks": {}}
    first = {"resispec": [], "specinfer": []}
    closed = []

    def trace(kind, mode, w, out):
        h = host_tree(w)
        B, N = h["parent"].shape
        if kind == "root8":
            rows = np.arange(B) * N
            orc = oracle_nodes(h, w, mode, rows=rows)
            gc = out["node_child"].cpu().numpy()[:, 0]
            gk = out["node_token"].cpu().numpy()[:, 0]
            gs = out["node_status"].cpu().numpy()[:, 0]
            summary = compare_node_outcomes(gc, gk, gs, orc, h, w, mode, rows=rows)
            seen["root8"].setdefault(mode, []).append(gc)
            first[mode].append(gc == 1)
            if mode == "resispec":
                for b in range(B):
                    p = O.softmax(h["target"][b, 0], w["temperature"])
                    q = O.softmax(h["draft"][b, 0], w["temperature"])
                    closed.append(np.minimum(p, q).sum())
            _log("root8", mode, summary)
        else:
            orc = oracle_walk(h, w, mode)
            compare_walk(out, orc, h, w, mode)
            seen["walks"].setdefault((kind, mode), []).append(
                (out["accepted_len"].cpu().numpy(), orc["accepted_len"], orc["flagged"]))

    res = bench.run_study(gpu_lib, torch, np, synth, B_root=B_root, B_tree=B_tree,
                          n_root=n_root, n_tree=n_tree, trace=trace)

    # the study's figures are the checked outcomes
    for mode in ("resispec", "specinfer"):
        c = np.concatenate(seen["root8"][mode])
        rec = res["accept_by_candidate_index"][mode]
        assert rec["trials"] == B_root * n_root == c.size
        assert rec["P(accept candidate i), i=1..8"] == [float(np.mean(c == i + 1)) for i in range(8)]
        assert rec["P(all rejected)"] == float(np.mean(c < 0))
    for name, r in res["mean_accepted_length_by_shape"].items():
        for mode in ("resispec", "specinfer"):
            parts = seen["walks"][(name, mode)]
            gl = np.concatenate([p[0] for p in parts])
            ol = np.concatenate([p[1] for p in parts])
            fl = np.concatenate([p[2] for p in parts]).astype(bool)
            assert r[mode] == float(gl.mean())
            assert (gl[~fl] == ol[~fl]).all()
    widths = res["mean_accepted_length_by_width_depth3"]
    for mode in ("resispec", "specinfer"):
        eta = res["eta_marginal_gain_per_extra_candidate"][mode]
        for k in ("2", "3", "4", "6", "8"):
            assert eta[k] == pytest.approx((widths[k][mode] - widths["1"][mode]) / (int(k) - 1))
        # one candidate per level: both residual rules take the same decisions
        assert widths["1"]["resispec"] == widths["1"]["specinfer"]

    # the first candidate's acceptance against sum_x min(p, q), one entry per trial (the
    # rows repeat across trials; only the draws change)
    closed = np.array(closed)
    expect = float(closed.mean())
    sigma = float(np.sqrt((closed * (1 - closed)).sum())) / closed.size
    for mode in ("resispec", "specinfer"):
        got = float(np.concatenate(first[mode]).mean())
        _log("first-candidate acceptance", mode, got, "closed form", expect, "sigma", sigma)
        assert abs(got - expect) <= 4 * sigma
    assert np.array_equal(np.concatenate(first["resispec"]), np.concatenate(first["specinfer"]))
