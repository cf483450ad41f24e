"""Shared helpers of the GPU parity tests: run the HIP path and the oracle on the same
seeded buffers and compare.

Every decision is checked.  Outside the 1e-6 flag window (|u - ratio| for accept tests,
the inverse-CDF margin relative to the total for draws) the GPU must equal the oracle
bit for bit.  A node or sequence with a decision inside the window must still be
admissible: the oracle's outcome check replays the GPU's claimed path and lets only the
windowed decisions go the other way.  Within the window, decisions whose oracle margin is
at least 1e-7 must still agree exactly (the kernel's own error is below 3e-8).

The oracle runs on host threads (one call per chunk of rows or per sequence; the C code
is re-entrant and ctypes releases the interpreter lock around it)."""
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import torch

import oracle as O
from paper_2608_24411_amd import synth

STATUS_MAP = {O.OK: 0, O.BAD_TOKEN: 1, O.ZERO_DRAFT: 2, O.UNDERFLOW: 3, O.BAD_TREE: 4,
              O.BAD_UNIFORM: 5, O.DEPTH_EXCEEDED: 6}
# host threads for the oracle: the CPU share of one GPU on the test machines
THREADS = max(1, min(16, len(os.sched_getaffinity(0))))


def host_tree(w, seqs=None):
    sel = slice(None) if seqs is None else torch.as_tensor(seqs, device=w["target"].device)
    return dict(target=synth.to_host(w["target"][sel]), draft=synth.to_host(w["draft"][sel]),
                node_token=synth.to_host(w["node_token"][sel]),
                parent=synth.to_host(w["parent"][sel]),
                u_accept=synth.to_host(w["u_accept"][sel]),
                u_resample=synth.to_host(w["u_resample"][sel]))


def gpu_tree(native, w, mode, debug=False, want_residual=False, max_depth=None, bonus=True):
    md = w["max_depth"] if max_depth is None else max_depth
    kw = dict(temperature=w["temperature"], max_depth=md, mode=mode,
              without_replacement=w["without_replacement"], bonus=bonus)
    args = (w["target"], w["draft"], w["node_token"], w["parent"], w["u_accept"], w["u_resample"])
    if debug:
        out = native.resispec_verify_tree_debug(*args, want_residual=want_residual, **kw)
    else:
        t, l, s = native.resispec_verify_tree(*args, **kw)
        out = {"tokens": t, "accepted_len": l, "status": s}
    torch.cuda.synchronize()
    return out


def _tree_args(h):
    return (h["target"], h["draft"], h["node_token"], h["parent"], h["u_accept"], h["u_resample"])


def _tree_kw(w, mode, bonus):
    return dict(temperature=w["temperature"], mode=mode,
                without_replacement=w["without_replacement"], bonus=bonus)


def _pool_map(fn, items):
    if len(items) <= 1 or THREADS == 1:
        return [fn(x) for x in items]
    with ThreadPoolExecutor(THREADS) as ex:
        return list(ex.map(fn, items))


def oracle_walk(h, w, mode, max_depth=None, bonus=True):
    """The oracle's sequential walk of every sequence of h (threads over sequences)."""
    md = w["max_depth"] if max_depth is None else max_depth
    B = h["parent"].shape[0]

    def one(b):
        hb = {k: v[b:b + 1] for k, v in h.items()}
        return O.verify_tree_walk(*_tree_args(hb), max_depth=md, **_tree_kw(w, mode, bonus))
    parts = _pool_map(one, list(range(B)))
    if not parts:
        return {"tokens": np.empty((0, md + 1), np.int32), "accepted_len": np.empty(0, np.int32),
                "status": np.empty(0, np.int32), "flagged": np.empty(0, np.int32)}
    return {k: np.concatenate([p[k] for p in parts]) for k in parts[0]}


def oracle_nodes(h, w, mode, rows=None, bonus=True, want_residual=False):
    """The oracle's independent evaluation of the given rows (all of them by default),
    threads over chunks of rows."""
    B, N = h["parent"].shape
    rows = np.arange(B * N) if rows is None else np.asarray(rows, dtype=np.int64)
    if want_residual:
        return O.verify_tree_nodes(*_tree_args(h), rows, want_residual=True,
                                   **_tree_kw(w, mode, bonus))
    chunks = [c for c in np.array_split(rows, max(1, min(len(rows), 4 * THREADS))) if c.size]
    parts = _pool_map(lambda c: O.verify_tree_nodes(*_tree_args(h), c, **_tree_kw(w, mode, bonus)),
                      chunks)
    if not parts:
        return {"child": np.empty(0, np.int32), "token": np.empty(0, np.int32),
                "status": np.empty(0, np.int32), "flagged": np.empty(0, np.int32),
                "margin": np.empty(0)}
    return {k: np.concatenate([p[k] for p in parts]) for k in parts[0]}


def check_claims(h, w, mode, rows, child, token, status, bonus=True):
    """Oracle verdicts (1 exact, 2 admissible through a windowed decision, 0 not
    admissible) of claimed node outcomes; GPU status codes 0-6 are the oracle's."""
    rows = np.asarray(rows, dtype=np.int64)
    if rows.size == 0:
        return np.empty(0, np.int32)
    idx = np.array_split(np.arange(rows.size), max(1, min(rows.size, 4 * THREADS)))
    idx = [i for i in idx if i.size]
    child, token, status = (np.asarray(a, dtype=np.int32) for a in (child, token, status))
    parts = _pool_map(lambda i: O.check_tree_nodes(*_tree_args(h), rows[i], child[i], token[i],
                                                   status[i], **_tree_kw(w, mode, bonus)), idx)
    return np.concatenate(parts)


def walk_claims(h, b, tokens, length, status):
    """The per-node claims a walk result makes for sequence b of h: the path follows, at
    each node, the first child (ascending index) whose token is the next output token,
    and ends with the node's drawn (or absent) token.  None when the tokens do not form a
    path of the tree."""
    if status != 0:
        return None
    par = h["parent"][b]
    ntok = h["node_token"][b]
    N = par.shape[0]
    claims, n = [], 0
    for i in range(int(length)):
        kids = [c for c in range(n + 1, N) if par[c] == n and ntok[c] == tokens[i]]
        if not kids:
            return None
        claims.append((b * N + n, kids[0], int(tokens[i]), 0))
        n = kids[0]
    last = int(tokens[length]) if length < tokens.shape[0] else -1
    claims.append((b * N + n, -1, last, 0))
    return claims


def compare_walk(gpu, orc, h, w, mode, seqs=None, bonus=True, exclude=None):
    """Walk results (tokens, lengths, statuses) against the oracle's walk on every
    sequence of h.  Unflagged sequences are bit-exact; flagged ones must be admissible
    path by path (every node claim the GPU walk makes passes the oracle's outcome check).
    `exclude` (bool per sequence) leaves sequences out whose inputs the oracle did not
    see.  Returns (exact, flagged)."""
    gt = gpu["tokens"].cpu().numpy()
    gl = gpu["accepted_len"].cpu().numpy()
    gs = gpu["status"].cpu().numpy()
    if seqs is not None:
        gt, gl, gs = gt[seqs], gl[seqs], gs[seqs]
    fl = orc["flagged"].astype(bool)
    skip = np.zeros_like(fl) if exclude is None else np.asarray(exclude, dtype=bool)
    exp_status = np.vectorize(STATUS_MAP.get)(orc["status"]) if orc["status"].size else orc["status"]
    keep = ~fl & ~skip
    bad = np.flatnonzero(keep & ((gl != orc["accepted_len"]) | (gs != exp_status)
                                 | (gt != orc["tokens"]).any(axis=1)))
    assert bad.size == 0, (
        "walk mismatch at sequences %s: gpu len %s tok %s st %s / oracle len %s tok %s st %s" % (
            bad[:5], gl[bad[:5]], gt[bad[:5]], gs[bad[:5]], orc["accepted_len"][bad[:5]],
            orc["tokens"][bad[:5]], orc["status"][bad[:5]]))
    # flagged sequences: identical results need no replay; the rest are replayed
    flagged = np.flatnonzero(fl & ~skip)
    differ = [b for b in flagged if not (gl[b] == orc["accepted_len"][b] and gs[b] == exp_status[b]
                                        and (gt[b] == orc["tokens"][b]).all())]
    rows, cc, ct, cs, owner = [], [], [], [], []
    for b in differ:
        claims = walk_claims(h, b, gt[b], gl[b], gs[b])
        assert claims is not None, (
            "flagged sequence %d: gpu walk (len %s, status %s, tokens %s) is not a path of its "
            "tree or ends in a fault the oracle's walk (status %s) does not share" % (
                b, gl[b], gs[b], gt[b], orc["status"][b]))
        for r, c, t, s in claims:
            rows.append(r); cc.append(c); ct.append(t); cs.append(s); owner.append(b)
    v = check_claims(h, w, mode, rows, cc, ct, cs, bonus)
    assert (v != 0).all(), "flagged sequences with an inadmissible walk: %s" % (
        sorted(set(np.asarray(owner)[v == 0].tolist())),)
    compare_walk.last = {"compared": int((~skip).sum()), "exact": int(keep.sum()),
                         "flagged": int(flagged.size), "flagged_identical": int(flagged.size - len(differ)),
                         "flagged_admissible": int(len(differ))}
    return int(keep.sum()), int(flagged.size)


def compare_node_outcomes(gc, gk, gs, orc, h, w, mode, bonus=True, rows=None):
    """Per-node outcomes (child, token, status arrays over `rows`, all rows of h by
    default) against the oracle's: bit-exact outside the window, at least 1e-7 inside it
    too, and every other flagged node admissible.  Returns a summary dict."""
    B, N = h["parent"].shape
    rows = np.arange(B * N) if rows is None else np.asarray(rows, dtype=np.int64)
    fl = orc["flagged"].astype(bool)
    exp_status = np.vectorize(STATUS_MAP.get)(orc["status"]) if orc["status"].size else orc["status"]
    diff = (gc != orc["child"]) | (gk != orc["token"]) | (gs != exp_status)
    bad = np.flatnonzero(~fl & diff)
    assert bad.size == 0, (
        "node mismatch at rows %s: gpu child %s tok %s st %s / oracle child %s tok %s st %s" % (
            rows[bad[:5]], gc[bad[:5]], gk[bad[:5]], gs[bad[:5]], orc["child"][bad[:5]],
            orc["token"][bad[:5]], orc["status"][bad[:5]]))
    tight = fl & (orc["margin"] >= 1e-7) & diff
    assert not tight.any(), "flagged rows with margin >= 1e-7 that differ: %s" % rows[tight][:5]
    # flagged rows that differ: their claimed outcome must be admissible
    redo = np.flatnonzero(fl & diff)
    v = check_claims(h, w, mode, rows[redo], gc[redo], gk[redo], gs[redo], bonus)
    assert (v != 0).all(), "inadmissible flagged node outcomes at rows %s" % rows[redo][v == 0][:5]
    return {"compared": int(rows.size), "exact": int((~fl).sum()), "flagged": int(fl.sum()),
            "flagged_identical": int((fl & ~diff).sum()), "flagged_admissible": int(redo.size),
            "mismatches": 0}


def compare_nodes(gpu, h, w, mode, seqs=None, bonus=True, residual_rows=None):
    """Every node outcome of a debug call against the oracle (compare_node_outcomes);
    optionally the drawn distributions of `residual_rows` within 1e-5 absolute per entry
    and 1e-4 L1 per row.  Returns (exact, flagged, oracle outcomes); the summary is in
    compare_nodes.last."""
    B, N = h["parent"].shape
    orc = oracle_nodes(h, w, mode, bonus=bonus, want_residual=residual_rows is not None)
    gc = gpu["node_child"].cpu().numpy()
    gk = gpu["node_token"].cpu().numpy()
    gs = gpu["node_status"].cpu().numpy()
    if seqs is not None:
        gc, gk, gs = gc[seqs], gk[seqs], gs[seqs]
    gc, gk, gs = gc.reshape(-1), gk.reshape(-1), gs.reshape(-1)
    summary = compare_node_outcomes(gc, gk, gs, orc, h, w, mode, bonus)
    compare_nodes.last = summary
    keep = ~orc["flagged"].astype(bool)
    if residual_rows is not None:
        gr = gpu["residual"]
        if seqs is not None:
            gr = gr[torch.as_tensor(seqs, device=gr.device)]
        gr = gr.reshape(B * N, -1)
        for r in residual_rows:
            if not keep[r] or orc["child"][r] >= 0 or orc["token"][r] < 0:
                continue
            ref = orc["final_R"][r]
            got = gr[r].double().cpu().numpy()
            assert np.abs(got - ref).max() <= 1e-5, (r, np.abs(got - ref).max())
            assert np.abs(got - ref).sum() <= 1e-4, (r, np.abs(got - ref).sum())
    return summary["exact"], summary["flagged"], orc
