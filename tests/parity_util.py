"""Shared helpers of the GPU parity tests: run the HIP path and the oracle on the same
seeded buffers and compare.  Decisions whose oracle margin falls inside the 1e-6 flag
window (|u - ratio| for accept tests, the inverse-CDF margin relative to the total for
draws) are excluded from the exact comparison and counted."""
import numpy as np
import torch

import oracle as O
from paper_2608_24411_amd import synth

STATUS_MAP = {O.OK: 0, O.BAD_TOKEN: 1, O.ZERO_DRAFT: 2, O.UNDERFLOW: 3, O.BAD_TREE: 4,
              O.BAD_UNIFORM: 5, O.DEPTH_EXCEEDED: 6}


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


def oracle_walk(h, w, mode, max_depth=None, bonus=True):
    md = w["max_depth"] if max_depth is None else max_depth
    return O.verify_tree_walk(h["target"], h["draft"], h["node_token"], h["parent"], h["u_accept"],
                              h["u_resample"], temperature=w["temperature"], max_depth=md,
                              mode=mode, without_replacement=w["without_replacement"],
                              bonus=bonus)


def compare_walk(gpu, orc, seqs=None):
    """Exact equality of tokens / lengths / status on every unflagged sequence.
    Returns (compared, flagged)."""
    gt = gpu["tokens"].cpu().numpy()
    gl = gpu["accepted_len"].cpu().numpy()
    gs = gpu["status"].cpu().numpy()
    if seqs is not None:
        gt, gl, gs = gt[seqs], gl[seqs], gs[seqs]
    fl = orc["flagged"].astype(bool)
    exp_status = np.vectorize(STATUS_MAP.get)(orc["status"])
    keep = ~fl
    bad = np.flatnonzero(keep & ((gl != orc["accepted_len"]) | (gs != exp_status)
                                 | (gt != orc["tokens"]).any(axis=1)))
    assert bad.size == 0, (
        "walk mismatch at sequences %s: gpu len %s tok %s st %s / oracle len %s tok %s st %s" % (
            bad[:5], gl[bad[:5]], gt[bad[:5]], gs[bad[:5]], orc["accepted_len"][bad[:5]],
            orc["tokens"][bad[:5]], orc["status"][bad[:5]]))
    return int(keep.sum()), int(fl.sum())


def compare_nodes(gpu, h, w, mode, seqs=None, bonus=True, residual_rows=None):
    """Exact equality of every unflagged node outcome; optionally the drawn
    distributions within 1e-5 absolute per entry and 1e-4 L1 per row."""
    B, N = h["parent"].shape
    rows = np.arange(B * N)
    orc = O.verify_tree_nodes(h["target"], h["draft"], h["node_token"], h["parent"], h["u_accept"],
                              h["u_resample"], rows, temperature=w["temperature"], mode=mode,
                              without_replacement=w["without_replacement"], bonus=bonus,
                              want_residual=residual_rows is not None)
    gc = gpu["node_child"].cpu().numpy()
    gk = gpu["node_token"].cpu().numpy()
    gs = gpu["node_status"].cpu().numpy()
    if seqs is not None:
        gc, gk, gs = gc[seqs], gk[seqs], gs[seqs]
    gc, gk, gs = gc.reshape(-1), gk.reshape(-1), gs.reshape(-1)
    fl = orc["flagged"].astype(bool)
    exp_status = np.vectorize(STATUS_MAP.get)(orc["status"])
    keep = ~fl
    bad = np.flatnonzero(keep & ((gc != orc["child"]) | (gk != orc["token"]) | (gs != exp_status)))
    assert bad.size == 0, (
        "node mismatch at rows %s: gpu child %s tok %s st %s / oracle child %s tok %s st %s" % (
            bad[:5], gc[bad[:5]], gk[bad[:5]], gs[bad[:5]], orc["child"][bad[:5]],
            orc["token"][bad[:5]], orc["status"][bad[:5]]))
    # flagged rows: how many still agree, and whether any with margin >= 1e-7 disagree
    diff = (gc != orc["child"]) | (gk != orc["token"]) | (gs != exp_status)
    tight = fl & (orc["margin"] >= 1e-7)
    compare_nodes.last = {"flagged": int(fl.sum()), "flagged_agree": int((fl & ~diff).sum()),
                          "mismatch_margin_ge_1e-7": int((tight & diff).sum())}
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
    return int(keep.sum()), int(fl.sum()), orc
