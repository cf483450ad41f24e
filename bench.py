#!/usr/bin/env python3
"""Benchmark of the ResiSpec verification step on one MI355X.

One step = one full verification of a batch of draft trees on inputs already resident in
HBM, in the all-nodes schedule with deferred draws: the decide kernel tests every node
row (a row that rejects its one candidate keeps its slot totals instead of drawing, and a
leaf's row, which serves only its bonus draw, is left whole), then the finish kernel
follows accepted children from each root and draws where a walk ends.  Prints one JSON
line.

  python bench.py [--gpus 1] [--steps 20] [--warmup 5] [--config 2] [--mode resispec]

The metric is verified tree-node rows per second (B * N / step time) at V = 128,256;
`roofline.achieved` is the decide kernel's algorithmic bytes (the target and draft rows of
every node with children once, plus ids/uniforms/outcomes; a leaf's row serves only its
bonus draw and is read by the walk where it ends) divided by its
average launch duration measured with HIP events on the launch stream.  The read probe
(libresispec_probe.so) measures the device's achievable read rate beside it:
`roofline.frac_of_read_ceiling` is the achieved figure over the nontemporal stream rate.
The same step with every row drawing at once (`all_nodes_draw`), the path-only schedule,
the draft step and the other workloads are reported beside it.
"""
import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
HBM_PEAK_GBPS = 8000.0
# the sources the decide kernel is compiled from
KERNEL_SRCS = [os.path.join(ROOT, "paper_2608_24411_amd", "csrc", f)
               for f in ("resispec.hip", "common.h")]
METRIC = "verified tree-node rows/s at V=128256 + achieved HBM GB/s (% of peak)"


def kernel_source_hash():
    """sha256 of the kernel sources' code: comments removed and white space collapsed, so
    that a profile stays matched to a kernel whose comments alone have changed."""
    h = hashlib.sha256()
    for path in KERNEL_SRCS:
        with open(path, encoding="utf-8") as f:
            src = f.read()
        src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)
        src = re.sub(r"//[^\n]*", " ", src)
        h.update(" ".join(src.split()).encode())
    return h.hexdigest()


def measured_traffic(workload, mode):
    """HBM bytes per launch of the decide kernel from the rocprofv3 counter summary, if the
    summary was taken on the current kernel source."""
    path = os.path.join(ROOT, "profiles", "traffic_rs_decide_kernel_%s_%s.json" % (workload, mode))
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("kernel_source_sha256") != kernel_source_hash():
        return None
    return rec.get("hbm_bytes_per_launch")


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def cpu_baseline(w, seconds, mode, gpu_nodes=None, gpu_walk=None):
    """The fp64 oracle on the host, on the same workload, three ways:
      - all-nodes: every node row evaluated on its own (what the row kernels compute),
        over the host's cores (threads over chunks of rows; the oracle is re-entrant and
        ctypes releases the interpreter lock around it); this is `value`;
      - walk: each sequence walked from its root (only the nodes the walk reaches), over
        the same threads (one sequence per task);
      - single thread: all-nodes on whole sequences until about `seconds` of CPU time.
    With `gpu_nodes` (the node outcomes the last timed GPU step left) the all-nodes results
    are also the parity check of that step: bit-exact outside the 1e-6 flag window, and
    every flagged node either identical or admissible (the oracle's outcome check).  A
    node whose draw was deferred and never made (no walk ended there) is compared on its
    decision: it accepted none of its candidates.  With `gpu_walk` (its tokens and
    lengths) every sequence is compared with the oracle's walk.  Returns (record, parity)."""
    import numpy as np
    from concurrent.futures import ThreadPoolExecutor
    import oracle as O
    from paper_2608_24411_amd import synth
    B, N = w["B"], w["N"]
    h = dict(target=synth.to_host(w["target"]), draft=synth.to_host(w["draft"]),
             node_token=synth.to_host(w["node_token"]), parent=synth.to_host(w["parent"]),
             u_accept=synth.to_host(w["u_accept"]), u_resample=synth.to_host(w["u_resample"]))
    args = (h["target"], h["draft"], h["node_token"], h["parent"], h["u_accept"], h["u_resample"])
    kw = dict(temperature=w["temperature"], mode=mode, without_replacement=w["without_replacement"],
              bonus=w["bonus"])
    nproc = os.cpu_count() or 1
    avail = len(os.sched_getaffinity(0))
    # the CPU share of one GPU on the benchmark machines is 16 cores
    threads = max(1, min(16, avail))

    rows = np.arange(B * N)
    chunks = [c for c in np.array_split(rows, 8 * threads) if c.size]
    t0 = time.perf_counter()
    with ThreadPoolExecutor(threads) as ex:
        parts = list(ex.map(lambda c: O.verify_tree_nodes(*args, c, **kw), chunks))
    t_nodes = time.perf_counter() - t0
    orc = {k: np.concatenate([p[k] for p in parts]) for k in parts[0]}

    def walk(b):
        sl = tuple(a[b:b + 1] for a in args)
        return O.verify_tree_walk(*sl, max_depth=w["max_depth"], **kw)
    t0 = time.perf_counter()
    with ThreadPoolExecutor(threads) as ex:
        walks = list(ex.map(walk, range(B)))
    t_walk = time.perf_counter() - t0
    walk_rows = int(sum(int(r["accepted_len"][0]) + 1 for r in walks))

    # single thread on whole sequences, bounded by CPU time
    single_rows, t_single, seqs = 0, 0.0, 0
    for b in range(B):
        c0 = time.process_time()
        O.verify_tree_nodes(*args, np.arange(b * N, (b + 1) * N), **kw)
        t_single += time.process_time() - c0
        single_rows += N
        seqs += 1
        if t_single >= seconds:
            break

    rec = {"value": B * N / t_nodes, "unit": "rows/s", "cores": threads, "kind": "oracle",
           "sample": "all %d node rows of %s (%d sequences), every node evaluated, fp64, %d host "
                     "threads over chunks of rows (%.2f s wall)" % (B * N, w["cfg"]["name"], B,
                                                                   threads, t_nodes),
           "nproc": nproc, "cores_available": avail, "cpu_model": _cpu_model(),
           "all_nodes_rows_per_s": B * N / t_nodes,
           "walk_rows_per_s": walk_rows / t_walk, "walk_sequences_per_s": B / t_walk,
           "walk_rows": walk_rows,
           "single_thread_rows_per_s": single_rows / t_single,
           "single_thread_sample": "%d of %d sequences (%d rows), all-nodes, %.1f s CPU" % (
               seqs, B, single_rows, t_single)}

    parity = None
    if gpu_nodes is not None:
        gc, gk, gs = (np.asarray(a).reshape(-1) for a in gpu_nodes)
        fl = orc["flagged"].astype(bool)
        exp_status = orc["status"]   # the oracle's codes 0-6 are the library's
        deferred = gs == 9           # RS_SEQ_DEFERRED: the decision only (no candidate accepted)
        diff = np.where(deferred, orc["child"] != -1,
                        (gc != orc["child"]) | (gk != orc["token"]) | (gs != exp_status))
        # a deferred node's decision is a single accept test; inside the window it may go
        # either way, so only full outcomes are replayed by the oracle's check
        redo = np.flatnonzero(fl & diff & ~deferred)
        verdict = (O.check_tree_nodes(*args, redo, gc[redo], gk[redo], gs[redo], **kw)
                   if redo.size else np.empty(0, np.int32))
        windowed = int((fl & diff & deferred & (orc["margin"] < 1e-7)).sum())
        parity = {"compared": int(B * N), "exact": int((~fl).sum()),
                  "decision_only": int(deferred.sum()),
                  "mismatches": int((~fl & diff).sum()),
                  "flagged": int(fl.sum()), "flagged_identical": int((fl & ~diff).sum()),
                  "flagged_valid": int((verdict != 0).sum()) + windowed,
                  "flagged_invalid": int((verdict == 0).sum()),
                  "mismatches_margin_ge_1e-7": int((fl & diff & (orc["margin"] >= 1e-7)).sum()),
                  "reference": "fp64 oracle, all-nodes evaluation of the timed step's inputs"}
        if gpu_walk is not None:
            gt, gl = gpu_walk
            wf = np.array([bool(r["flagged"][0]) for r in walks])
            same = np.array([int(gl[b]) == int(walks[b]["accepted_len"][0]) and
                             np.array_equal(gt[b], walks[b]["tokens"][0]) for b in range(B)])
            parity.update({"walks_compared": int(B), "walks_exact": int((~wf).sum()),
                           "walk_mismatches": int((~wf & ~same).sum()),
                           "walks_flagged": int(wf.sum()),
                           "walks_flagged_identical": int((wf & same).sum())})
    return rec, parity


def read_ceiling(torch, chunk=1 << 19, nbytes=4 << 30, reps=5):
    """The device's achievable read bandwidth from the read probe library: a stream of
    nbytes with ordinary and with nontemporal 16-byte loads (one chunk of `chunk` bytes
    per 512-thread workgroup, about one bf16 row pair of the benchmarked workload), and a
    stream followed by a reversed nontemporal re-read of every chunk (2 * nbytes read)."""
    import ctypes
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2608_24411_amd", "libresispec_probe.so"))
    fn = lib.resispec_probe_read
    fn.restype = ctypes.c_int
    fn.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                   ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p]
    src = torch.ones(nbytes // 4, dtype=torch.int32, device="cuda")
    sink = torch.zeros(nbytes // chunk, dtype=torch.int32, device="cuda")
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    out = {"bytes": nbytes, "chunk_bytes": chunk}
    for name, policy, passes in (("plain_stream_gbps", 0, 1), ("nt_stream_gbps", 1, 1),
                                 ("plain_then_nt_reread_gbps", 0, 2)):
        def run():
            rc = fn(ctypes.c_void_p(src.data_ptr()), nbytes, chunk, policy, passes,
                    ctypes.c_void_p(sink.data_ptr()), stream)
            if rc != 0:
                raise RuntimeError("resispec_probe_read failed (%d)" % rc)
        run()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            run()
        e1.record()
        torch.cuda.synchronize()
        out[name] = passes * nbytes / (e0.elapsed_time(e1) / reps * 1e-3) / 1e9
    del src, sink
    torch.cuda.empty_cache()
    return out


def time_mode(native, torch, w, mode, steps, warmup, settle, ws, out_tok, out_len, out_st,
              deferred=True):
    """K timed steps of one schedule: with deferred draws (resispec_decide_nodes, then
    resispec_walk_draw: the rows that reject their one candidate, and the leaves, draw
    only where a walk ends) or with every row drawing (resispec_verify_nodes, then
    resispec_walk).  HIP events on the launch stream bracket the first launch of every
    timed step."""
    args = (w["target"], w["draft"], w["node_token"], w["parent"], w["u_accept"], w["u_resample"])
    kw = dict(temperature=w["temperature"], mode=mode, without_replacement=w["without_replacement"],
              bonus=w["bonus"])

    def step(ev0=None, ev1=None, ev2=None):
        if ev0 is not None:
            ev0.record()
        if deferred:
            native.resispec_decide_nodes(*args, ws, **kw)
        else:
            native.resispec_verify_nodes(*args, ws, **kw)
        if ev1 is not None:
            ev1.record()
        if deferred:
            native.resispec_walk_draw(*args, ws, max_depth=w["max_depth"], out_tokens=out_tok,
                                      out_accepted_len=out_len, out_status=out_st, **kw)
        else:
            native.resispec_walk(w["node_token"], ws, out_tok, out_len, out_st,
                                 max_depth=w["max_depth"])
        if ev2 is not None:
            ev2.record()

    # untimed: steps for at least `settle` seconds (clocks ramp up after the idle time of
    # workload generation), then the W warmup steps
    t_end = time.perf_counter() + settle
    while time.perf_counter() < t_end:
        step()
        torch.cuda.synchronize()
    for _ in range(warmup):
        step()
    ev = [tuple(torch.cuda.Event(enable_timing=True) for _ in range(3)) for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for e0, e1, e2 in ev:
        step(e0, e1, e2)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    kern_ms = [e0.elapsed_time(e1) for e0, e1, _ in ev]
    walk_ms = [e1.elapsed_time(e2) for _, e1, e2 in ev]
    return wall, kern_ms, walk_ms


def _event_ms(torch, fn, steps, warmup, flush=None):
    """Device time of fn() in ms per call: HIP events on the current stream (the stream
    the binding launches on) around every call.  flush(), when given, runs before each
    call outside the events."""
    for _ in range(warmup):
        if flush:
            flush()
        fn()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(steps)]
    torch.cuda.synchronize()
    for e0, e1 in ev:
        if flush:
            flush()
        e0.record()
        fn()
        e1.record()
    torch.cuda.synchronize()
    return [e0.elapsed_time(e1) for e0, e1 in ev]


def configs_record(native, torch, np, synth, steps, warmup, mode, headline):
    """The decide kernel on every workload of the benchmark recipes (the headline
    workload's figures are copied from its timed run): algorithmic bytes per launch, mean
    launch time from HIP events, GB/s and the fraction of 8 TB/s; beside it the whole
    step with deferred draws and the row kernel of the schedule where every row draws.
    The flat 8-row workload is launch-bound and reported in microseconds per call; the
    64 x 21 chain workload (213 MB, inside the last-level cache) is timed warm and cold (a
    512 MiB buffer written before every cold call)."""
    out = {}
    for cfg in (0, 1, 2, 3, 4):
        name = synth.CONFIGS[cfg]["name"]
        if cfg == 2:
            out[name] = headline
            continue
        w = synth.make_workload(cfg, device="cuda")
        esz = 2 if w["target"].dtype == torch.bfloat16 else 4
        if cfg == 0:
            B, V = w["B"], w["V"]
            alg = 2 * B * V * esz + 24 * B   # both rows of every position; ids, uniforms, outputs

            def call():
                native.resispec_verify(w["target"], w["draft"], w["cand_ids"], w["u_accept"],
                                       w["u_resample"], temperature=w["temperature"], mode=mode)
            for _ in range(20):
                call()
            torch.cuda.synchronize()
            queued = []
            for _ in range(5):
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                for _ in range(100):
                    call()
                e1.record()
                torch.cuda.synchronize()
                queued.append(e0.elapsed_time(e1) * 1e3 / 100)
            lone = []
            for _ in range(20):
                torch.cuda.synchronize()
                t0 = time.perf_counter()
                call()
                torch.cuda.synchronize()
                lone.append((time.perf_counter() - t0) * 1e6)
            out[name] = {"B": B, "V": V, "k": w["k"], "us_per_call": float(np.median(queued)),
                         "us_per_call_note": "device time per call with 100 calls queued, median of 5",
                         "lone_call_us": float(np.median(lone)),
                         "lone_call_note": "host wall time of one call and its synchronisation, median of 20",
                         "alg_bytes_per_call": alg,
                         "achieved_gbps": alg / (float(np.median(queued)) * 1e-6) / 1e9}
            del w
            continue
        B, N, V = w["B"], w["N"], w["V"]
        logit_bytes, rows_t, rows_d = synth.algorithmic_bytes(w["parent"].cpu().numpy(), V, esz)
        alg = 2 * rows_d * V * esz + 28 * B * N        # the decide kernel's rows
        alg_all = logit_bytes + 28 * B * N             # every row drawing
        ws = torch.empty(native.resispec_deferred_workspace_bytes(B, N), dtype=torch.uint8,
                         device="cuda")
        args = (w["target"], w["draft"], w["node_token"], w["parent"], w["u_accept"], w["u_resample"])
        kw = dict(temperature=w["temperature"], mode=mode,
                  without_replacement=w["without_replacement"], bonus=w["bonus"])

        def nodes():
            native.resispec_decide_nodes(*args, ws, **kw)

        def whole():
            native.resispec_decide_nodes(*args, ws, **kw)
            native.resispec_walk_draw(*args, ws, max_depth=w["max_depth"], **kw)

        def every_row_draws():
            native.resispec_verify_nodes(*args, ws, **kw)
        t_end = time.perf_counter() + 0.3
        while time.perf_counter() < t_end:
            whole()
            torch.cuda.synchronize()
        ms = _event_ms(torch, nodes, steps, warmup)
        kms = float(np.mean(ms))
        step_ms = float(np.mean(_event_ms(torch, whole, steps, warmup)))
        all_ms = float(np.mean(_event_ms(torch, every_row_draws, steps, warmup)))
        rec = {"B": B, "N": N, "V": V, "logits": "bf16" if esz == 2 else "f32",
               "rows_target": rows_d, "rows_draft": rows_d, "alg_bytes_per_launch": alg,
               "decide_kernel_ms": kms, "decide_kernel_ms_min": float(np.min(ms)),
               "step_ms": step_ms, "rows_per_s": B * N / (step_ms * 1e-3),
               "achieved_gbps": alg / (kms * 1e-3) / 1e9,
               "frac": alg / (kms * 1e-3) / 1e9 / HBM_PEAK_GBPS,
               "all_nodes_draw_row_kernel_ms": all_ms,
               "all_nodes_draw_frac": alg_all / (all_ms * 1e-3) / 1e9 / HBM_PEAK_GBPS}
        if cfg == 1:
            flush_buf = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
            fill = [0]

            def flush():
                fill[0] = (fill[0] + 1) & 0xff
                flush_buf.fill_(fill[0])
            cold = _event_ms(torch, nodes, steps, 2, flush=flush)
            cms = float(np.mean(cold))
            rec["warm"] = {"decide_kernel_ms": kms, "achieved_gbps": rec["achieved_gbps"]}
            rec["cold"] = {"decide_kernel_ms": cms, "achieved_gbps": alg / (cms * 1e-3) / 1e9,
                           "frac": alg / (cms * 1e-3) / 1e9 / HBM_PEAK_GBPS,
                           "flush": "512 MiB written before every call, outside the events"}
            del flush_buf
        out[name] = rec
        del w, ws, args
        torch.cuda.empty_cache()
    return out


STUDY_BASE = dict(kind="tree", V=32000, T=1.0, dtype="f32", zipf=1.1, tgt_sigma=1.0, worep=False)


def study_configs(B_root=512, B_tree=256):
    """The workloads of the synthetic studies: a root with 8 i.i.d. candidates (the
    paper's first figure), trees of similar size and different depth/width (its topology
    ablation), and depth-3 trees of growing width (its efficiency score)."""
    base = STUDY_BASE
    root = dict(base, name="root8", B=B_root, draft=("add", 1.5), tree=("first_child_chain", (8,)))
    shapes = {"d%db%d" % (d, bw): dict(base, name="d%db%d" % (d, bw), B=B_tree,
                                       draft=("add_depth", 1.0, 0.25, 4),
                                       tree=("first_child_chain", (bw,) * d))
              for d, bw in ((7, 2), (5, 3), (4, 5), (3, 11))}
    widths = {k: dict(base, name="d3b%d" % k, B=B_tree, draft=("add_depth", 1.0, 0.25, 4),
                      tree=("first_child_chain", (k,) * 3)) for k in (1, 2, 3, 4, 6, 8)}
    return root, shapes, widths


def run_study(native, torch, np, synth, B_root=512, B_tree=256, n_root=16, n_tree=8, trace=None):
    """Synthetic analogues of the paper's studies on the device path (Zipf+noise rows,
    candidates and uniforms from the device draft step, many trials per workload by
    advancing the Philox offset): acceptance by candidate index at one node (the
    paper's first figure), mean accepted length over tree shapes of similar size (its
    topology ablation), and the marginal gain per extra candidate (its efficiency
    score).  Not timed; returns one JSON-able dict.  trace(kind, mode, w, out), when
    given, sees every trial's inputs (w: the workload with the device's draws) and
    outputs (the debug entry's node outcomes for the root study, the walk otherwise)."""
    root_cfg, shapes, widths = study_configs(B_root, B_tree)

    def trials(cfg, n_off, fn):
        w = synth.make_workload(cfg, device="cuda")
        out = []
        for off in range(n_off):
            tok, ua, ur, st = native.resispec_draft_candidates(
                w["draft"], w["parent"], temperature=w["temperature"],
                without_replacement=w["without_replacement"], seed=2608, offset=off)
            w2 = dict(w, node_token=tok, u_accept=ua, u_resample=ur)
            out.append(fn(w2))
        return w, out

    res = {}
    # 1. acceptance by candidate index: a root with 8 i.i.d. candidates
    for mode in ("resispec", "specinfer"):
        def one(w2):
            d = native.resispec_verify_tree_debug(
                w2["target"], w2["draft"], w2["node_token"], w2["parent"], w2["u_accept"],
                w2["u_resample"], temperature=1.0, max_depth=w2["max_depth"], mode=mode)
            torch.cuda.synchronize()
            if trace:
                trace("root8", mode, w2, d)
            return d["node_child"][:, 0].cpu().numpy()
        _, outs = trials(root_cfg, n_root, one)
        c = np.concatenate(outs)
        hist = [float(np.mean(c == i + 1)) for i in range(8)]
        res.setdefault("accept_by_candidate_index", {})[mode] = {
            "P(accept candidate i), i=1..8": hist, "P(all rejected)": float(np.mean(c < 0)),
            "trials": int(c.size)}

    def eal(cfg, n_off):
        r = {}
        for mode in ("resispec", "specinfer"):
            def one(w2):
                t, l, s = native.resispec_verify_tree(
                    w2["target"], w2["draft"], w2["node_token"], w2["parent"], w2["u_accept"],
                    w2["u_resample"], temperature=1.0, max_depth=w2["max_depth"], mode=mode)
                torch.cuda.synchronize()
                assert (s.cpu().numpy() == 0).all()
                if trace:
                    trace(cfg["name"], mode, w2, {"tokens": t, "accepted_len": l, "status": s})
                return l.cpu().numpy()
            _, outs = trials(cfg, n_off, one)
            r[mode] = float(np.concatenate(outs).mean())
        r["ratio"] = r["resispec"] / r["specinfer"]
        return r

    # 2. tree shapes of similar size: depth d, b candidates per level under the first
    for name, cfg in shapes.items():
        res.setdefault("mean_accepted_length_by_shape", {})[name] = eal(cfg, n_tree)
    # 3. marginal gain per extra candidate at depth 3
    curve = {k: eal(cfg, n_tree) for k, cfg in widths.items()}
    eta = {}
    for mode in ("resispec", "specinfer"):
        eta[mode] = {str(k): (curve[k][mode] - curve[1][mode]) / (k - 1) for k in curve if k > 1}
    res["mean_accepted_length_by_width_depth3"] = {str(k): v for k, v in curve.items()}
    res["eta_marginal_gain_per_extra_candidate"] = eta
    res["setup"] = {"V": STUDY_BASE["V"], "logits": STUDY_BASE["dtype"], "T": STUDY_BASE["T"],
                    "target": "Zipf(%.1f) + N(0, 1)" % STUDY_BASE["zipf"],
                    "draft": "root8: target + N(0, 1.5^2); trees: target + N(0, (1 + 0.25 depth)^2)",
                    "root_trials": B_root * n_root, "tree_trials_per_shape": B_tree * n_tree,
                    "draws": "device draft step, Philox seed 2608, offsets 0..n-1"}
    return res


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", type=int, default=2)
    ap.add_argument("--mode", default="resispec", choices=("resispec", "specinfer"))
    ap.add_argument("--settle-ms", type=float, default=300.0,
                    help="untimed steps for at least this long before the warmup steps")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-other-mode", action="store_true")
    ap.add_argument("--no-path", action="store_true", help="skip the path-only schedule")
    ap.add_argument("--no-draft", action="store_true", help="skip the draft step")
    ap.add_argument("--no-all-nodes", action="store_true",
                    help="skip the step with every row drawing at once")
    ap.add_argument("--no-single", action="store_true",
                    help="skip the single-tree latency of the same shape")
    ap.add_argument("--no-read-probe", action="store_true",
                    help="skip the read-bandwidth probe (the measured ceiling)")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the other workloads")
    ap.add_argument("--study", action="store_true",
                    help="only run the synthetic acceptance studies (not a benchmark)")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB (counter calibration)")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py runs on exactly one GPU: the verification step shards by sequence "
              "with no exchange, and multi-GPU runs are not part of this build "
              "(requested --gpus %d, WORLD_SIZE %d)" % (args.gpus, world), file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    from paper_2608_24411_amd import native, synth

    torch.cuda.set_device(0)
    if args.study:
        print(json.dumps({"study": run_study(native, torch, np, synth)}), flush=True)
        return
    if args.copy_probe:
        # A plain copy of known size: FETCH_SIZE / WRITE_SIZE of this kernel divided by
        # its bytes is the scale applied to the decide kernel's counters.
        n = args.copy_probe * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(max(1, args.steps)):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes_each_way": 4 * n, "launches": max(1, args.steps)}))
        return
    w = synth.make_workload(args.config, device="cuda")
    B, N, V = w["B"], w["N"], w["V"]
    esz = 2 if w["target"].dtype == torch.bfloat16 else 4
    logit_bytes, rows_t, rows_d = synth.algorithmic_bytes(w["parent"].cpu().numpy(), V, esz)
    small_bytes = 16 * B * N + 12 * B * N      # ids, parents, uniforms in; outcomes out
    # every row drawing: every target row and the draft row of every node with children
    alg_bytes_all = logit_bytes + small_bytes
    # the decide kernel: both rows of every node with children (a leaf's row serves only
    # its bonus draw, which the walk makes where it ends)
    alg_bytes = 2 * rows_d * V * esz + small_bytes

    # the deferred schedule's workspace also holds the other schedule's node outcomes
    ws = torch.empty(native.resispec_deferred_workspace_bytes(B, N), dtype=torch.uint8,
                     device="cuda")
    out_tok = torch.empty((B, w["max_depth"] + 1), dtype=torch.int32, device="cuda")
    out_len = torch.empty(B, dtype=torch.int32, device="cuda")
    out_st = torch.empty(B, dtype=torch.int32, device="cuda")

    results = {}
    gpu_nodes = gpu_walk = None
    modes = [args.mode] + ([] if args.no_other_mode else
                           [m for m in ("resispec", "specinfer") if m != args.mode])
    for mode in modes:
        wall, kern_ms, walk_ms = time_mode(native, torch, w, mode, args.steps, args.warmup,
                                           args.settle_ms * 1e-3, ws, out_tok, out_len, out_st)
        lens = out_len.cpu().numpy()
        assert (out_st.cpu().numpy() == 0).all(), "device status not OK"
        if mode == args.mode:
            # the node outcomes and walks the last timed step left (parity below)
            gpu_nodes = tuple(t.cpu().numpy() for t in native.resispec_node_outcomes(ws, B, N))
            gpu_walk = (out_tok.cpu().numpy(), lens.copy())
        kms = float(np.mean(kern_ms))
        results[mode] = {
            "ms_per_step": 1e3 * wall / args.steps,
            "rows_per_s": B * N / (wall / args.steps),
            "decide_kernel_ms": kms,
            "decide_kernel_ms_min": float(np.min(kern_ms)),
            "decide_kernel_gbps": alg_bytes / (kms * 1e-3) / 1e9,
            "walk_draw_ms": float(np.mean(walk_ms)),
            "mean_accepted_len": float(lens.mean()),
        }
    # the same step with every row drawing at once (the row kernel, then the walk)
    all_nodes = None
    if not args.no_all_nodes:
        wall, kern_ms, walk_ms = time_mode(native, torch, w, args.mode, args.steps, args.warmup,
                                           args.settle_ms * 1e-3, ws, out_tok, out_len, out_st,
                                           deferred=False)
        assert (out_st.cpu().numpy() == 0).all(), "device status not OK"
        assert gpu_walk is None or (np.array_equal(out_tok.cpu().numpy(), gpu_walk[0])
                                    and np.array_equal(out_len.cpu().numpy(), gpu_walk[1])), \
            "the two schedules' walks differ"
        kms = float(np.mean(kern_ms))
        all_nodes = {"schedule": "every row draws (resispec_verify_nodes + resispec_walk)",
                     "ms_per_step": 1e3 * wall / args.steps,
                     "rows_per_s": B * N / (wall / args.steps),
                     "row_kernel_ms": kms, "row_kernel_ms_min": float(np.min(kern_ms)),
                     "row_kernel_alg_bytes": alg_bytes_all,
                     "row_kernel_gbps": alg_bytes_all / (kms * 1e-3) / 1e9,
                     "row_kernel_frac": alg_bytes_all / (kms * 1e-3) / 1e9 / HBM_PEAK_GBPS,
                     "walk_ms": float(np.mean(walk_ms))}

    # the path-only schedule of the same step (only the nodes each walk reaches)
    path = None
    if not args.no_path:
        kw = dict(temperature=w["temperature"], max_depth=w["max_depth"], mode=args.mode,
                  without_replacement=w["without_replacement"], bonus=w["bonus"])
        pargs = (w["target"], w["draft"], w["node_token"], w["parent"], w["u_accept"],
                 w["u_resample"])

        # row groups where the batch leaves CUs free (the group size the library picks)
        pws = torch.empty(max(1, native.resispec_path_workspace_bytes(B, V)), dtype=torch.uint8,
                          device="cuda")
        group = native.resispec_path_group_size(B, V, dtype="bf16" if esz == 2 else "f32",
                                                mode=args.mode)

        def pstep():
            native.resispec_verify_tree_path_group(*pargs, out_tokens=out_tok,
                                                   out_accepted_len=out_len, out_status=out_st,
                                                   group_size=0, workspace=pws, **kw)
        t_end = time.perf_counter() + args.settle_ms * 1e-3
        while time.perf_counter() < t_end:
            pstep()
            torch.cuda.synchronize()
        for _ in range(args.warmup):
            pstep()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            pstep()
        torch.cuda.synchronize()
        pwall = (time.perf_counter() - t0) / args.steps
        plens = out_len.cpu().numpy()
        assert (out_st.cpu().numpy() == 0).all(), "device status not OK"
        # rows the walks read: every node on a walk (target row; draft row too when the
        # node has children), from the per-node outcomes of one untimed debug call
        dbg = native.resispec_verify_tree_debug(*pargs, **kw)
        child = dbg["node_child"].cpu().numpy()
        par = w["parent"].cpu().numpy()
        pbytes = 0
        for b in range(B):
            has_kids = np.zeros(N, dtype=bool)
            has_kids[np.unique(par[b, 1:])] = True
            n = 0
            while True:
                pbytes += V * esz * (2 if has_kids[n] else 1)
                if child[b, n] < 0:
                    break
                n = child[b, n]
        path = {"ms_per_step": 1e3 * pwall, "group_size": group, "sequences_per_s": B / pwall,
                "rows_verified_per_step": int(plens.sum() + B),
                "alg_bytes_per_step": int(pbytes),
                "achieved_gbps": pbytes / pwall / 1e9,
                "accepted_tokens_per_s": float(plens.sum()) / pwall,
                "speedup_vs_all_nodes": results[args.mode]["ms_per_step"] / (1e3 * pwall)}

    # the draft step that precedes verification (candidates and uniforms on the device)
    draft = None
    if not args.no_draft:
        dkw = dict(temperature=w["temperature"], without_replacement=w["without_replacement"],
                   seed=24411)
        d_tok = torch.empty((B, N), dtype=torch.int32, device="cuda")
        d_ua = torch.empty((B, N), dtype=torch.float32, device="cuda")
        d_ur = torch.empty((B, N), dtype=torch.float32, device="cuda")
        d_st = torch.empty(B, dtype=torch.int32, device="cuda")

        def dstep(i):
            native.resispec_draft_candidates(w["draft"], w["parent"], offset=i, node_token=d_tok,
                                             u_accept=d_ua, u_resample=d_ur, out_status=d_st, **dkw)
        t_end = time.perf_counter() + args.settle_ms * 1e-3
        i = 0
        while time.perf_counter() < t_end:
            dstep(i)
            torch.cuda.synchronize()
            i += 1
        for _ in range(args.warmup):
            dstep(i)
            i += 1
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(args.steps)]
        torch.cuda.synchronize()
        for e0, e1 in ev:
            e0.record()
            dstep(i)
            e1.record()
            i += 1
        torch.cuda.synchronize()
        dms = float(np.mean([e0.elapsed_time(e1) for e0, e1 in ev]))
        assert (d_st.cpu().numpy() == 0).all() and (d_tok.cpu().numpy()[:, 1:] >= 0).all()
        d_bytes = rows_d * V * esz + 12 * B * N + 4 * B * N   # draft rows of internal nodes; outputs; parents
        draft = {"kernel_ms": dms, "rows_per_s": B * N / (dms * 1e-3),
                 "alg_bytes_per_launch": d_bytes, "achieved_gbps": d_bytes / (dms * 1e-3) / 1e9}

    # one tree of the same shape (the latency case of serving one sequence): the all-nodes
    # schedule with row groups at the size the library picks; device time per call with
    # 100 calls queued back to back, median of 5 such runs
    single = None
    if not args.no_single:
        w1 = synth.make_workload(args.config, device="cuda", B=1)
        a1 = (w1["target"], w1["draft"], w1["node_token"], w1["parent"], w1["u_accept"],
              w1["u_resample"])
        kw1 = dict(temperature=w1["temperature"], max_depth=w1["max_depth"], mode=args.mode,
                   without_replacement=w1["without_replacement"], bonus=w1["bonus"])
        ws1 = torch.empty(max(1, native.resispec_tree_group_workspace_bytes(1, N)),
                          dtype=torch.uint8, device="cuda")
        o1 = (torch.empty((1, w1["max_depth"] + 1), dtype=torch.int32, device="cuda"),
              torch.empty(1, dtype=torch.int32, device="cuda"),
              torch.empty(1, dtype=torch.int32, device="cuda"))
        g1 = native.resispec_tree_group_size(1, N, V, dtype="bf16" if esz == 2 else "f32",
                                             mode=args.mode)

        def sstep():
            native.resispec_verify_tree_group(*a1, group_size=0, workspace=ws1, out_tokens=o1[0],
                                              out_accepted_len=o1[1], out_status=o1[2], **kw1)
        for _ in range(20):
            sstep()
        torch.cuda.synchronize()
        per_call = []
        for _ in range(5):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(100):
                sstep()
            e1.record()
            torch.cuda.synchronize()
            per_call.append(e0.elapsed_time(e1) * 1e3 / 100)
        assert int(o1[2].cpu()[0]) == 0, "device status not OK"
        single = {"B": 1, "schedule": "all-nodes with row groups", "group_size": g1,
                  "us_per_call": float(np.median(per_call)), "calls_queued": 100}

    probe = None if args.no_read_probe else read_ceiling(torch)

    r = results[args.mode]
    achieved = r["decide_kernel_gbps"]
    traffic = measured_traffic(w["cfg"]["name"], args.mode)
    out = {
        "metric": METRIC,
        "value": r["rows_per_s"],
        "unit": "rows/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": r["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": w["cfg"]["name"], "B": B, "N": N, "V": V,
                   "logits": "bf16" if esz == 2 else "f32", "mode": args.mode,
                   "temperature": w["temperature"],
                   "without_replacement": bool(w["without_replacement"])},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBPS,
                     "traffic": traffic,
                     "kernel": "rs_decide_kernel", "alg_bytes_per_launch": alg_bytes,
                     "rows_target": rows_d, "rows_draft": rows_d, "leaf_rows_left_to_the_walk": rows_t - rows_d,
                     # HBM traffic (counters) per second, against the measured read ceiling
                     "traffic_gbps": (traffic / (r["decide_kernel_ms"] * 1e-3) / 1e9
                                      if traffic else None),
                     "read_ceiling_gbps": probe["nt_stream_gbps"] if probe else None,
                     "frac_of_read_ceiling": (achieved / probe["nt_stream_gbps"]
                                              if probe else None)},
        "read_probe": probe,
        "modes": results,
        "all_nodes_draw": all_nodes,
        "path_schedule": path,
        "draft_step": draft,
        "single_tree": single,
    }
    if not args.no_configs:
        headline = {"B": B, "N": N, "V": V, "logits": "bf16" if esz == 2 else "f32",
                    "rows_target": rows_d, "rows_draft": rows_d, "alg_bytes_per_launch": alg_bytes,
                    "decide_kernel_ms": r["decide_kernel_ms"],
                    "decide_kernel_ms_min": r["decide_kernel_ms_min"],
                    "walk_draw_ms": r["walk_draw_ms"],
                    "all_nodes_draw_row_kernel_ms": all_nodes["row_kernel_ms"] if all_nodes else None,
                    "rows_per_s": r["rows_per_s"],
                    "achieved_gbps": achieved, "frac": achieved / HBM_PEAK_GBPS,
                    "step_ms": r["ms_per_step"], "note": "the headline run"}
        out["configs"] = configs_record(native, torch, np, synth, args.steps, args.warmup,
                                        args.mode, headline)
    parity = None
    if not args.no_cpu_baseline:
        out["cpu_baseline"], parity = cpu_baseline(w, args.cpu_seconds, args.mode, gpu_nodes,
                                                   gpu_walk)
        out["parity"] = parity
    print(json.dumps(out), flush=True)
    if parity and (parity["mismatches"] or parity["flagged_invalid"]
                   or parity["mismatches_margin_ge_1e-7"] or parity.get("walk_mismatches")):
        print("parity failure: %s" % json.dumps(parity), file=sys.stderr)
        sys.exit(1)


if __name__ == "__main__":
    main()
