"""HIP graph capture of the entry points (GPU).

The entry points allocate nothing, take every buffer from the caller and clear their
counters with a kernel, so a serving loop can capture a step once and replay it without
the host's per-call cost.  Each test captures a step into a graph, then replays it
several times with eager work and synchronisations in between, and checks every replay
against an eager call on the same inputs: the first replay on the captured inputs, the
next after new uniforms were written into the same buffers (the graph must read them),
the last on the captured inputs again.
"""
import pytest
import torch

from paper_2608_24411_amd import synth

pytestmark = pytest.mark.gpu


def _log(*a):
    print(*a, flush=True)


def _same(a, b):
    for k in ("tokens", "accepted_len", "status"):
        assert torch.equal(a[k], b[k]), (k, a[k], b[k])


def _capture(fn):
    """Warm up on a side stream of default priority, then capture fn() into a graph."""
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for _ in range(2):
            fn()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    torch.cuda.synchronize()
    return g


def _outputs(B, max_depth):
    return {"tokens": torch.empty((B, max_depth + 1), dtype=torch.int32, device="cuda"),
            "accepted_len": torch.empty(B, dtype=torch.int32, device="cuda"),
            "status": torch.empty(B, dtype=torch.int32, device="cuda")}


def _check_replays(w, step, name):
    """step(out) runs one verification of w into the dict of output tensors out."""
    static = _outputs(w["B"], w["max_depth"])
    g = _capture(lambda: step(static))
    u0 = w["u_accept"].clone()
    u1 = torch.rand_like(u0)
    for i, u in enumerate((u0, u1, u0)):
        w["u_accept"].copy_(u)
        ref = _outputs(w["B"], w["max_depth"])
        step(ref)                      # eager, on the same buffers
        torch.cuda.synchronize()
        for k in static:
            static[k].fill_(-7)
        g.replay()
        torch.cuda.synchronize()
        _log(name, "replay", i, "accepted lengths", static["accepted_len"][:8].tolist())
        _same(static, ref)
    w["u_accept"].copy_(u0)


def _tree_args(w):
    return (w["target"], w["draft"], w["node_token"], w["parent"], w["u_accept"], w["u_resample"])


def _kw(w, mode):
    return dict(temperature=w["temperature"], max_depth=w["max_depth"], mode=mode,
                without_replacement=w["without_replacement"])


@pytest.mark.parametrize("mode", ["resispec", "specinfer"])
def test_graph_all_nodes(gpu_lib, mode):
    w = synth.make_workload(2, device="cuda", B=4, V=40000)
    ws = torch.empty(gpu_lib.resispec_workspace_bytes(w["B"], w["N"]), dtype=torch.uint8,
                     device="cuda")

    def step(out):
        gpu_lib.resispec_verify_tree(*_tree_args(w), **_kw(w, mode), workspace=ws,
                                     out_tokens=out["tokens"], out_accepted_len=out["accepted_len"],
                                     out_status=out["status"])
    _check_replays(w, step, "all-nodes " + mode)


@pytest.mark.parametrize("mode", ["resispec", "specinfer"])
def test_graph_deferred(gpu_lib, mode):
    """The all-nodes schedule with deferred draws: both launches in the graph; replays whose
    new uniforms move the walks' ends to other rows still agree with eager calls."""
    w = synth.make_workload(2, device="cuda", B=4, V=40000)
    ws = torch.empty(gpu_lib.resispec_deferred_workspace_bytes(w["B"], w["N"]), dtype=torch.uint8,
                     device="cuda")

    def step(out):
        gpu_lib.resispec_verify_tree_deferred(*_tree_args(w), **_kw(w, mode), workspace=ws,
                                              out_tokens=out["tokens"],
                                              out_accepted_len=out["accepted_len"],
                                              out_status=out["status"])
    _check_replays(w, step, "deferred " + mode)


@pytest.mark.parametrize("mode", ["resispec", "specinfer"])
def test_graph_path_groups(gpu_lib, mode):
    """The path schedule with row groups: the counter-clearing kernel and the group launch
    are both in the graph."""
    w = synth.make_workload(4, device="cuda", B=3, V=40000)
    ws = torch.empty(gpu_lib.resispec_path_workspace_bytes(w["B"], w["V"]), dtype=torch.uint8,
                     device="cuda")

    def step(out):
        gpu_lib.resispec_verify_tree_path_group(
            *_tree_args(w), **_kw(w, mode), group_size=3, workspace=ws,
            out_tokens=out["tokens"], out_accepted_len=out["accepted_len"],
            out_status=out["status"])
    _check_replays(w, step, "path groups " + mode)


def test_graph_row_groups(gpu_lib):
    w = synth.make_workload(2, device="cuda", B=1)
    ws = torch.empty(gpu_lib.resispec_tree_group_workspace_bytes(w["B"], w["N"]),
                     dtype=torch.uint8, device="cuda")

    def step(out):
        gpu_lib.resispec_verify_tree_group(
            *_tree_args(w), **_kw(w, "resispec"), group_size=0, workspace=ws,
            out_tokens=out["tokens"], out_accepted_len=out["accepted_len"],
            out_status=out["status"])
    _check_replays(w, step, "row groups")


def test_graph_draft_then_verify(gpu_lib):
    """The device hand-off in one graph: the draft step writes every node's token and
    uniforms, the path schedule verifies them.  Replays with a new seed offset are
    compared with eager calls."""
    w = synth.make_workload(2, device="cuda", B=4, V=40000)
    B, N = w["B"], w["N"]
    tok = torch.empty((B, N), dtype=torch.int32, device="cuda")
    ua = torch.empty((B, N), dtype=torch.float32, device="cuda")
    ur = torch.empty((B, N), dtype=torch.float32, device="cuda")
    dst = torch.empty(B, dtype=torch.int32, device="cuda")

    def step(out, offset):
        gpu_lib.resispec_draft_candidates(w["draft"], w["parent"], temperature=w["temperature"],
                                          without_replacement=w["without_replacement"],
                                          seed=24411, offset=offset, node_token=tok, u_accept=ua,
                                          u_resample=ur, out_status=dst)
        gpu_lib.resispec_verify_tree_path(w["target"], w["draft"], tok, w["parent"], ua, ur,
                                          **_kw(w, "resispec"), out_tokens=out["tokens"],
                                          out_accepted_len=out["accepted_len"],
                                          out_status=out["status"])
    static = _outputs(B, w["max_depth"])
    g = _capture(lambda: step(static, 7))
    for i in range(3):
        ref = _outputs(B, w["max_depth"])
        step(ref, 7)
        torch.cuda.synchronize()
        ref_tok = tok.clone()
        step(_outputs(B, w["max_depth"]), 100 + i)   # other eager work on the same buffers
        torch.cuda.synchronize()
        for k in static:
            static[k].fill_(-7)
        g.replay()
        torch.cuda.synchronize()
        _log("draft then verify, replay", i, static["accepted_len"].tolist())
        assert torch.equal(tok, ref_tok)
        _same(static, ref)


def test_binding_stream_is_torch_current_stream(gpu_lib):
    """The binding launches on torch's current stream: the default one, a side stream in a
    stream context, and the capture stream (covered by the graph tests above)."""
    from paper_2608_24411_amd import native

    def handle(stream):
        return native._stream(stream).value or 0   # a NULL handle reads as None
    assert handle(None) == torch.cuda.current_stream().cuda_stream
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):
        assert handle(None) == side.cuda_stream
        assert handle(None) == torch.cuda.current_stream().cuda_stream
    assert handle(side) == side.cuda_stream
