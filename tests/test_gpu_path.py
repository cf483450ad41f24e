"""Path-only schedule (resispec_verify_tree_path): one workgroup per sequence verifies
only the nodes its walk reaches.  Its tokens, lengths and statuses must equal the
all-nodes schedule's bit for bit (the per-node outcome is the same function of the
node's rows and uniforms), and the oracle's walk on unflagged sequences."""
import numpy as np
import pytest
import torch

from paper_2608_24411_amd import synth
from parity_util import compare_walk, gpu_tree, host_tree, oracle_walk

pytestmark = pytest.mark.gpu
MODES = ("resispec", "specinfer")


def _log(*a):
    print(*a, flush=True)


def path_tree(native, w, mode, max_depth=None, bonus=True):
    md = w["max_depth"] if max_depth is None else max_depth
    t, l, s = native.resispec_verify_tree_path(
        w["target"], w["draft"], w["node_token"], w["parent"], w["u_accept"], w["u_resample"],
        temperature=w["temperature"], max_depth=md, mode=mode,
        without_replacement=w["without_replacement"], bonus=bonus)
    torch.cuda.synchronize()
    return {"tokens": t, "accepted_len": l, "status": s}


def same(a, b):
    for k in ("tokens", "accepted_len", "status"):
        assert torch.equal(a[k], b[k]), k


CASES = [(1, dict(B=8)), (2, dict(B=4)), (3, dict(B=3)), (4, dict(B=8)),
         (1, dict(B=4, V=32003)), (2, dict(B=2, V=100003, dtype="f32")),
         (3, dict(B=2, V=65537, dtype="bf16")), (4, dict(B=3, V=4099))]


@pytest.mark.parametrize("cfg,over", CASES, ids=[f"cfg{c}-{o}" for c, o in CASES])
@pytest.mark.parametrize("mode", MODES)
def test_path_equals_all_nodes_and_oracle(gpu_lib, cfg, over, mode):
    _log("path parity", cfg, over, mode)
    w = synth.make_workload(cfg, device="cuda", **over)
    p = path_tree(gpu_lib, w, mode)
    same(p, gpu_tree(gpu_lib, w, mode))
    compare_walk(p, oracle_walk(host_tree(w), w, mode))


@pytest.mark.parametrize("cfg", [2, 4])
def test_path_full_size(gpu_lib, cfg):
    """Full configurations: the path schedule equals the all-nodes schedule."""
    _log("path full size", cfg)
    w = synth.make_workload(cfg, device="cuda")
    for mode in MODES:
        p = path_tree(gpu_lib, w, mode)
        same(p, gpu_tree(gpu_lib, w, mode))
        assert (p["status"].cpu().numpy() == 0).all()


def test_path_edges(gpu_lib):
    """Faults met on the walk, bonus off, a short max_depth, root-only trees, B = 0."""
    w = synth.make_workload(1, device="cuda", B=6, V=3001)
    w["u_accept"][2, 1:5] = 0.999
    w["node_token"][3, 2] = 3001
    w["parent"][4, 7] = 9
    w["u_resample"][5, :] = 1.0
    h = host_tree(w)
    for mode in MODES:
        for bonus in (True, False):
            p = path_tree(gpu_lib, w, mode, bonus=bonus)
            same(p, gpu_tree(gpu_lib, w, mode, bonus=bonus))
            compare_walk(p, oracle_walk(h, w, mode, bonus=bonus))
        short = path_tree(gpu_lib, w, mode, max_depth=1)
        same(short, gpu_tree(gpu_lib, w, mode, max_depth=1))
        assert p["status"].cpu().numpy()[4] == 4
    w1 = synth.make_workload(1, device="cuda", B=5, V=777)
    for k in ("target", "draft", "node_token", "parent", "u_accept", "u_resample"):
        w1[k] = w1[k][:, :1].contiguous()
    w1["max_depth"] = 0
    p = path_tree(gpu_lib, w1, "resispec")
    same(p, gpu_tree(gpu_lib, w1, "resispec"))
    assert (p["accepted_len"].cpu() == 0).all()
    e = {k: (v[:0] if isinstance(v, torch.Tensor) else v) for k, v in w.items()}
    t, l, s = gpu_lib.resispec_verify_tree_path(e["target"], e["draft"], e["node_token"],
                                                e["parent"], e["u_accept"], e["u_resample"],
                                                temperature=1.0, max_depth=5)
    torch.cuda.synchronize()
    assert t.numel() == 0


def test_path_side_stream(gpu_lib):
    w = synth.make_workload(3, device="cuda", B=4, V=20000)
    ref = path_tree(gpu_lib, w, "resispec")
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        t, l, st = gpu_lib.resispec_verify_tree_path(
            w["target"], w["draft"], w["node_token"], w["parent"], w["u_accept"],
            w["u_resample"], temperature=w["temperature"], max_depth=w["max_depth"],
            stream=s)
    s.synchronize()
    assert torch.equal(t, ref["tokens"]) and torch.equal(l, ref["accepted_len"])
