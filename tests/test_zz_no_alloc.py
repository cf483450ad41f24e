"""The entry point that allocates nothing (resispec_verify_tree_noalloc) against
resispec_verify_tree: the same kernels, so the same outputs bit for bit, on two calls in a
row with the second on a smaller batch (the shared scratch keeps the first call's
contents), in both modes; and the size limit."""
import pytest
import torch

from paper_2608_24411_amd import native, synth

pytestmark = pytest.mark.gpu


def _outs(B, md):
    return (torch.full((B, md + 1), -7, dtype=torch.int32, device="cuda"),
            torch.full((B,), -7, dtype=torch.int32, device="cuda"),
            torch.full((B,), -7, dtype=torch.int32, device="cuda"))


@pytest.mark.parametrize("mode", ["resispec", "specinfer"])
def test_noalloc_equals_verify_tree(gpu_lib, mode):
    for cfg, over in ((4, dict(B=40, V=20000)), (2, dict(B=3, V=40003)), (3, dict(B=2))):
        w = synth.make_workload(cfg, device="cuda", **over)
        args = (w["target"], w["draft"], w["node_token"], w["parent"], w["u_accept"],
                w["u_resample"])
        kw = dict(temperature=w["temperature"], max_depth=w["max_depth"], mode=mode,
                  without_replacement=w["without_replacement"])
        rt, rl, rs = gpu_lib.resispec_verify_tree(*args, **kw)
        ot, ol, os_ = _outs(w["B"], w["max_depth"])
        gpu_lib.resispec_verify_tree_noalloc(*args, out_tokens=ot, out_accepted_len=ol,
                                             out_status=os_, **kw)
        torch.cuda.synchronize()
        print("no-alloc", cfg, over, mode, "rows", w["B"] * w["N"], flush=True)
        assert torch.equal(ot, rt) and torch.equal(ol, rl) and torch.equal(os_, rs)
        assert (rs.cpu() == 0).all()


def test_noalloc_size_limit(gpu_lib):
    B, N, V = native.RS_NOALLOC_MAX_ROWS + 1, 1, 8
    t = torch.zeros((B, N, V), dtype=torch.float32, device="cuda")
    par = torch.full((B, N), -1, dtype=torch.int32, device="cuda")
    tok = torch.zeros((B, N), dtype=torch.int32, device="cuda")
    u = torch.zeros((B, N), dtype=torch.float32, device="cuda")
    ot, ol, os_ = _outs(B, 0)
    with pytest.raises(native.ResiSpecError):
        gpu_lib.resispec_verify_tree_noalloc(t, t, tok, par, u, u, temperature=1.0, max_depth=0,
                                             out_tokens=ot, out_accepted_len=ol, out_status=os_)
    torch.cuda.synchronize()
    assert (ol.cpu() == -7).all()     # nothing was launched
    # at the limit it runs (root-only trees draw their bonus token)
    B = native.RS_NOALLOC_MAX_ROWS
    ot, ol, os_ = _outs(B, 0)
    t = torch.randn((B, N, V), device="cuda")
    gpu_lib.resispec_verify_tree_noalloc(t, t, tok[:B], par[:B], u[:B], u[:B], temperature=1.0,
                                         max_depth=0, out_tokens=ot, out_accepted_len=ol,
                                         out_status=os_)
    rt, rl, rs = gpu_lib.resispec_verify_tree(t, t, tok[:B], par[:B], u[:B], u[:B],
                                              temperature=1.0, max_depth=0)
    torch.cuda.synchronize()
    assert torch.equal(ot, rt) and torch.equal(ol, rl) and torch.equal(os_, rs)
