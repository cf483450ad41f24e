"""Python binding of libresispec.so: argument marshalling only.

Every entry point of include/resispec.h has a function of the same name here.  Torch
is used for device memory and the current HIP stream; every step of the verification
runs in the library's kernels.  There is no fallback: if the library cannot be loaded
the import fails.
"""
import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
# an instrumented build (the sanitizer run of the CPU tests) is picked with this variable
LIB_PATH = os.environ.get("RESISPEC_LIBRARY") or os.path.join(HERE, "libresispec.so")

RS_OK, RS_ERR_INVALID_ARG, RS_ERR_WORKSPACE, RS_ERR_UNSUPPORTED, RS_ERR_HIP = range(5)
(RS_SEQ_OK, RS_SEQ_BAD_TOKEN, RS_SEQ_ZERO_DRAFT, RS_SEQ_UNDERFLOW, RS_SEQ_BAD_TREE,
 RS_SEQ_BAD_UNIFORM, RS_SEQ_DEPTH_EXCEEDED, RS_SEQ_TOO_MANY_CHILDREN, RS_SEQ_GROUP_TIMEOUT,
 RS_SEQ_DEFERRED) = range(10)
RS_MODE_RESISPEC, RS_MODE_SPECINFER = 0, 1
RS_F32, RS_BF16 = 0, 1
RS_MAX_CANDIDATES = 64

MODES = {"resispec": RS_MODE_RESISPEC, "specinfer": RS_MODE_SPECINFER}

# Every symbol include/resispec.h declares.
EXPORTS = ("resispec_verify", "resispec_verify_tree", "resispec_verify_tree_noalloc",
           "resispec_verify_tree_deferred", "resispec_decide_nodes", "resispec_walk_draw",
           "resispec_deferred_workspace_bytes",
           "resispec_verify_tree_path",
           "resispec_verify_tree_path_group", "resispec_path_workspace_bytes",
           "resispec_path_group_size", "resispec_debug_set_group_waits",
           "resispec_verify_tree_group", "resispec_tree_group_workspace_bytes",
           "resispec_tree_group_size",
           "resispec_draft_candidates",
           "resispec_verify_nodes", "resispec_walk", "resispec_node_outcomes",
           "resispec_workspace_bytes", "resispec_validate_tree_host",
           "resispec_verify_tree_debug", "resispec_status_string", "resispec_abi_version")


class RsParams(ctypes.Structure):
    _fields_ = [("mode", ctypes.c_int32), ("logits_dtype", ctypes.c_int32),
                ("temperature", ctypes.c_float), ("without_replacement", ctypes.c_int32),
                ("bonus", ctypes.c_int32)]


class ResiSpecError(RuntimeError):
    pass


def _load():
    if not os.path.exists(LIB_PATH):
        from . import build as _build
        _build.build()
    lib = ctypes.CDLL(LIB_PATH)
    P, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    prm = ctypes.POINTER(RsParams)
    lib.resispec_verify.argtypes = [P, P, P, P, P, i32, i32, i32, prm, P, P, P, P]
    lib.resispec_verify.restype = i32
    lib.resispec_verify_tree.argtypes = [P, P, P, P, P, P, i32, i32, i32, i32, prm, P, P, P,
                                         P, sz, P]
    lib.resispec_verify_tree.restype = i32
    lib.resispec_verify_tree_noalloc.argtypes = [P, P, P, P, P, P, i32, i32, i32, i32, prm, P, P,
                                                 P, P]
    lib.resispec_verify_tree_noalloc.restype = i32
    lib.resispec_verify_tree_path.argtypes = [P, P, P, P, P, P, i32, i32, i32, i32, prm, P, P, P,
                                              P]
    lib.resispec_verify_tree_path.restype = i32
    lib.resispec_verify_tree_path_group.argtypes = [P, P, P, P, P, P, i32, i32, i32, i32, prm, P,
                                                    P, P, i32, P, sz, P]
    lib.resispec_verify_tree_path_group.restype = i32
    lib.resispec_path_workspace_bytes.argtypes = [i32, i32]
    lib.resispec_path_workspace_bytes.restype = sz
    lib.resispec_path_group_size.argtypes = [i32, i32, prm]
    lib.resispec_path_group_size.restype = i32
    lib.resispec_debug_set_group_waits.argtypes = [ctypes.c_uint64, ctypes.c_uint64]
    lib.resispec_debug_set_group_waits.restype = i32
    lib.resispec_verify_tree_group.argtypes = [P, P, P, P, P, P, i32, i32, i32, i32, prm, P, P, P,
                                               i32, P, sz, P]
    lib.resispec_verify_tree_group.restype = i32
    lib.resispec_tree_group_workspace_bytes.argtypes = [i32, i32]
    lib.resispec_tree_group_workspace_bytes.restype = sz
    lib.resispec_tree_group_size.argtypes = [i32, i32, i32, prm]
    lib.resispec_tree_group_size.restype = i32
    lib.resispec_draft_candidates.argtypes = [P, P, i32, i32, i32, prm, ctypes.c_uint64,
                                              ctypes.c_uint64, P, P, P, P, P]
    lib.resispec_draft_candidates.restype = i32
    lib.resispec_verify_tree_debug.argtypes = [P, P, P, P, P, P, i32, i32, i32, i32, prm, P, P,
                                               P, P, sz, P, P, P, P, P]
    lib.resispec_verify_tree_debug.restype = i32
    lib.resispec_verify_tree_deferred.argtypes = [P, P, P, P, P, P, i32, i32, i32, i32, prm, P, P,
                                                  P, P, sz, P]
    lib.resispec_verify_tree_deferred.restype = i32
    lib.resispec_decide_nodes.argtypes = [P, P, P, P, P, P, i32, i32, i32, prm, P, sz, P]
    lib.resispec_decide_nodes.restype = i32
    lib.resispec_walk_draw.argtypes = [P, P, P, P, P, P, i32, i32, i32, i32, prm, P, sz, P, P, P, P]
    lib.resispec_walk_draw.restype = i32
    lib.resispec_deferred_workspace_bytes.argtypes = [i32, i32]
    lib.resispec_deferred_workspace_bytes.restype = sz
    lib.resispec_verify_nodes.argtypes = [P, P, P, P, P, P, i32, i32, i32, prm, P, sz, P]
    lib.resispec_verify_nodes.restype = i32
    lib.resispec_walk.argtypes = [P, i32, i32, i32, P, sz, P, P, P, P]
    lib.resispec_walk.restype = i32
    lib.resispec_node_outcomes.argtypes = [P, sz, i32, i32, P, P, P, P]
    lib.resispec_node_outcomes.restype = i32
    lib.resispec_workspace_bytes.argtypes = [i32, i32]
    lib.resispec_workspace_bytes.restype = sz
    lib.resispec_validate_tree_host.argtypes = [P, P, i32, i32, i32, ctypes.POINTER(i64)]
    lib.resispec_validate_tree_host.restype = i32
    lib.resispec_status_string.argtypes = [i32]
    lib.resispec_status_string.restype = ctypes.c_char_p
    lib.resispec_abi_version.argtypes = []
    lib.resispec_abi_version.restype = i32
    return lib


lib = _load()


# ------------------------------------------------------------ plain entries --

def resispec_status_string(status: int) -> str:
    return lib.resispec_status_string(int(status)).decode()


def resispec_abi_version() -> int:
    return lib.resispec_abi_version()


def resispec_workspace_bytes(B: int, N: int) -> int:
    return lib.resispec_workspace_bytes(int(B), int(N))


def resispec_validate_tree_host(parent, node_token, V: int):
    """parent, node_token: host int32 arrays [B, N] (numpy).  Returns (status, first_bad)."""
    import numpy as np
    par = np.ascontiguousarray(parent, dtype=np.int32)
    tok = np.ascontiguousarray(node_token, dtype=np.int32)
    B, N = par.shape
    bad = ctypes.c_int64(-1)
    st = lib.resispec_validate_tree_host(par.ctypes.data, tok.ctypes.data, B, N, int(V),
                                         ctypes.byref(bad))
    return st, bad.value


# ------------------------------------------------------- torch marshalling --

def _params(logits, temperature, mode, without_replacement, bonus):
    import torch
    if logits.dtype == torch.float32:
        dt = RS_F32
    elif logits.dtype == torch.bfloat16:
        dt = RS_BF16
    else:
        raise TypeError("logits must be float32 or bfloat16")
    return RsParams(MODES[mode] if isinstance(mode, str) else int(mode), dt, float(temperature),
                    int(bool(without_replacement)), int(bool(bonus)))


def _dev(t, dtype, name):
    import torch
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError("%s must be a device tensor" % name)
    if t.dtype != dtype:
        raise TypeError("%s must be %s" % (name, dtype))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    return t.data_ptr()


def _shape(t, shape, name):
    if tuple(t.shape) != tuple(shape):
        raise ValueError("%s has shape %s, expected %s" % (name, tuple(t.shape), tuple(shape)))


def _same_device(*ts):
    devs = {t.device for t in ts if t is not None}
    if len(devs) > 1:
        raise ValueError("all tensors must be on one device, got %s" % devs)


def _check_tree_shapes(target_logits, draft_logits, node_token, parent, u_accept, u_resample):
    if target_logits.dim() != 3:
        raise ValueError("target_logits must be [B, N, V]")
    B, N, V = target_logits.shape
    _shape(draft_logits, (B, N, V), "draft_logits")
    for t, name in ((node_token, "node_token"), (parent, "parent"), (u_accept, "u_accept"),
                    (u_resample, "u_resample")):
        _shape(t, (B, N), name)
    _same_device(target_logits, draft_logits, node_token, parent, u_accept, u_resample)
    return B, N, V


def _stream(stream):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _check(st):
    if st != RS_OK:
        raise ResiSpecError(resispec_status_string(st))


def resispec_verify(target_logits, draft_logits, cand_ids, u_accept, u_resample, *,
                    temperature, mode="resispec", out_token=None, out_accepted_len=None,
                    out_status=None, stream=None):
    """Flat verify of B rows with k candidates each; returns (token, accepted_len, status)."""
    import torch
    if target_logits.dim() != 2 or cand_ids.dim() != 2:
        raise ValueError("target_logits must be [B, V] and cand_ids [B, k]")
    B, V = target_logits.shape
    k = cand_ids.shape[1]
    _shape(draft_logits, (B, V), "draft_logits")
    _shape(cand_ids, (B, k), "cand_ids")
    _shape(u_accept, (B, k), "u_accept")
    _shape(u_resample, (B,), "u_resample")
    _same_device(target_logits, draft_logits, cand_ids, u_accept, u_resample)
    dev = target_logits.device
    if out_token is None:
        out_token = torch.empty(B, dtype=torch.int32, device=dev)
    if out_accepted_len is None:
        out_accepted_len = torch.empty(B, dtype=torch.int32, device=dev)
    if out_status is None:
        out_status = torch.empty(B, dtype=torch.int32, device=dev)
    for t, name in ((out_token, "out_token"), (out_accepted_len, "out_accepted_len"),
                    (out_status, "out_status")):
        _shape(t, (B,), name)
    prm = _params(target_logits, temperature, mode, False, True)
    st = lib.resispec_verify(
        _dev(target_logits, target_logits.dtype, "target_logits"),
        _dev(draft_logits, target_logits.dtype, "draft_logits"),
        _dev(cand_ids, torch.int32, "cand_ids"), _dev(u_accept, torch.float32, "u_accept"),
        _dev(u_resample, torch.float32, "u_resample"), B, V, k, ctypes.byref(prm),
        _dev(out_token, torch.int32, "out_token"),
        _dev(out_accepted_len, torch.int32, "out_accepted_len"),
        _dev(out_status, torch.int32, "out_status"), _stream(stream))
    _check(st)
    return out_token, out_accepted_len, out_status


def _tree_common(target_logits, draft_logits, node_token, parent, u_accept, u_resample,
                 max_depth):
    if max_depth is None or int(max_depth) < 0:
        raise ValueError("max_depth (>= 0) is required")
    return _check_tree_shapes(target_logits, draft_logits, node_token, parent, u_accept,
                              u_resample)


def resispec_verify_tree(target_logits, draft_logits, node_token, parent, u_accept, u_resample,
                         *, temperature, max_depth, mode="resispec", without_replacement=False,
                         bonus=True, out_tokens=None, out_accepted_len=None, out_status=None,
                         workspace=None, stream=None):
    """Tree verify; returns (tokens [B, max_depth+1], accepted_len [B], status [B])."""
    import torch
    B, N, V = _tree_common(target_logits, draft_logits, node_token, parent, u_accept, u_resample,
                           max_depth)
    dev = target_logits.device
    if out_tokens is None:
        out_tokens = torch.empty((B, max_depth + 1), dtype=torch.int32, device=dev)
    if out_accepted_len is None:
        out_accepted_len = torch.empty(B, dtype=torch.int32, device=dev)
    if out_status is None:
        out_status = torch.empty(B, dtype=torch.int32, device=dev)
    _shape(out_tokens, (B, max_depth + 1), "out_tokens")
    _shape(out_accepted_len, (B,), "out_accepted_len")
    _shape(out_status, (B,), "out_status")
    wsb = resispec_workspace_bytes(B, N)
    if workspace is None:
        workspace = torch.empty(max(wsb, 1), dtype=torch.uint8, device=dev)
    prm = _params(target_logits, temperature, mode, without_replacement, bonus)
    st = lib.resispec_verify_tree(
        _dev(target_logits, target_logits.dtype, "target_logits"),
        _dev(draft_logits, target_logits.dtype, "draft_logits"),
        _dev(node_token, torch.int32, "node_token"), _dev(parent, torch.int32, "parent"),
        _dev(u_accept, torch.float32, "u_accept"), _dev(u_resample, torch.float32, "u_resample"),
        B, N, V, int(max_depth), ctypes.byref(prm),
        _dev(out_tokens, torch.int32, "out_tokens"),
        _dev(out_accepted_len, torch.int32, "out_accepted_len"),
        _dev(out_status, torch.int32, "out_status"),
        _dev(workspace, torch.uint8, "workspace"), workspace.numel(), _stream(stream))
    _check(st)
    return out_tokens, out_accepted_len, out_status


RS_NOALLOC_MAX_ROWS = 65536


def resispec_verify_tree_noalloc(target_logits, draft_logits, node_token, parent, u_accept,
                                 u_resample, *, temperature, max_depth, mode="resispec",
                                 without_replacement=False, bonus=True, out_tokens, out_accepted_len,
                                 out_status=None, stream=None):
    """resispec_verify_tree with the library's static per-GPU scratch instead of a
    workspace (B * N <= RS_NOALLOC_MAX_ROWS); the caller passes the outputs.  Calls that
    overlap on one GPU race."""
    import torch
    B, N, V = _tree_common(target_logits, draft_logits, node_token, parent, u_accept, u_resample,
                           max_depth)
    _shape(out_tokens, (B, max_depth + 1), "out_tokens")
    _shape(out_accepted_len, (B,), "out_accepted_len")
    if out_status is not None:
        _shape(out_status, (B,), "out_status")
    prm = _params(target_logits, temperature, mode, without_replacement, bonus)
    st = lib.resispec_verify_tree_noalloc(
        _dev(target_logits, target_logits.dtype, "target_logits"),
        _dev(draft_logits, target_logits.dtype, "draft_logits"),
        _dev(node_token, torch.int32, "node_token"), _dev(parent, torch.int32, "parent"),
        _dev(u_accept, torch.float32, "u_accept"), _dev(u_resample, torch.float32, "u_resample"),
        B, N, V, int(max_depth), ctypes.byref(prm),
        _dev(out_tokens, torch.int32, "out_tokens"),
        _dev(out_accepted_len, torch.int32, "out_accepted_len"),
        _dev(out_status, torch.int32, "out_status") if out_status is not None else None,
        _stream(stream))
    _check(st)
    return out_tokens, out_accepted_len, out_status


def resispec_verify_tree_path(target_logits, draft_logits, node_token, parent, u_accept,
                              u_resample, *, temperature, max_depth, mode="resispec",
                              without_replacement=False, bonus=True, out_tokens=None,
                              out_accepted_len=None, out_status=None, stream=None):
    """Path-only schedule of resispec_verify_tree (same results); returns
    (tokens [B, max_depth+1], accepted_len [B], status [B])."""
    import torch
    B, N, V = _tree_common(target_logits, draft_logits, node_token, parent, u_accept, u_resample,
                           max_depth)
    dev = target_logits.device
    if out_tokens is None:
        out_tokens = torch.empty((B, max_depth + 1), dtype=torch.int32, device=dev)
    if out_accepted_len is None:
        out_accepted_len = torch.empty(B, dtype=torch.int32, device=dev)
    if out_status is None:
        out_status = torch.empty(B, dtype=torch.int32, device=dev)
    _shape(out_tokens, (B, max_depth + 1), "out_tokens")
    _shape(out_accepted_len, (B,), "out_accepted_len")
    _shape(out_status, (B,), "out_status")
    prm = _params(target_logits, temperature, mode, without_replacement, bonus)
    st = lib.resispec_verify_tree_path(
        _dev(target_logits, target_logits.dtype, "target_logits"),
        _dev(draft_logits, target_logits.dtype, "draft_logits"),
        _dev(node_token, torch.int32, "node_token"), _dev(parent, torch.int32, "parent"),
        _dev(u_accept, torch.float32, "u_accept"), _dev(u_resample, torch.float32, "u_resample"),
        B, N, V, int(max_depth), ctypes.byref(prm),
        _dev(out_tokens, torch.int32, "out_tokens"),
        _dev(out_accepted_len, torch.int32, "out_accepted_len"),
        _dev(out_status, torch.int32, "out_status"), _stream(stream))
    _check(st)
    return out_tokens, out_accepted_len, out_status


def resispec_path_workspace_bytes(B: int, V: int) -> int:
    return lib.resispec_path_workspace_bytes(int(B), int(V))


def resispec_path_group_size(B: int, V: int, *, dtype, mode="resispec") -> int:
    """Members per sequence the grouped path schedule picks by itself (dtype: "bf16" or
    "f32"); -1 for invalid arguments."""
    prm = RsParams(MODES[mode], RS_BF16 if dtype == "bf16" else RS_F32, 1.0, 0, 1)
    return lib.resispec_path_group_size(int(B), int(V), ctypes.byref(prm))


def resispec_tree_group_workspace_bytes(B: int, N: int) -> int:
    return lib.resispec_tree_group_workspace_bytes(int(B), int(N))


def resispec_tree_group_size(B: int, N: int, V: int, *, dtype, mode="resispec") -> int:
    """Members per row the grouped all-nodes schedule picks by itself (dtype: "bf16" or
    "f32"); -1 for invalid arguments."""
    prm = RsParams(MODES[mode], RS_BF16 if dtype == "bf16" else RS_F32, 1.0, 0, 1)
    return lib.resispec_tree_group_size(int(B), int(N), int(V), ctypes.byref(prm))


def resispec_verify_tree_group(target_logits, draft_logits, node_token, parent, u_accept,
                               u_resample, *, temperature, max_depth, mode="resispec",
                               without_replacement=False, bonus=True, group_size=0,
                               workspace=None, out_tokens=None, out_accepted_len=None,
                               out_status=None, stream=None):
    """All-nodes verification with row groups (group_size workgroups per node row, 0 =
    automatic); same results as resispec_verify_tree.  Returns (tokens [B, max_depth+1],
    accepted_len [B], status [B])."""
    import torch
    B, N, V = _tree_common(target_logits, draft_logits, node_token, parent, u_accept, u_resample,
                           max_depth)
    dev = target_logits.device
    if out_tokens is None:
        out_tokens = torch.empty((B, max_depth + 1), dtype=torch.int32, device=dev)
    if out_accepted_len is None:
        out_accepted_len = torch.empty(B, dtype=torch.int32, device=dev)
    if out_status is None:
        out_status = torch.empty(B, dtype=torch.int32, device=dev)
    if workspace is None:
        workspace = torch.empty(max(1, resispec_tree_group_workspace_bytes(B, N)),
                                dtype=torch.uint8, device=dev)
    _shape(out_tokens, (B, max_depth + 1), "out_tokens")
    _shape(out_accepted_len, (B,), "out_accepted_len")
    _shape(out_status, (B,), "out_status")
    prm = _params(target_logits, temperature, mode, without_replacement, bonus)
    st = lib.resispec_verify_tree_group(
        _dev(target_logits, target_logits.dtype, "target_logits"),
        _dev(draft_logits, target_logits.dtype, "draft_logits"),
        _dev(node_token, torch.int32, "node_token"), _dev(parent, torch.int32, "parent"),
        _dev(u_accept, torch.float32, "u_accept"), _dev(u_resample, torch.float32, "u_resample"),
        B, N, V, int(max_depth), ctypes.byref(prm),
        _dev(out_tokens, torch.int32, "out_tokens"),
        _dev(out_accepted_len, torch.int32, "out_accepted_len"),
        _dev(out_status, torch.int32, "out_status"), int(group_size),
        _dev(workspace, torch.uint8, "workspace"), workspace.numel(), _stream(stream))
    _check(st)
    return out_tokens, out_accepted_len, out_status


def resispec_debug_set_group_waits(barrier=None, formation=None) -> None:
    """Testing hook: time limits of row groups in later launches (ticks of the 100 MHz
    device clock): `barrier` for every wait of a formed group for its members' slot
    totals, `formation` for its workgroups to start.  None restores a default (20 ms,
    20 us)."""
    none = (1 << 64) - 1
    _check(lib.resispec_debug_set_group_waits(
        ctypes.c_uint64(none if barrier is None else int(barrier)),
        ctypes.c_uint64(none if formation is None else int(formation))))


def resispec_verify_tree_path_group(target_logits, draft_logits, node_token, parent, u_accept,
                                    u_resample, *, temperature, max_depth, mode="resispec",
                                    without_replacement=False, bonus=True, group_size=0,
                                    workspace=None, out_tokens=None, out_accepted_len=None,
                                    out_status=None, stream=None):
    """Path-only schedule with row groups (group_size workgroups per sequence, 0 =
    automatic); same results as resispec_verify_tree_path.  Returns (tokens [B,
    max_depth+1], accepted_len [B], status [B])."""
    import torch
    B, N, V = _tree_common(target_logits, draft_logits, node_token, parent, u_accept, u_resample,
                           max_depth)
    dev = target_logits.device
    if out_tokens is None:
        out_tokens = torch.empty((B, max_depth + 1), dtype=torch.int32, device=dev)
    if out_accepted_len is None:
        out_accepted_len = torch.empty(B, dtype=torch.int32, device=dev)
    if out_status is None:
        out_status = torch.empty(B, dtype=torch.int32, device=dev)
    if workspace is None:
        workspace = torch.empty(max(1, resispec_path_workspace_bytes(B, V)), dtype=torch.uint8,
                                device=dev)
    _shape(out_tokens, (B, max_depth + 1), "out_tokens")
    _shape(out_accepted_len, (B,), "out_accepted_len")
    _shape(out_status, (B,), "out_status")
    prm = _params(target_logits, temperature, mode, without_replacement, bonus)
    st = lib.resispec_verify_tree_path_group(
        _dev(target_logits, target_logits.dtype, "target_logits"),
        _dev(draft_logits, target_logits.dtype, "draft_logits"),
        _dev(node_token, torch.int32, "node_token"), _dev(parent, torch.int32, "parent"),
        _dev(u_accept, torch.float32, "u_accept"), _dev(u_resample, torch.float32, "u_resample"),
        B, N, V, int(max_depth), ctypes.byref(prm),
        _dev(out_tokens, torch.int32, "out_tokens"),
        _dev(out_accepted_len, torch.int32, "out_accepted_len"),
        _dev(out_status, torch.int32, "out_status"), int(group_size),
        _dev(workspace, torch.uint8, "workspace"), workspace.numel(), _stream(stream))
    _check(st)
    return out_tokens, out_accepted_len, out_status


def resispec_draft_candidates(draft_logits, parent, *, temperature, without_replacement=False,
                              seed=0, offset=0, node_token=None, u_accept=None, u_resample=None,
                              out_status=None, stream=None):
    """The draft step on the device: children's candidate tokens drawn from each node's
    draft row, and every node's uniforms (Philox4x32-10 under seed / offset).
    Returns (node_token [B, N], u_accept [B, N], u_resample [B, N], status [B])."""
    import torch
    if draft_logits.dim() != 3:
        raise ValueError("draft_logits must be [B, N, V]")
    B, N, V = draft_logits.shape
    _shape(parent, (B, N), "parent")
    dev = draft_logits.device
    _same_device(draft_logits, parent, node_token, u_accept, u_resample, out_status)
    if node_token is None:
        node_token = torch.empty((B, N), dtype=torch.int32, device=dev)
    if u_accept is None:
        u_accept = torch.empty((B, N), dtype=torch.float32, device=dev)
    if u_resample is None:
        u_resample = torch.empty((B, N), dtype=torch.float32, device=dev)
    if out_status is None:
        out_status = torch.empty(B, dtype=torch.int32, device=dev)
    for t, nm in ((node_token, "node_token"), (u_accept, "u_accept"), (u_resample, "u_resample")):
        _shape(t, (B, N), nm)
    _shape(out_status, (B,), "out_status")
    prm = _params(draft_logits, temperature, "resispec", without_replacement, False)
    st = lib.resispec_draft_candidates(
        _dev(draft_logits, draft_logits.dtype, "draft_logits"), _dev(parent, torch.int32, "parent"),
        B, N, V, ctypes.byref(prm), int(seed) & 0xFFFFFFFFFFFFFFFF, int(offset) & 0xFFFFFFFFFFFFFFFF,
        _dev(node_token, torch.int32, "node_token"), _dev(u_accept, torch.float32, "u_accept"),
        _dev(u_resample, torch.float32, "u_resample"), _dev(out_status, torch.int32, "out_status"),
        _stream(stream))
    _check(st)
    return node_token, u_accept, u_resample, out_status


def resispec_deferred_workspace_bytes(B: int, N: int) -> int:
    return lib.resispec_deferred_workspace_bytes(int(B), int(N))


def _logit_args(target_logits, draft_logits, node_token, parent, u_accept, u_resample):
    import torch
    return (_dev(target_logits, target_logits.dtype, "target_logits"),
            _dev(draft_logits, target_logits.dtype, "draft_logits"),
            _dev(node_token, torch.int32, "node_token"), _dev(parent, torch.int32, "parent"),
            _dev(u_accept, torch.float32, "u_accept"), _dev(u_resample, torch.float32, "u_resample"))


def _tree_outputs(B, max_depth, dev, out_tokens, out_accepted_len, out_status):
    import torch
    if out_tokens is None:
        out_tokens = torch.empty((B, max_depth + 1), dtype=torch.int32, device=dev)
    if out_accepted_len is None:
        out_accepted_len = torch.empty(B, dtype=torch.int32, device=dev)
    if out_status is None:
        out_status = torch.empty(B, dtype=torch.int32, device=dev)
    _shape(out_tokens, (B, max_depth + 1), "out_tokens")
    _shape(out_accepted_len, (B,), "out_accepted_len")
    _shape(out_status, (B,), "out_status")
    return out_tokens, out_accepted_len, out_status


def resispec_verify_tree_deferred(target_logits, draft_logits, node_token, parent, u_accept,
                                  u_resample, *, temperature, max_depth, mode="resispec",
                                  without_replacement=False, bonus=True, out_tokens=None,
                                  out_accepted_len=None, out_status=None, workspace=None,
                                  stream=None):
    """resispec_verify_tree with deferred draws (a row's draw made only where a walk ends);
    returns (tokens [B, max_depth+1], accepted_len [B], status [B])."""
    import torch
    B, N, V = _tree_common(target_logits, draft_logits, node_token, parent, u_accept, u_resample,
                           max_depth)
    dev = target_logits.device
    out_tokens, out_accepted_len, out_status = _tree_outputs(B, max_depth, dev, out_tokens,
                                                             out_accepted_len, out_status)
    if workspace is None:
        workspace = torch.empty(max(resispec_deferred_workspace_bytes(B, N), 1),
                                dtype=torch.uint8, device=dev)
    prm = _params(target_logits, temperature, mode, without_replacement, bonus)
    st = lib.resispec_verify_tree_deferred(
        *_logit_args(target_logits, draft_logits, node_token, parent, u_accept, u_resample),
        B, N, V, int(max_depth), ctypes.byref(prm),
        _dev(out_tokens, torch.int32, "out_tokens"),
        _dev(out_accepted_len, torch.int32, "out_accepted_len"),
        _dev(out_status, torch.int32, "out_status"),
        _dev(workspace, torch.uint8, "workspace"), workspace.numel(), _stream(stream))
    _check(st)
    return out_tokens, out_accepted_len, out_status


def resispec_decide_nodes(target_logits, draft_logits, node_token, parent, u_accept, u_resample,
                          workspace, *, temperature, mode="resispec", without_replacement=False,
                          bonus=True, stream=None):
    """First launch of resispec_verify_tree_deferred: every node's tests into `workspace`
    (resispec_deferred_workspace_bytes), draws deferred where they can be."""
    import torch
    B, N, V = _check_tree_shapes(target_logits, draft_logits, node_token, parent, u_accept,
                                 u_resample)
    prm = _params(target_logits, temperature, mode, without_replacement, bonus)
    st = lib.resispec_decide_nodes(
        *_logit_args(target_logits, draft_logits, node_token, parent, u_accept, u_resample),
        B, N, V, ctypes.byref(prm), _dev(workspace, torch.uint8, "workspace"), workspace.numel(),
        _stream(stream))
    _check(st)


def resispec_walk_draw(target_logits, draft_logits, node_token, parent, u_accept, u_resample,
                       workspace, *, temperature, max_depth, mode="resispec",
                       without_replacement=False, bonus=True, out_tokens=None,
                       out_accepted_len=None, out_status=None, stream=None):
    """Second launch of resispec_verify_tree_deferred: the walks, with the deferred draw
    where a walk ends; returns (tokens, accepted_len, status)."""
    import torch
    B, N, V = _tree_common(target_logits, draft_logits, node_token, parent, u_accept, u_resample,
                           max_depth)
    out_tokens, out_accepted_len, out_status = _tree_outputs(B, max_depth, target_logits.device,
                                                             out_tokens, out_accepted_len,
                                                             out_status)
    prm = _params(target_logits, temperature, mode, without_replacement, bonus)
    st = lib.resispec_walk_draw(
        *_logit_args(target_logits, draft_logits, node_token, parent, u_accept, u_resample),
        B, N, V, int(max_depth), ctypes.byref(prm), _dev(workspace, torch.uint8, "workspace"),
        workspace.numel(), _dev(out_tokens, torch.int32, "out_tokens"),
        _dev(out_accepted_len, torch.int32, "out_accepted_len"),
        _dev(out_status, torch.int32, "out_status"), _stream(stream))
    _check(st)
    return out_tokens, out_accepted_len, out_status


def resispec_verify_nodes(target_logits, draft_logits, node_token, parent, u_accept, u_resample,
                          workspace, *, temperature, mode="resispec", without_replacement=False,
                          bonus=True, stream=None):
    """First stage of resispec_verify_tree: every node's outcome into `workspace`."""
    import torch
    B, N, V = _check_tree_shapes(target_logits, draft_logits, node_token, parent, u_accept,
                                 u_resample)
    prm = _params(target_logits, temperature, mode, without_replacement, bonus)
    st = lib.resispec_verify_nodes(
        _dev(target_logits, target_logits.dtype, "target_logits"),
        _dev(draft_logits, target_logits.dtype, "draft_logits"),
        _dev(node_token, torch.int32, "node_token"), _dev(parent, torch.int32, "parent"),
        _dev(u_accept, torch.float32, "u_accept"), _dev(u_resample, torch.float32, "u_resample"),
        B, N, V, ctypes.byref(prm), _dev(workspace, torch.uint8, "workspace"), workspace.numel(),
        _stream(stream))
    _check(st)


def resispec_walk(node_token, workspace, out_tokens, out_accepted_len, out_status=None, *,
                  max_depth, stream=None):
    """Second stage of resispec_verify_tree: walk every root over the node outcomes."""
    import torch
    B, N = node_token.shape
    _shape(out_tokens, (B, int(max_depth) + 1), "out_tokens")
    _shape(out_accepted_len, (B,), "out_accepted_len")
    if out_status is not None:
        _shape(out_status, (B,), "out_status")
    st = lib.resispec_walk(
        _dev(node_token, torch.int32, "node_token"), B, N, int(max_depth),
        _dev(workspace, torch.uint8, "workspace"), workspace.numel(),
        _dev(out_tokens, torch.int32, "out_tokens"),
        _dev(out_accepted_len, torch.int32, "out_accepted_len"),
        _dev(out_status, torch.int32, "out_status") if out_status is not None else None,
        _stream(stream))
    _check(st)


def resispec_node_outcomes(workspace, B: int, N: int, *, stream=None):
    """Every node's outcome left in `workspace` by resispec_verify_nodes, or by
    resispec_decide_nodes (and resispec_walk_draw, which fills in the nodes it draws for;
    the others report RS_SEQ_DEFERRED): (node_child, node_token, node_status), [B, N]
    int32 each."""
    import torch
    dev = workspace.device
    out = [torch.empty((B, N), dtype=torch.int32, device=dev) for _ in range(3)]
    st = lib.resispec_node_outcomes(_dev(workspace, torch.uint8, "workspace"), workspace.numel(),
                                    int(B), int(N), *[o.data_ptr() for o in out], _stream(stream))
    _check(st)
    return tuple(out)


def resispec_verify_tree_debug(target_logits, draft_logits, node_token, parent, u_accept,
                               u_resample, *, temperature, max_depth, mode="resispec",
                               without_replacement=False, bonus=True, want_residual=False,
                               stream=None):
    """Tree verify that also returns every node's outcome (and optionally the normalised
    distribution each drawing node sampled from)."""
    import torch
    B, N, V = _tree_common(target_logits, draft_logits, node_token, parent, u_accept, u_resample,
                           max_depth)
    dev = target_logits.device
    out_tokens = torch.empty((B, max_depth + 1), dtype=torch.int32, device=dev)
    out_len = torch.empty(B, dtype=torch.int32, device=dev)
    out_status = torch.empty(B, dtype=torch.int32, device=dev)
    node_child = torch.empty((B, N), dtype=torch.int32, device=dev)
    node_tok = torch.empty((B, N), dtype=torch.int32, device=dev)
    node_status = torch.empty((B, N), dtype=torch.int32, device=dev)
    resid = torch.empty((B, N, V), dtype=torch.float32, device=dev) if want_residual else None
    prm = _params(target_logits, temperature, mode, without_replacement, bonus)
    st = lib.resispec_verify_tree_debug(
        _dev(target_logits, target_logits.dtype, "target_logits"),
        _dev(draft_logits, target_logits.dtype, "draft_logits"),
        _dev(node_token, torch.int32, "node_token"), _dev(parent, torch.int32, "parent"),
        _dev(u_accept, torch.float32, "u_accept"), _dev(u_resample, torch.float32, "u_resample"),
        B, N, V, int(max_depth), ctypes.byref(prm), out_tokens.data_ptr(), out_len.data_ptr(),
        out_status.data_ptr(), None, 0, node_child.data_ptr(), node_tok.data_ptr(),
        node_status.data_ptr(), resid.data_ptr() if resid is not None else None, _stream(stream))
    _check(st)
    return {"tokens": out_tokens, "accepted_len": out_len, "status": out_status,
            "node_child": node_child, "node_token": node_tok, "node_status": node_status,
            "residual": resid}
