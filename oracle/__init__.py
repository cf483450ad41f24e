"""fp64 CPU oracle of the ResiSpec verification step (numpy front end over liboracle.so).

TEST INFRASTRUCTURE ONLY.  Only the test suite, the package smoke check and the
benchmark's CPU-baseline leg may import this module.  It imports nothing from the
GPU package and the GPU package imports nothing from it; the two meet only through
the seeded input buffers the tests hand to both.

Paper anchors of each function are given in resispec_oracle.c.  Parity status:
every function here is pinned by CPU tests against values the paper or the
mathematics fix (hand-derived GetProxy examples, exact enumeration equal to p for
the standard recurrence, closed-form acceptance rates, invariants of Definition 1 /
Proposition 1 / Theorem 2, brute-force inverse CDF, library softmax).
"""
import ctypes
import os

import numpy as np

from . import build as _build

_HERE = os.path.dirname(os.path.abspath(__file__))
# an instrumented build (the sanitizer run of the CPU tests) is picked with this variable
_LIB_PATH = os.environ.get("RESISPEC_ORACLE_LIBRARY") or os.path.join(_HERE, "liboracle.so")

OK, BAD_TOKEN, ZERO_DRAFT, UNDERFLOW, BAD_TREE, BAD_UNIFORM, DEPTH_EXCEEDED = range(7)
MODE_RESISPEC, MODE_SPECINFER = 0, 1
F32, BF16 = 0, 1
KIND_ACCEPT, KIND_RESAMPLE, KIND_BONUS, KIND_NONE, KIND_FAULT = range(5)
FLAG_WINDOW = 1e-6

_MODES = {"resispec": MODE_RESISPEC, "specinfer": MODE_SPECINFER,
          MODE_RESISPEC: MODE_RESISPEC, MODE_SPECINFER: MODE_SPECINFER}


class NodeResult(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("accepted_index", ctypes.c_int32),
                ("token", ctypes.c_int32), ("status", ctypes.c_int32),
                ("n_tests", ctypes.c_int32), ("flagged", ctypes.c_int32),
                ("min_accept_margin", ctypes.c_double), ("sample_margin", ctypes.c_double)]


class ProxyInfo(ctypes.Structure):
    _fields_ = [("Z", ctypes.c_double), ("M", ctypes.c_double),
                ("delta", ctypes.c_double), ("C", ctypes.c_double)]


_lib = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        _build.build()
    lib = ctypes.CDLL(_LIB_PATH)
    P = ctypes.c_void_p
    i32, i64, f32 = ctypes.c_int32, ctypes.c_int64, ctypes.c_float
    lib.or_softmax.argtypes = [P, i32, i64, f32, P]
    lib.or_get_proxy.argtypes = [P, P, i64, i64, P, P, P, ctypes.POINTER(ProxyInfo)]
    lib.or_residual_update.argtypes = [P, P, i64, P]
    lib.or_draft_remove.argtypes = [P, i64, i64]
    lib.or_invcdf.argtypes = [P, i64, ctypes.c_double, P, P]
    lib.or_verify_node.argtypes = [P, P, i64, P, P, i32, f32, i32, i32,
                                   ctypes.POINTER(NodeResult), P]
    lib.or_check_node_outcome.argtypes = [P, P, i64, P, P, i32, f32, i32, i32, i32, i32, P]
    lib.or_check_tree_nodes.argtypes = [P, P, i32, P, P, P, P, i32, i32, i64, f32,
                                        i32, i32, i32, P, i64, P, P, P, P]
    lib.or_verify_node_batch.argtypes = [P, P, i64, P, P, P, i32, i64, i32, i32, P, P]
    lib.or_enumerate.argtypes = [P, P, i32, i32, i32, i32, P]
    lib.or_verify_tree_walk.argtypes = [P, P, i32, P, P, P, P, i32, i32, i64, i32, f32,
                                        i32, i32, i32, P, P, P, P]
    lib.or_verify_tree_nodes.argtypes = [P, P, i32, P, P, P, P, i32, i32, i64, f32,
                                         i32, i32, i32, P, i64, P, P, P, P, P, P]
    u32, u64 = ctypes.c_uint32, ctypes.c_uint64
    lib.or_philox4x32_10.argtypes = [P, P, P]
    lib.or_philox4x32_10.restype = None
    lib.or_u01.argtypes = [u32]
    lib.or_u01.restype = f32
    lib.or_node_uniforms.argtypes = [u64, u64, i32, i32, P, P, P]
    lib.or_node_uniforms.restype = None
    lib.or_sample_candidates.argtypes = [P, i32, i64, f32, i32, i32, P, P, P]
    lib.or_check_candidates.argtypes = [P, i32, i64, f32, i32, i32, P, P, P]
    lib.or_draft_tree.argtypes = [P, i32, P, i32, i32, i64, f32, i32, u64, u64, P, P, P, P, P]
    for name in ("or_softmax", "or_get_proxy", "or_residual_update", "or_draft_remove",
                 "or_invcdf", "or_verify_node", "or_verify_node_batch", "or_enumerate",
                 "or_verify_tree_walk", "or_verify_tree_nodes", "or_sample_candidates",
                 "or_check_node_outcome", "or_check_tree_nodes", "or_check_candidates",
                 "or_draft_tree"):
        getattr(lib, name).restype = i32
    _lib = lib
    return lib


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p) if a is not None else None


def _logits(a):
    """float32 array, or bf16 given as uint16 bit patterns."""
    a = np.ascontiguousarray(a)
    if a.dtype == np.float32:
        return a, F32
    if a.dtype == np.uint16:
        return a, BF16
    raise TypeError("logits must be float32 or uint16 (bf16 bit patterns), got %s" % a.dtype)


def softmax(logits, temperature):
    a, dt = _logits(logits)
    out = np.empty(a.shape[-1], dtype=np.float64)
    st = _load().or_softmax(_ptr(a), dt, a.shape[-1], float(temperature), _ptr(out))
    if st not in (OK, UNDERFLOW):
        raise ValueError("or_softmax failed (%d)" % st)
    return out


def get_proxy(R, D, x0):
    R, D = _f64(R), _f64(D)
    V = R.shape[0]
    r, s, K = np.empty(V), np.empty(V), np.empty(V)
    info = ProxyInfo()
    st = _load().or_get_proxy(_ptr(R), _ptr(D), V, int(x0), _ptr(r), _ptr(s), _ptr(K),
                              ctypes.byref(info))
    if st != OK:
        raise ValueError("or_get_proxy failed (%d)" % st)
    return {"r": r, "s": s, "K": K, "Z": info.Z, "M": info.M, "delta": info.delta, "C": info.C}


def residual_update(R, K):
    R, K = _f64(R), _f64(K)
    out = np.empty_like(R)
    st = _load().or_residual_update(_ptr(R), _ptr(K), R.shape[0], _ptr(out))
    return out, st


def draft_remove(D, x):
    D = _f64(D).copy()
    st = _load().or_draft_remove(_ptr(D), D.shape[0], int(x))
    return D, st


def invcdf(R, u):
    R = _f64(R)
    tok = ctypes.c_int32(-1)
    margin = ctypes.c_double(0.0)
    st = _load().or_invcdf(_ptr(R), R.shape[0], float(u), ctypes.byref(tok), ctypes.byref(margin))
    return tok.value, margin.value, st


def verify_node(p, q, cand, ua, ur, mode="resispec", without_replacement=False,
                want_residual=False):
    p = _f64(p)
    V = p.shape[0]
    cand = np.ascontiguousarray(cand, dtype=np.int32)
    ua = np.ascontiguousarray(ua, dtype=np.float32)
    b = cand.shape[0]
    q = _f64(q) if q is not None else np.zeros(V)
    res = NodeResult()
    fr = np.empty(V) if want_residual else None
    st = _load().or_verify_node(_ptr(p), _ptr(q), V, _ptr(cand), _ptr(ua), b, float(ur),
                                _MODES[mode], int(bool(without_replacement)),
                                ctypes.byref(res), _ptr(fr))
    if st != OK:
        raise ValueError("or_verify_node failed (%d)" % st)
    out = {f[0]: getattr(res, f[0]) for f in NodeResult._fields_}
    if want_residual:
        out["final_R"] = fr
    return out


def check_node_outcome(p, q, cand, ua, ur, claim_index, claim_token, mode="resispec",
                       without_replacement=False):
    """Whether a claimed outcome of one node is admissible with decisions inside the flag
    window free to go either way: 1 (agrees outside the window), 2 (only through a
    windowed decision), 0 (not admissible)."""
    p = _f64(p)
    V = p.shape[0]
    cand = np.ascontiguousarray(cand, dtype=np.int32)
    ua = np.ascontiguousarray(ua, dtype=np.float32)
    q = _f64(q) if q is not None else np.zeros(V)
    verdict = ctypes.c_int32(-1)
    st = _load().or_check_node_outcome(_ptr(p), _ptr(q), V, _ptr(cand), _ptr(ua), cand.shape[0],
                                       float(ur), _MODES[mode], int(bool(without_replacement)),
                                       int(claim_index), int(claim_token), ctypes.byref(verdict))
    if st != OK:
        raise ValueError("or_check_node_outcome failed (%d)" % st)
    return verdict.value


def verify_node_batch(p, q, cand, ua, ur, mode="resispec", without_replacement=False):
    p, q = _f64(p), _f64(q)
    cand = np.ascontiguousarray(cand, dtype=np.int32)
    ua = np.ascontiguousarray(ua, dtype=np.float32)
    ur = np.ascontiguousarray(ur, dtype=np.float32)
    n, b = cand.shape
    tok = np.empty(n, dtype=np.int32)
    acc = np.empty(n, dtype=np.int32)
    st = _load().or_verify_node_batch(_ptr(p), _ptr(q), p.shape[0], _ptr(cand), _ptr(ua),
                                      _ptr(ur), b, n, _MODES[mode], int(bool(without_replacement)),
                                      _ptr(tok), _ptr(acc))
    if st != OK:
        raise ValueError("or_verify_node_batch failed (%d)" % st)
    return tok, acc


def enumerate_output(p, q, k, mode="resispec", without_replacement=False):
    p, q = _f64(p), _f64(q)
    out = np.empty_like(p)
    st = _load().or_enumerate(_ptr(p), _ptr(q), p.shape[0], int(k), _MODES[mode],
                              int(bool(without_replacement)), _ptr(out))
    if st != OK:
        raise ValueError("or_enumerate failed (%d)" % st)
    return out


def _tree_inputs(target, draft, node_token, parent, u_accept, u_resample):
    t, dt = _logits(target)
    d, dd = _logits(draft)
    if dt != dd or t.shape != d.shape or t.ndim != 3:
        raise ValueError("target/draft must share dtype and [B,N,V] shape")
    tok = np.ascontiguousarray(node_token, dtype=np.int32)
    par = np.ascontiguousarray(parent, dtype=np.int32)
    ua = np.ascontiguousarray(u_accept, dtype=np.float32)
    ur = np.ascontiguousarray(u_resample, dtype=np.float32)
    return t, d, dt, tok, par, ua, ur


def verify_tree_walk(target, draft, node_token, parent, u_accept, u_resample, *,
                     temperature, max_depth, mode="resispec", without_replacement=False,
                     bonus=True):
    t, d, dt, tok, par, ua, ur = _tree_inputs(target, draft, node_token, parent, u_accept,
                                              u_resample)
    B, N, V = t.shape
    out_tok = np.empty((B, max_depth + 1), dtype=np.int32)
    out_len = np.empty(B, dtype=np.int32)
    out_st = np.empty(B, dtype=np.int32)
    out_fl = np.empty(B, dtype=np.int32)
    st = _load().or_verify_tree_walk(_ptr(t), _ptr(d), dt, _ptr(tok), _ptr(par), _ptr(ua),
                                     _ptr(ur), B, N, V, int(max_depth), float(temperature),
                                     _MODES[mode], int(bool(without_replacement)),
                                     int(bool(bonus)), _ptr(out_tok), _ptr(out_len),
                                     _ptr(out_st), _ptr(out_fl))
    if st != OK:
        raise ValueError("or_verify_tree_walk failed (%d)" % st)
    return {"tokens": out_tok, "accepted_len": out_len, "status": out_st, "flagged": out_fl}


def verify_tree_nodes(target, draft, node_token, parent, u_accept, u_resample, rows, *,
                      temperature, mode="resispec", without_replacement=False, bonus=True,
                      want_residual=False):
    t, d, dt, tok, par, ua, ur = _tree_inputs(target, draft, node_token, parent, u_accept,
                                              u_resample)
    B, N, V = t.shape
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    n = rows.shape[0]
    child = np.empty(n, dtype=np.int32)
    token = np.empty(n, dtype=np.int32)
    status = np.empty(n, dtype=np.int32)
    flagged = np.empty(n, dtype=np.int32)
    margin = np.empty(n, dtype=np.float64)
    fr = np.empty((n, V)) if want_residual else None
    st = _load().or_verify_tree_nodes(_ptr(t), _ptr(d), dt, _ptr(tok), _ptr(par), _ptr(ua),
                                      _ptr(ur), B, N, V, float(temperature), _MODES[mode],
                                      int(bool(without_replacement)), int(bool(bonus)),
                                      _ptr(rows), n, _ptr(child), _ptr(token), _ptr(status),
                                      _ptr(flagged), _ptr(margin), _ptr(fr))
    if st != OK:
        raise ValueError("or_verify_tree_nodes failed (%d)" % st)
    out = {"child": child, "token": token, "status": status, "flagged": flagged,
           "margin": margin}
    if want_residual:
        out["final_R"] = fr
    return out


def check_tree_nodes(target, draft, node_token, parent, u_accept, u_resample, rows, claim_child,
                     claim_token, claim_status, *, temperature, mode="resispec",
                     without_replacement=False, bonus=True):
    """Verdicts (1, 2 or 0 as in check_node_outcome) of claimed (child, token, status)
    outcomes of the given rows."""
    t, d, dt, tok, par, ua, ur = _tree_inputs(target, draft, node_token, parent, u_accept,
                                              u_resample)
    B, N, V = t.shape
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    cc = np.ascontiguousarray(claim_child, dtype=np.int32)
    ct = np.ascontiguousarray(claim_token, dtype=np.int32)
    cs = np.ascontiguousarray(claim_status, dtype=np.int32)
    if not (rows.shape == cc.shape == ct.shape == cs.shape):
        raise ValueError("rows and claims must have one entry each")
    verdict = np.empty(rows.shape[0], dtype=np.int32)
    st = _load().or_check_tree_nodes(_ptr(t), _ptr(d), dt, _ptr(tok), _ptr(par), _ptr(ua),
                                     _ptr(ur), B, N, V, float(temperature), _MODES[mode],
                                     int(bool(without_replacement)), int(bool(bonus)),
                                     _ptr(rows), rows.shape[0], _ptr(cc), _ptr(ct), _ptr(cs),
                                     _ptr(verdict))
    if st != OK:
        raise ValueError("or_check_tree_nodes failed (%d)" % st)
    return verdict


# ------------------------------------------------------------------ draft step ----

def philox4x32_10(counter, key):
    """Philox4x32-10 of a 4-word counter under a 2-word key -> 4 uint32 words."""
    c = np.ascontiguousarray(counter, dtype=np.uint32)
    k = np.ascontiguousarray(key, dtype=np.uint32)
    out = np.empty(4, dtype=np.uint32)
    _load().or_philox4x32_10(_ptr(c), _ptr(k), _ptr(out))
    return out


def u01(word):
    return _load().or_u01(int(word))


def node_uniforms(seed, offset, b, n):
    """(u_accept, u_resample, u_cand) of node n of sequence b."""
    ua, ur, uc = ctypes.c_float(), ctypes.c_float(), ctypes.c_float()
    _load().or_node_uniforms(int(seed), int(offset), int(b), int(n), ctypes.byref(ua),
                             ctypes.byref(ur), ctypes.byref(uc))
    return ua.value, ur.value, uc.value


def sample_candidates(draft_row, k, uc, *, temperature, without_replacement=False):
    a, dt = _logits(draft_row)
    uc = np.ascontiguousarray(uc, dtype=np.float32)
    tok = np.empty(k, dtype=np.int32)
    mg = np.empty(k, dtype=np.float64)
    st = _load().or_sample_candidates(_ptr(a), dt, a.shape[-1], float(temperature), int(k),
                                      int(bool(without_replacement)), _ptr(uc), _ptr(tok), _ptr(mg))
    return tok, mg, st


def check_candidates(draft_row, claimed, uc, *, temperature, without_replacement=False):
    """Verdict (1 exact, 2 admissible through a windowed draw, 0 not admissible) of
    claimed candidate draws from one draft row with uniforms uc."""
    a, dt = _logits(draft_row)
    claimed = np.ascontiguousarray(claimed, dtype=np.int32)
    uc = np.ascontiguousarray(uc, dtype=np.float32)
    verdict = ctypes.c_int32(-1)
    st = _load().or_check_candidates(_ptr(a), dt, a.shape[-1], float(temperature),
                                     claimed.shape[0], int(bool(without_replacement)), _ptr(uc),
                                     _ptr(claimed), ctypes.byref(verdict))
    if st != OK:
        raise ValueError("or_check_candidates failed (%d)" % st)
    return verdict.value


def draft_tree(draft, parent, *, temperature, without_replacement=False, seed=0, offset=0):
    """The draft step of a tree batch: node_token, u_accept, u_resample, flagged, margin
    (all [B, N]) and the status (OK or BAD_TREE)."""
    d, dt = _logits(draft)
    par = np.ascontiguousarray(parent, dtype=np.int32)
    B, N, V = d.shape
    tok = np.empty((B, N), dtype=np.int32)
    ua = np.empty((B, N), dtype=np.float32)
    ur = np.empty((B, N), dtype=np.float32)
    fl = np.empty((B, N), dtype=np.int32)
    mg = np.empty((B, N), dtype=np.float64)
    st = _load().or_draft_tree(_ptr(d), dt, _ptr(par), B, N, V, float(temperature),
                               int(bool(without_replacement)), int(seed), int(offset), _ptr(tok),
                               _ptr(ua), _ptr(ur), _ptr(fl), _ptr(mg))
    return {"node_token": tok, "u_accept": ua, "u_resample": ur, "flagged": fl, "margin": mg,
            "status": st}
