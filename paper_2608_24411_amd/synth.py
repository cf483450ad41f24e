"""Seeded synthetic workloads (logits, trees, candidates, uniforms).

This module holds none of the verification arithmetic.  It stands in for the paper's
models and datasets (Llama-2 / Llama-68M / EAGLE drafters on CNN/DM, OpenWebText, C4),
which are not available: target logits follow a Zipf law over a random per-row rank
permutation plus Gaussian noise, draft logits are noisy copies of the target, and
candidates are drawn from the draft's temperature softmax with the Gumbel-max trick
(Gumbel-top-k for draws without replacement).  Sequence b of a batch uses seed
`seed + b`, as the paper's reproducibility protocol seeds the i-th prompt with s + i.

Workloads (one per evaluation configuration):
  0  flat      B=8,    V=32000,  k=4 i.i.d.,          T=1.0, fp32, Zipf 1.1, draft sigma 1.5
  1  chain     B=64,   N=21, V=32000, depth 5, 4 candidates per level under the first
               candidate, T=1.0, fp32, Zipf 1.1, draft sigma 1.0 + 0.25 * depth (1.0 -> 2.0)
  2  wide      B=128,  N=33, V=128256, root with 8 i.i.d. children each continued by a
               3-node chain, T=0.7, bf16, Zipf 1.0, draft sigma 1.25
  3  dynamic   B=32,   N=60, V=128256, random breadth-first trees (depth <= 6, branching
               1/2/3/4 with probability .4/.3/.2/.1), T=1.0, fp32, Zipf 1.1,
               draft = 0.8 * target + N(0, 1)
  4  serving   B=1024, N=26, V=151936, widths 10/8/5/2 along the first-ranked path,
               without replacement, T=0.8, bf16, Zipf 1.2 with N(0, 1.5^2) noise, draft
               sigma 1.5
"""
import numpy as np
import torch

SEED = 24411

CONFIGS = {
    0: dict(name="flat-b8-v32000-f32", kind="flat", B=8, V=32000, k=4, T=1.0, dtype="f32",
            zipf=1.1, tgt_sigma=1.0, draft=("add", 1.5), worep=False),
    1: dict(name="chain-b64-n21-v32000-f32", kind="tree", B=64, V=32000, T=1.0, dtype="f32",
            zipf=1.1, tgt_sigma=1.0, draft=("add_depth", 1.0, 0.25, 4),
            tree=("first_child_chain", (4, 4, 4, 4, 4)), worep=False),
    2: dict(name="wide-b128-n33-v128256-bf16", kind="tree", B=128, V=128256, T=0.7,
            dtype="bf16", zipf=1.0, tgt_sigma=1.0, draft=("add", 1.25),
            tree=("fan_chains", 8, 3), worep=False),
    3: dict(name="dynamic-b32-n60-v128256-f32", kind="tree", B=32, V=128256, T=1.0,
            dtype="f32", zipf=1.1, tgt_sigma=1.0, draft=("corr", 0.8, 1.0),
            tree=("random_bfs", 60, 6, (0.4, 0.3, 0.2, 0.1)), worep=False),
    4: dict(name="serving-b1024-n26-v151936-bf16", kind="tree", B=1024, V=151936, T=0.8,
            dtype="bf16", zipf=1.2, tgt_sigma=1.5, draft=("add", 1.5),
            tree=("first_child_chain", (10, 8, 5, 2)), worep=True),
}


# ----------------------------------------------------------------- trees ----

def first_child_chain(widths):
    """Root gets widths[0] children; the first child of each expanded node gets the next
    width.  Breadth-first numbering."""
    parent = [-1]
    expand = 0
    for w in widths:
        first = len(parent)
        parent.extend([expand] * w)
        expand = first
    return np.array(parent, dtype=np.int32)


def fan_chains(fan, chain):
    """Root with `fan` children, each continued by a chain of `chain` single children."""
    parent = [-1] + [0] * fan
    prev = list(range(1, fan + 1))
    for _ in range(chain):
        cur = []
        for p in prev:
            cur.append(len(parent))
            parent.append(p)
        prev = cur
    return np.array(parent, dtype=np.int32)


def random_bfs(rng, n_nodes, max_depth, probs):
    """Breadth-first random tree; every expanded node draws its branching factor from
    {1, .., len(probs)}.  Redrawn until it reaches n_nodes nodes."""
    while True:
        parent = [-1]
        depth = [0]
        head = 0
        while head < len(parent) and len(parent) < n_nodes:
            if depth[head] < max_depth:
                nb = int(rng.choice(len(probs), p=probs)) + 1
                for _ in range(nb):
                    if len(parent) == n_nodes:
                        break
                    parent.append(head)
                    depth.append(depth[head] + 1)
            head += 1
        if len(parent) == n_nodes:
            return np.array(parent, dtype=np.int32)


def depths(parent):
    d = np.zeros(len(parent), dtype=np.int64)
    for n in range(1, len(parent)):
        d[n] = d[parent[n]] + 1
    return d


def tree_for(cfg, b, seed, N=None):
    kind = cfg["tree"][0]
    if kind == "first_child_chain":
        return first_child_chain(cfg["tree"][1])
    if kind == "fan_chains":
        return fan_chains(cfg["tree"][1], cfg["tree"][2])
    if kind == "random_bfs":
        rng = np.random.default_rng([seed + b, 7])
        return random_bfs(rng, N or cfg["tree"][1], cfg["tree"][2], np.array(cfg["tree"][3]))
    raise ValueError(kind)


# ---------------------------------------------------------------- logits ----

def _zipf_rows(g, rows, V, a, sigma, device):
    """-a * ln(rank) over a random rank permutation per row, plus N(0, sigma^2)."""
    keys = torch.rand((rows, V), generator=g, device=device)
    perm = torch.argsort(keys, dim=1)
    ladder = -a * torch.log(torch.arange(1, V + 1, device=device, dtype=torch.float32))
    t = torch.empty((rows, V), device=device, dtype=torch.float32)
    t.scatter_(1, perm, ladder.expand(rows, V).contiguous())
    t += sigma * torch.randn((rows, V), generator=g, device=device)
    return t


def _draft_rows(g, t, spec, row_depth):
    kind = spec[0]
    noise = torch.randn(t.shape, generator=g, device=t.device)
    if kind == "add":
        return t + spec[1] * noise
    if kind == "add_depth":
        s0, step, cap = spec[1], spec[2], spec[3]
        sig = torch.tensor([s0 + step * min(int(d), cap) for d in row_depth],
                           device=t.device, dtype=torch.float32)[:, None]
        return t + sig * noise
    if kind == "corr":
        return spec[1] * t + spec[2] * noise
    raise ValueError(kind)


def _gumbel(g, shape, device):
    u = torch.rand(shape, generator=g, device=device).clamp_(min=1e-20)
    return -torch.log(-torch.log(u))


def _store(x, dtype):
    return x.to(torch.bfloat16) if dtype == "bf16" else x.contiguous()


def make_workload(cfg_id, *, seed=SEED, device="cpu", B=None, V=None, N=None, dtype=None,
                  T=None):
    """Generate one workload.  cfg_id: a key of CONFIGS, or a config dict of the same
    form.  Overrides (B, V, N for random trees, dtype, T) give smaller or ragged
    variants of the same recipe for tests."""
    cfg = dict(CONFIGS[cfg_id]) if not isinstance(cfg_id, dict) else dict(cfg_id)
    if B is not None:
        cfg["B"] = B
    if V is not None:
        cfg["V"] = V
    if dtype is not None:
        cfg["dtype"] = dtype
    if T is not None:
        cfg["T"] = T
    B, V, Tm = cfg["B"], cfg["V"], cfg["T"]
    device = torch.device(device)
    if cfg["kind"] == "flat":
        return _make_flat(cfg, seed, device)

    parents = [tree_for(cfg, b, seed, N) for b in range(B)]
    n_nodes = len(parents[0])
    tl = torch.empty((B, n_nodes, V), dtype=torch.bfloat16 if cfg["dtype"] == "bf16" else torch.float32,
                     device=device)
    dl = torch.empty_like(tl)
    node_token = torch.zeros((B, n_nodes), dtype=torch.int32)
    ua = torch.empty((B, n_nodes), dtype=torch.float32)
    ur = torch.empty((B, n_nodes), dtype=torch.float32)
    max_depth = 0
    for b in range(B):
        par = parents[b]
        dep = depths(par)
        max_depth = max(max_depth, int(dep.max()))
        g = torch.Generator(device=device)
        g.manual_seed(seed + b)
        t = _zipf_rows(g, n_nodes, V, cfg["zipf"], cfg["tgt_sigma"], device)
        d = _draft_rows(g, t, cfg["draft"], dep)
        tl[b] = _store(t, cfg["dtype"])
        dl[b] = _store(d, cfg["dtype"])
        # candidates: children of node n are drawn from the temperature softmax of the
        # draft row n as stored (Gumbel-max; Gumbel-top-k without replacement)
        dstored = dl[b].float() / Tm
        for n in np.unique(par[1:]):
            kids = np.flatnonzero(par == n)
            row = dstored[n]
            if cfg["worep"]:
                top = torch.topk(row + _gumbel(g, (V,), device), len(kids)).indices
            else:
                top = torch.argmax(row[None, :] + _gumbel(g, (len(kids), V), device), dim=1)
            node_token[b, torch.as_tensor(kids)] = top.to(torch.int32).cpu()
        gu = torch.Generator().manual_seed(seed + b)
        ua[b] = torch.rand(n_nodes, generator=gu)
        ur[b] = torch.rand(n_nodes, generator=gu)
    parent = torch.as_tensor(np.stack(parents), dtype=torch.int32)
    return dict(cfg=cfg, kind="tree", target=tl, draft=dl, node_token=node_token.to(device),
                parent=parent.to(device), u_accept=ua.to(device), u_resample=ur.to(device),
                temperature=Tm, without_replacement=cfg["worep"], bonus=True,
                max_depth=max_depth, B=B, N=n_nodes, V=V)


def _make_flat(cfg, seed, device):
    B, V, k, Tm = cfg["B"], cfg["V"], cfg["k"], cfg["T"]
    tl = torch.empty((B, V), dtype=torch.bfloat16 if cfg["dtype"] == "bf16" else torch.float32,
                     device=device)
    dl = torch.empty_like(tl)
    cand = torch.empty((B, k), dtype=torch.int32)
    ua = torch.empty((B, k), dtype=torch.float32)
    ur = torch.empty(B, dtype=torch.float32)
    for b in range(B):
        g = torch.Generator(device=device)
        g.manual_seed(seed + b)
        t = _zipf_rows(g, 1, V, cfg["zipf"], cfg["tgt_sigma"], device)
        d = _draft_rows(g, t, cfg["draft"], [0])
        tl[b] = _store(t, cfg["dtype"])[0]
        dl[b] = _store(d, cfg["dtype"])[0]
        row = dl[b].float() / Tm
        cand[b] = torch.argmax(row[None, :] + _gumbel(g, (k, V), device), dim=1).to(torch.int32).cpu()
        gu = torch.Generator().manual_seed(seed + b)
        ua[b] = torch.rand(k, generator=gu)
        ur[b] = torch.rand(1, generator=gu)[0]
    return dict(cfg=cfg, kind="flat", target=tl, draft=dl, cand_ids=cand.to(device),
                u_accept=ua.to(device), u_resample=ur.to(device), temperature=Tm, B=B, V=V, k=k)


def to_host(x):
    """numpy view for host consumers: float32 as is, bf16 as its uint16 bit patterns."""
    x = x.detach().cpu().contiguous()
    if x.dtype == torch.bfloat16:
        return x.view(torch.int16).numpy().view(np.uint16)
    return x.numpy()


def algorithmic_bytes(parent, V, elem_bytes):
    """Bytes a verification of one tree must read at least once: the target row of
    every node and the draft row of every node with children."""
    par = np.asarray(parent)
    internal = np.zeros(par.shape, dtype=bool)
    for b in range(par.shape[0]):
        internal[b, np.unique(par[b, 1:])] = True
    rows_t = par.size
    rows_d = int(internal.sum())
    return (rows_t + rows_d) * V * elem_bytes, rows_t, rows_d
