"""Seeded synthetic Tree-of-Thoughts KV workloads.

This module only draws inputs: tree shapes, K/V/Q values, heavy tokens, the
controller signals v_i and the raw uncertainty u_i, the active leaves and the
initial (fully retained) paged-pool layout.  It contains none of the method's
arithmetic, so both the HIP path and the CPU oracle can be fed from it.

Shapes follow the paper's problem statement (a rooted tree of thought blocks,
each a contiguous token span, Sec. 3) at the sizes of the synthetic
configurations below.  Every array is drawn from torch generators seeded per
purpose, so the bytes depend only on (config, seed, device).

Layouts (P = page size, d = head_dim, G = query heads per KV head):
  pool K/V      [L][num_pages][Hkv][P][d]   (dtype bf16 or f32)
  slot_pos      [num_pages][P] int32        node-local position, -1 = empty
  page_table    [page_off[V]] int32         physical page of logical page q of node i
  host store    [N][L][Hkv][d]              token-major copy of every token's K/V
  q_win         [n_obs][S][Hq][W][d]        window queries of each observer node
  q_dec         [n_leaves][L][Hq][d]        one decode query per active leaf
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field, replace

import torch

PAGE_SIZE = 16


@dataclass(frozen=True)
class Config:
    name: str
    layers: int
    kv_heads: int
    q_per_kv: int
    head_dim: int
    dtype: str                 # "bf16" | "f32"
    branching: int
    depth: int
    root_tokens: int
    node_tokens: int
    window: int
    heavy_frac: float
    rho: float
    n_active: int
    seed: int
    # method parameters (the paper prints no values; these are the defaults
    # this library proposes, see the parameter struct in include/arbor.h)
    params: dict = field(default_factory=dict)
    walk_backtrack: float = 0.0
    walk_steps: int = 0

    @property
    def q_heads(self) -> int:
        return self.kv_heads * self.q_per_kv

    @property
    def slice_layers(self) -> list[int]:
        if self.layers == 1:
            return [0]
        return [self.layers // 2, self.layers - 1]


DEFAULT_PARAMS = dict(alpha_max=math.inf, gamma=2.0, lambda_d=0.0, lambda_delta=0.5,
                      eta=0.8, r_min=0.05, k_min=4, l_tail=8,
                      theta=(1.0, 1.0, 1.0), select_mode=0, score_self_window=0)
TINY_PARAMS = dict(DEFAULT_PARAMS, k_min=2, l_tail=4, r_min=0.0)

CONFIGS = {
    # 1 layer, 4 KV heads, d=64, fp32; binary tree of depth 2 (7 nodes, root 64,
    # others 32); window 8; 5 % heavy tokens; budget 50 %; one active leaf.
    "tiny": Config("tiny", 1, 4, 1, 64, "f32", 2, 2, 64, 32, 8, 0.05, 0.5, 1, 0,
                   params=TINY_PARAMS),
    # Llama-3-8B-shaped KV: 32 layers, 8 KV heads (32 q heads), d=128, bf16;
    # root 1024, branching 4, depth 3, 256 tokens/node; 4 active leaves; 25 %.
    "llama8b": Config("llama8b", 32, 8, 4, 128, "bf16", 4, 3, 1024, 256, 32, 0.02, 0.25, 4, 1,
                      params=DEFAULT_PARAMS),
    # DPTS-like wide frontier: branching 4, depth 4 (341 nodes), 128 tokens/node,
    # 16 active leaves decoding one token each.
    "dpts": Config("dpts", 32, 8, 4, 128, "bf16", 4, 4, 1024, 128, 32, 0.02, 0.25, 16, 2,
                   params=DEFAULT_PARAMS),
    # Deep backtracking tree: branching 3, depth 8 (9,841 nodes), 64 tokens/node,
    # random walk with 30 % backtracking; budget 20 %.
    "deep": Config("deep", 32, 8, 4, 128, "bf16", 3, 8, 1024, 64, 32, 0.02, 0.20, 1, 3,
                   params=DEFAULT_PARAMS, walk_backtrack=0.3, walk_steps=256),
    # 70B-shaped KV: 80 layers, 8 KV heads (64 q heads); root 4096, branching 4,
    # depth 4, 512 tokens/node; 8 active leaves; 25 %.
    "llama70b": Config("llama70b", 80, 8, 8, 128, "bf16", 4, 4, 4096, 512, 32, 0.02, 0.25, 8, 4,
                       params=DEFAULT_PARAMS),
}


def complete_tree(branching: int, depth: int, root_tokens: int, node_tokens: int):
    """Complete tree in BFS order: children of a node are consecutive ids."""
    sizes = [branching ** lvl for lvl in range(depth + 1)]
    v = sum(sizes)
    parent = [-1] + [(i - 1) // branching for i in range(1, v)]
    n_full = [root_tokens] + [node_tokens] * (v - 1)
    return parent, n_full


def random_tree(num_nodes: int, max_tokens: int, seed: int, min_tokens: int = 1,
                max_children: int | None = None):
    """Random rooted tree with parent[i] < i and ragged token counts."""
    g = torch.Generator().manual_seed(seed)
    parent = [-1]
    kids = [0] * num_nodes
    for i in range(1, num_nodes):
        while True:
            p = int(torch.randint(0, i, (1,), generator=g))
            if max_children is None or kids[p] < max_children:
                break
        kids[p] += 1
        parent.append(p)
    n_full = [int(x) for x in torch.randint(min_tokens, max_tokens + 1, (num_nodes,), generator=g)]
    return parent, n_full


def tree_depths(parent):
    d = [0] * len(parent)
    for i in range(1, len(parent)):
        d[i] = d[parent[i]] + 1
    return d


def deepest_leaves_evenly(parent, n_active: int):
    """Evenly spaced picks (index floor(k*n/n_a)) among the deepest leaves in id order."""
    d = tree_depths(parent)
    has_child = [False] * len(parent)
    for i in range(1, len(parent)):
        has_child[parent[i]] = True
    dmax = max(d)
    leaves = [i for i in range(len(parent)) if d[i] == dmax and not has_child[i]]
    return [leaves[(k * len(leaves)) // n_active] for k in range(n_active)]


def _gen(seed: int, purpose: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed * 7919 + purpose)
    return g


def _torch_dtype(name: str):
    return {"bf16": torch.bfloat16, "f32": torch.float32}[name]


def build_state(parent, n_full, *, layers, kv_heads, q_per_kv, head_dim, dtype="bf16",
                seed=0, device="cpu", page_size=PAGE_SIZE, heavy_frac=0.0, heavy_scale=4.0,
                shuffle_pages=False, spare_pages=0, observers=None, window=8,
                slice_layers=None, active=None, host_store=True, decode_queries=True,
                identical_keys=False):
    """Draw a fully retained tree KV state and the per-event inputs.

    Every node starts with all its tokens resident: slot s of node i holds
    position s.  Physical pages are either assigned in order or shuffled
    (seeded) so that page-table indirection is exercised.
    """
    dev = torch.device(device)
    V = len(parent)
    P = page_size
    n_full_t = torch.tensor(n_full, dtype=torch.int64)
    tok_off = torch.zeros(V + 1, dtype=torch.int64)
    tok_off[1:] = torch.cumsum(n_full_t, 0)
    pages_per = (n_full_t + P - 1) // P
    page_off = torch.zeros(V + 1, dtype=torch.int64)
    page_off[1:] = torch.cumsum(pages_per, 0)
    n_used = int(page_off[-1])
    num_pages = n_used + spare_pages
    N = int(tok_off[-1])

    if shuffle_pages:
        perm = torch.randperm(num_pages, generator=_gen(seed, 1, "cpu")).to(torch.int32)
    else:
        perm = torch.arange(num_pages, dtype=torch.int32)
    page_table = perm[:n_used].clone()
    free_stack = torch.full((num_pages,), -1, dtype=torch.int32)
    free_stack[:spare_pages] = perm[n_used:]
    free_top = torch.tensor([spare_pages], dtype=torch.int32)

    # logical token -> (physical page, slot)
    node_of_tok = torch.repeat_interleave(torch.arange(V), n_full_t)
    pos_of_tok = torch.arange(N, dtype=torch.int64) - tok_off[node_of_tok]
    phys_of_tok = page_table[(page_off[node_of_tok] + pos_of_tok // P)].to(torch.int64)
    slot_of_tok = pos_of_tok % P
    slot_pos = torch.full((num_pages, P), -1, dtype=torch.int32)
    slot_pos[phys_of_tok, slot_of_tok] = pos_of_tok.to(torch.int32)

    # heavy tokens: ceil(f * n_i) positions per node, uniform without replacement
    heavy = torch.zeros(N, dtype=torch.bool)
    if heavy_frac > 0:
        gh = _gen(seed, 2, "cpu")
        for i in range(V):
            m = math.ceil(heavy_frac * n_full[i])
            if m:
                idx = torch.randperm(n_full[i], generator=gh)[:m]
                heavy[int(tok_off[i]) + idx] = True

    L, Hkv, d = layers, kv_heads, head_dim
    Hq = Hkv * q_per_kv
    tdt = _torch_dtype(dtype)
    shape = (L, num_pages, Hkv, P, d)
    if identical_keys:
        k = torch.randn((L, 1, Hkv, 1, d), generator=_gen(seed, 3, dev), device=dev).expand(shape).clone()
    else:
        k = torch.randn(shape, generator=_gen(seed, 3, dev), device=dev)
    v = torch.randn(shape, generator=_gen(seed, 4, dev), device=dev)
    valid = torch.zeros((num_pages, P), dtype=torch.bool)
    valid[phys_of_tok, slot_of_tok] = True
    scale = torch.ones((num_pages, P), dtype=torch.float32)
    scale[phys_of_tok[heavy], slot_of_tok[heavy]] = heavy_scale
    scale = torch.where(valid, scale, torch.zeros_like(scale)).to(dev)
    k.mul_(scale.view(1, num_pages, 1, P, 1))
    v.mul_(valid.to(dev, torch.float32).view(1, num_pages, 1, P, 1))
    k = k.to(tdt)
    v = v.to(tdt)

    st = dict(parent=torch.tensor(parent, dtype=torch.int32), n_full=n_full_t.to(torch.int32),
              tok_off=tok_off, page_off=page_off, n_kept=n_full_t.to(torch.int32).clone(),
              page_table=page_table, slot_pos=slot_pos, free_stack=free_stack, free_top=free_top,
              k=k, v=v, heavy=heavy, num_pages=num_pages, page_size=P, layers=L, kv_heads=Hkv,
              q_per_kv=q_per_kv, head_dim=d, dtype=dtype, num_tokens=N)

    if host_store:
        pt = phys_of_tok.to(dev)
        sl = slot_of_tok.to(dev)
        # [L][N][Hkv][d] -> [N][L][Hkv][d]
        hk = k.permute(1, 3, 0, 2, 4)[pt, sl]
        hv = v.permute(1, 3, 0, 2, 4)[pt, sl]
        if host_store == "device":
            # the same token-major record kept in device memory (very large pools)
            st["host_k"] = hk.contiguous()
            st["host_v"] = hv.contiguous()
        elif dev.type == "cuda":
            st["host_k"] = torch.empty(hk.shape, dtype=tdt, pin_memory=True)
            st["host_v"] = torch.empty(hv.shape, dtype=tdt, pin_memory=True)
            st["host_k"].copy_(hk)
            st["host_v"].copy_(hv)
        else:
            st["host_k"] = hk.contiguous()
            st["host_v"] = hv.contiguous()
        del hk, hv

    if slice_layers is None:
        slice_layers = [0] if L == 1 else [L // 2, L - 1]
    st["slice_layers"] = list(slice_layers)
    if observers is None:
        observers = list(range(V))
    st["observers"] = torch.tensor(observers, dtype=torch.int32)
    st["window"] = window
    st["q_win"] = torch.randn((len(observers), len(slice_layers), Hq, window, d),
                              generator=_gen(seed, 5, dev), device=dev).to(tdt)
    gs = _gen(seed, 6, "cpu")
    st["v_sig"] = torch.rand(V, generator=gs)
    st["u_sig"] = torch.rand(V, generator=gs)
    if active is None:
        active = deepest_leaves_evenly(parent, 1)
    st["active"] = torch.tensor(active, dtype=torch.int32)
    if decode_queries:
        st["q_dec"] = torch.randn((len(active), L, Hq, d), generator=_gen(seed, 7, dev),
                                  device=dev).to(tdt)
    st["A"] = torch.zeros(N, dtype=torch.float32)
    st["rows_seen"] = torch.zeros(V, dtype=torch.int64)
    return st


def build_config(cfg: Config | str, device="cpu", **overrides):
    """Draw the workload of one named synthetic configuration."""
    if isinstance(cfg, str):
        cfg = CONFIGS[cfg]
    parent, n_full = complete_tree(cfg.branching, cfg.depth, cfg.root_tokens, cfg.node_tokens)
    active = deepest_leaves_evenly(parent, cfg.n_active)
    kw = dict(layers=cfg.layers, kv_heads=cfg.kv_heads, q_per_kv=cfg.q_per_kv,
              head_dim=cfg.head_dim, dtype=cfg.dtype, seed=cfg.seed, device=device,
              heavy_frac=cfg.heavy_frac, window=cfg.window, slice_layers=cfg.slice_layers,
              active=active)
    kw.update(overrides)
    st = build_state(parent, n_full, **kw)
    st["config"] = cfg
    st["budget"] = int(math.floor(cfg.rho * st["num_tokens"]))
    st["params"] = dict(cfg.params)
    return st


def boundary_logits(n_rows: int, vocab: int, seed: int, dtype="bf16", device="cpu"):
    """Seeded next-token logit rows standing in for a model's output at block
    boundaries: rows cycle through flat (std 0.5), spread (std 2), peaked (std 2
    with one token raised by 12) and coarsely quantised rows (std 2 rounded to
    multiples of 0.5, so many logits tie, also at any top-K boundary)."""
    g = _gen(seed, 17, "cpu")
    z = torch.randn(n_rows, vocab, generator=g, dtype=torch.float32)
    for r in range(n_rows):
        kind = r % 4
        if kind == 0:
            z[r] *= 0.5
        else:
            z[r] *= 2.0
        if kind == 2:
            z[r, int(torch.randint(vocab, (1,), generator=g))] += 12.0
        if kind == 3:
            z[r] = torch.round(z[r] * 2.0) / 2.0
    return z.to(_torch_dtype(dtype)).to(device)


def walk_targets(parent, steps: int, p_backtrack: float, seed: int, start: int):
    """Random walk over the tree: with probability p backtrack to a uniform proper
    ancestor and step into one of its children off the current path, otherwise
    descend into a uniform child; at a leaf always backtrack."""
    g = torch.Generator().manual_seed(seed * 7919 + 11)
    V = len(parent)
    children = [[] for _ in range(V)]
    for i in range(1, V):
        children[parent[i]].append(i)
    cur = start
    out = []
    for _ in range(steps):
        chain = []
        a = cur
        while a >= 0:
            chain.append(a)
            a = parent[a]
        r = float(torch.rand(1, generator=g))
        if children[cur] and r >= p_backtrack:
            cur = children[cur][int(torch.randint(0, len(children[cur]), (1,), generator=g))]
        else:
            anc = chain[1:]
            if not anc:
                continue
            a = anc[int(torch.randint(0, len(anc), (1,), generator=g))]
            opts = [c for c in children[a] if c not in chain]
            if not opts:
                continue
            cur = opts[int(torch.randint(0, len(opts), (1,), generator=g))]
        out.append(cur)
    return out
