"""Plain CPU oracle of the ArborKV eviction hot path (arxiv 2605.22106).

TEST INFRASTRUCTURE ONLY.  This module is the slow, obviously correct
reference that the HIP library is checked against.  Only the test suite, the
package smoke check and the benchmark's CPU-baseline leg may import it; the
product path never does.  It shares no code with the HIP library: it imports
numpy and the Python standard library and nothing else.

Arithmetic is fp64 throughout (bf16/fp32 inputs are widened exactly) and is
rounded to fp32 only where an output is fp32.  Every function cites the part
of the paper it follows:

  geometry          Sec. 3 (tree, depth d_i, distance Delta_i, Path*) and the
                    RootToLeaf / TreeDistance steps of Alg. 2
  score             Sec. 4 MSVE (accumulated attention A_i(t), block attention
                    a_i, s_i = clip(sigmoid(theta^T phi_i), 0, 1)); Alg. 1 MSVE
  uncertainty       Eq. 1 (normalised next-token entropy, optional top-K bucket)
  allocate          Eq. 2 and Eq. 3 (TAE ratio and keep-count), the KKT view
                    of Sec. 4 (alpha chosen so the budget is met), and the
                    Transition / Pressure branches of Alg. 2
  select            Sec. 4 Execution (tail set T_i + heavy hitters H_i, tail
                    first on overlap); Alg. 1 Evict
  compact           Sec. 4 Execution (token-extractive eviction frees KV
                    entries of the non-retained tokens), on a paged pool
  rehydrate         Sec. 4 lazy rehydration; Alg. 2 Transition branch
  tree_decode_attn  Sec. 1/3 (decoding depends only on the active leaf's
                    ancestor chain): softmax attention over the retained keys
                    of the chain
  decode_credit     Sec. 4 Execution (iii): A_i(t) grown from the attention
                    weights of the decoding step itself (thin slice of layers,
                    all heads), credited to proper ancestors of the query's leaf
  walk              Alg. 2 (event-driven controller): Transition events to a
                    sequence of active leaves with lazy rehydration, and the
                    Pressure event raised at B - delta

Readings of points the paper leaves open are listed next to the code that
takes them.  Parity status: every function here is pinned by the tests in
tests/test_oracle_*.py against closed forms, invariants, brute force or a
textbook routine; the paper prints no worked numeric example, so no value is
pinned to a printed number (the numeric values of the method are "parity
unpinned" with respect to the paper's own text).

State dictionary (numpy arrays), the paged tree KV pool:
  parent[V] int, n_full[V] int, tok_off[V+1], page_off[V+1], n_kept[V],
  page_table[page_off[V]] (physical page id, -1 = unused), slot_pos[pages][P]
  (node-local position held by a slot, -1 = empty), free_stack[pages] with
  free_top (entries [0, free_top) are free pages, the top is free_top-1),
  k, v [L][pages][Hkv][P][d] (any float dtype), page_size.
"""
from __future__ import annotations

import math

import numpy as np

OK = 0
OVER_BUDGET = 1
EINVAL = -1
ENOPAGES = -2
ENONFINITE = -5

TAIL_HEAVY = 0
TAIL_ONLY = 1
SINKS_TAIL = 2


# ----------------------------------------------------------------------------
# tree helpers
# ----------------------------------------------------------------------------
def chain(parent, i):
    """Nodes from the root down to i (inclusive)."""
    out = []
    while i >= 0:
        out.append(int(i))
        i = int(parent[i])
    return out[::-1]


def depths(parent):
    d = np.zeros(len(parent), dtype=np.int64)
    for i in range(len(parent)):
        d[i] = len(chain(parent, i)) - 1
    return d


def retained(st, i):
    """Retained tokens of node i in slot order: list of (slot, page, r, position)."""
    P = st["page_size"]
    out = []
    for s in range(int(st["n_kept"][i])):
        page = int(st["page_table"][int(st["page_off"][i]) + s // P])
        r = s % P
        out.append((s, page, r, int(st["slot_pos"][page, r])))
    return out


# ----------------------------------------------------------------------------
# O1  geometry  (Sec. 3; Alg. 2 RootToLeaf, TreeDistance)
# ----------------------------------------------------------------------------
def geometry(parent, active):
    """Path* is the union of the root-to-leaf chains of the active leaves (one
    leaf in the paper; a DPTS frontier has several).  Delta_i is the tree
    distance to the nearest active leaf: d_i + d_l - 2 d_lca(i, l)."""
    V = len(parent)
    d = depths(parent)
    on_path = np.zeros(V, dtype=np.uint8)
    chains = [chain(parent, int(l)) for l in active]
    for c in chains:
        for a in c:
            on_path[a] = 1
    delta = np.zeros(V, dtype=np.int64)
    for i in range(V):
        ci = chain(parent, i)
        best = None
        for cl in chains:
            common = 0
            while common < min(len(ci), len(cl)) and ci[common] == cl[common]:
                common += 1
            lca = ci[common - 1]
            dist = d[i] + d[cl[-1]] - 2 * d[lca]
            best = dist if best is None else min(best, dist)
        delta[i] = best
    return d, on_path, delta


# ----------------------------------------------------------------------------
# Eq. 1 uncertainty helper
# ----------------------------------------------------------------------------
def uncertainty(logits, top_k=None):
    """u = 1 - H / log|V| of the next-token softmax (Eq. 1).  With top_k the sum
    runs over the top-K probabilities plus one "other" outcome carrying the
    remaining mass."""
    z = np.asarray(logits, dtype=np.float64)
    p = np.exp(z - z.max())
    p /= p.sum()
    if top_k is not None and top_k < len(p):
        top = np.sort(p)[::-1][:top_k]
        other = max(0.0, 1.0 - top.sum())
        terms = list(top) + ([other] if other > 0 else [])
    else:
        terms = list(p)
    H = -sum(x * math.log(x) for x in terms if x > 0)
    return 1.0 - H / math.log(len(p))


# ----------------------------------------------------------------------------
# O2  score  (Sec. 4 MSVE; A_i(t); Alg. 1 MSVE)
# ----------------------------------------------------------------------------
def score(st, observers, q_win, window, slice_layers, q_per_kv, v_sig, u_sig, A, rows_seen,
          theta=(1.0, 1.0, 1.0), softmax_scale=None, self_window=0):
    """Accumulated attention of every observer's last-W window queries.

    For observer j, slice layer l and query head h, window query u (the last
    w_j = min(W, n_j) positions of j) attends with a softmax over its causal
    context: every retained token of j's proper ancestors, and j's own
    retained tokens at positions <= u.  The softmax probability of each token
    of a proper ancestor of j is added to A at that token (the paper sums over
    later positions u > b_i, layers of a thin slice and heads).  With
    self_window=1 the observer's own earlier tokens (p < u) are credited too.
    rows_seen_i counts the query rows that credited block i; the block
    attention is a_i = sum_p A_i(p) / rows_seen_i (0 if never observed), and
    s_i = clip(sigmoid(theta_v v_i + theta_u u_i + theta_a a_i), 0, 1).
    Returns (A_out fp32, rows_seen_out, a fp32, s fp32).
    """
    parent = st["parent"]
    n_full = st["n_full"]
    tok_off = st["tok_off"]
    K = st["k"]
    L, _, Hkv, P, dh = K.shape
    G = int(q_per_kv)
    Hq = Hkv * G
    if softmax_scale is None:
        softmax_scale = 1.0 / math.sqrt(dh)
    N = int(tok_off[-1])
    V = len(parent)
    contrib = np.zeros(N, dtype=np.float64)
    rows_seen = np.asarray(rows_seen, dtype=np.int64).copy()
    for o, j in enumerate(observers):
        j = int(j)
        ch = chain(parent, j)
        ctx = []  # (node, position, page, r)
        for a in ch:
            for (_, page, r, pos) in retained(st, a):
                ctx.append((a, pos, page, r))
        nj = int(n_full[j])
        wj = min(int(window), nj)
        if not ctx or wj == 0:
            for a in ch[:-1]:
                rows_seen[a] += len(slice_layers) * Hq * wj
            if self_window:
                rows_seen[j] += len(slice_layers) * Hq * wj
            continue
        node = np.array([c[0] for c in ctx])
        pos = np.array([c[1] for c in ctx])
        pages = np.array([c[2] for c in ctx])
        rs = np.array([c[3] for c in ctx])
        tok = tok_off[node] + pos
        u = nj - wj + np.arange(wj)                    # window positions
        allowed = (node[None, :] != j) | (pos[None, :] <= u[:, None])     # [wj, C]
        if self_window:
            credited = (node[None, :] != j) | (pos[None, :] < u[:, None])
        else:
            credited = np.broadcast_to(node[None, :] != j, allowed.shape)
        for si, l in enumerate(slice_layers):
            for h in range(Hq):
                g = h // G
                Kc = K[l, pages, g, rs, :].astype(np.float64)            # [C, d]
                q = q_win[o, si, h, :wj, :].astype(np.float64)            # [wj, d]
                z = softmax_scale * (q @ Kc.T)                            # [wj, C]
                z = np.where(allowed, z, -np.inf)
                for t in range(wj):
                    if not allowed[t].any():
                        continue
                    zt = z[t]
                    e = np.exp(zt - zt.max())
                    p = e / e.sum()
                    np.add.at(contrib, tok[credited[t]], p[credited[t]])
        for a in ch[:-1]:
            rows_seen[a] += len(slice_layers) * Hq * wj
        if self_window:
            rows_seen[j] += len(slice_layers) * Hq * wj
    A_out = (np.asarray(A, dtype=np.float64) + contrib).astype(np.float32)
    a = np.zeros(V, dtype=np.float64)
    for i in range(V):
        if rows_seen[i] > 0:
            seg = A_out[int(tok_off[i]):int(tok_off[i + 1])].astype(np.float64)
            a[i] = seg.sum() / float(rows_seen[i])
    th = [float(x) for x in theta]
    s = np.zeros(V, dtype=np.float64)
    for i in range(V):
        x = th[0] * float(v_sig[i]) + th[1] * float(u_sig[i]) + th[2] * a[i]
        s[i] = min(1.0, max(0.0, 1.0 / (1.0 + math.exp(-x))))
    return A_out, rows_seen, a.astype(np.float32), s.astype(np.float32)


# ----------------------------------------------------------------------------
# O3  allocate  (Eq. 2, Eq. 3, KKT view; Alg. 2 Transition / Pressure)
# ----------------------------------------------------------------------------
def power(s, gamma):
    """s^gamma of Eq. 2.  For an integer exponent up to 4 the plain product:
    s is an fp32 value, so s * s is exact in fp64 and one more product rounds
    once, which is the correctly rounded power; other exponents use math.pow."""
    s = float(s)
    if gamma in (1.0, 2.0, 3.0, 4.0):
        g = int(gamma)
        return s if g == 1 else (s * s if g == 2 else (s * s * s if g == 3 else (s * s) * (s * s)))
    return math.pow(s, gamma)


def value_geometry_weight(s, d, delta, p, on_path=False):
    """w_i = eta^[i not in Path*] * s_i^gamma * exp(-lambda_d d_i) * exp(-lambda_Delta Delta_i):
    the weight of Eq. 2 without alpha (the KKT weight).  The off-path discount
    eta applies to every block outside Path*; a Path* block only reaches Eq. 2
    under floor protection.  -0 is returned as +0 (s = -0 with an odd gamma),
    the same weight as s = +0."""
    eta = 1.0 if on_path else p["eta"]
    w = (eta * power(s, p["gamma"])) * math.exp(-p["lambda_d"] * float(d)) \
        * math.exp(-p["lambda_delta"] * float(delta))
    return 0.0 if w == 0.0 else w


def floor_count(n, c, p):
    """The keep-count of Eq. 3 at r_i = r_min, capped at the resident count c:
    min(c, min(n, max(K_min, |T_i|, floor(r_min n)))) with |T_i| = min(L_tail, n)."""
    f = max(int(p["k_min"]), min(int(p["l_tail"]), int(n)), int(math.floor(p["r_min"] * n)))
    return min(int(c), min(int(n), f))


def allocate(parent, n_full, n_kept, active, budget, s, p):
    """Keep-counts k_i under the global token budget B.

    Invariant (i), active-path protection, comes in two forms.  Full
    protection (p["k_protect"] = 0, the default) pins every Path* node at
    k_i = n_i, or at its resident count c_i when p["lazy_rehydration"] is 0
    (evicted tokens are never restored: the "w/o lazy rehydration" setting of
    Table 4).  Floor protection (k_protect > 0) lets Path* nodes take part in
    Eq. 2 and Eq. 3 like every other node, without the off-path discount eta,
    with a floor of k_protect tokens, up to n_i (up to c_i without
    rehydration).

    Every node that is not pinned gets r_i(alpha) = clip(alpha w_i, r_min, 1)
    from Eq. 2 and k_i(alpha) from Eq. 3; a node off the path never re-grows
    beyond its resident count c_i (Alg. 2 only lowers k off the path).  alpha
    is the one global scale of the KKT view, chosen as the largest alpha
    (<= alpha_max) whose total fits B.  Eq. 3 keeps the j-th token of block i
    exactly when floor(alpha w_i n_i) >= j, i.e. when alpha >= j / (w_i n_i):
    that quotient is the price of token j.  Equal prices enter together,
    because alpha is a single scalar.  If even the floors do not fit
    (Pressure), nodes off the path are lowered towards min(K_min, c_i) in
    ascending priority w_i (ties: lower id) until the total fits; if it still
    does not, the status is OVER_BUDGET.  Path* nodes keep their floors.
    Returns (k, delta, on_path, status).
    """
    V = len(parent)
    d, on_path, delta = geometry(parent, active)
    k = np.zeros(V, dtype=np.int64)
    rehyd = int(p.get("lazy_rehydration", 1)) != 0
    k_protect = int(p.get("k_protect", 0))
    pinned = [i for i in range(V) if on_path[i] and k_protect == 0]
    free = [i for i in range(V) if not (on_path[i] and k_protect == 0)]
    path_total = 0
    for i in pinned:
        k[i] = int(n_full[i]) if rehyd else int(n_kept[i])
        path_total += int(k[i])
    b_off = int(budget) - path_total
    # s_i = clip(sigmoid(theta^T phi_i), 0, 1) (Sec. 4 MSVE) lies in [0, 1]
    s_free = [float(s[i]) for i in free]
    if any(math.isnan(x) for x in s_free):
        return k.astype(np.int32), delta.astype(np.int32), on_path, ENONFINITE
    if any(not (0.0 <= x <= 1.0) for x in s_free):
        return k.astype(np.int32), delta.astype(np.int32), on_path, EINVAL
    # upper end of each node's count: resident tokens, or the whole span for
    # a Path* node that rehydration restores
    cap = {i: int(n_full[i]) if (on_path[i] and rehyd) else int(n_kept[i]) for i in free}
    F = {}
    for i in free:
        f = floor_count(n_full[i], cap[i], p)
        if on_path[i]:
            f = max(f, min(cap[i], k_protect))
        F[i] = f
    w = {i: value_geometry_weight(s[i], d[i], delta[i], p, bool(on_path[i])) for i in free}
    status = OK
    if sum(F.values()) <= b_off:
        extra = b_off - sum(F.values())
        prices = []
        for i in free:
            W = w[i] * float(n_full[i])
            for j in range(F[i] + 1, cap[i] + 1):
                price = float(j) / W if W > 0 else math.inf
                if math.isfinite(price) and price <= p["alpha_max"]:
                    prices.append((price, i))
        prices.sort(key=lambda t: t[0])
        if len(prices) <= extra:
            kept = prices
        else:
            cut = prices[extra][0]        # the first price that no longer fits
            kept = [t for t in prices if t[0] < cut]
        for i in free:
            k[i] = F[i]
        for (_, i) in kept:
            k[i] += 1
    else:
        for i in free:
            k[i] = F[i]
        excess = sum(F.values()) - b_off
        off = [i for i in free if not on_path[i]]
        for i in sorted(off, key=lambda i: (w[i], i)):
            if excess <= 0:
                break
            lo = min(int(p["k_min"]), int(n_kept[i]))
            red = min(int(k[i]) - lo, excess)
            if red > 0:
                k[i] -= red
                excess -= red
        if excess > 0:
            status = OVER_BUDGET
    return k.astype(np.int32), delta.astype(np.int32), on_path, status


# ----------------------------------------------------------------------------
# O4  select  (Sec. 4 Execution; Alg. 1 Evict)
# ----------------------------------------------------------------------------
def select(st, A, k, l_tail, select_mode=TAIL_HEAVY, n_sinks=0):
    """Retained set R'_i for every node whose count drops (k_i < c_i).

    The mandatory tail is the retained tokens among the last L_tail positions
    of the block.  If k_i does not exceed the tail (or in tail-only mode) the
    k_i most recent retained tokens are kept; otherwise the tail plus the
    m_i = k_i - |tail| non-tail tokens with the largest accumulated attention
    A_i(t), ties to the lower position.  Selection is nested: it picks from the
    current resident set only.

    Global sinks S (Sec. 4 Execution (i)) are the first n_sinks positions of
    the initial prompt, the root block 0.  When the root is cut, its resident
    sinks are kept before anything else (the k_i lowest of them if k_i is
    smaller), then the tail, then heavy hitters, all within k_i.  Modes, after
    Table 7: TAIL_HEAVY (sinks + tail + heavy hitters), TAIL_ONLY (the most
    recent k_i, no sinks), SINKS_TAIL (sinks, then the most recent of the
    rest).  Returns ({node: sorted positions}, status).
    """
    out = {}
    for i in range(len(st["parent"])):
        c = int(st["n_kept"][i])
        ki = int(k[i])
        if ki >= c:
            continue
        n = int(st["n_full"][i])
        R = [r[3] for r in retained(st, i)]
        base = int(st["tok_off"][i])
        vals = [float(np.float32(A[base + p_])) for p_ in R]
        if any(math.isnan(x) for x in vals):
            return {}, ENONFINITE
        n_s = int(n_sinks) if (i == 0 and select_mode != TAIL_ONLY) else 0
        sinks = [p_ for p_ in R if p_ < n_s]
        rest = [p_ for p_ in R if p_ >= n_s]
        if ki <= len(sinks):
            keep = sinks[:ki]
        elif select_mode in (TAIL_ONLY, SINKS_TAIL):
            m = ki - len(sinks)
            keep = sinks + rest[len(rest) - m:]
        else:
            m = ki - len(sinks)
            tail = [p_ for p_ in rest if p_ >= n - int(l_tail)]
            if m <= len(tail):
                keep = sinks + tail[len(tail) - m:]
            else:
                h = m - len(tail)
                cand = [p_ for p_ in rest if p_ < n - int(l_tail)]
                cand.sort(key=lambda p_: (-float(np.float32(A[base + p_])) + 0.0, p_))
                keep = sorted(sinks + cand[:h] + tail)
        out[i] = keep
    return out, OK


def selection_to_csr(sel, tok_off, N, fill=-1):
    arr = np.full(N, fill, dtype=np.int32)
    for i, keep in sel.items():
        b = int(tok_off[i])
        arr[b:b + len(keep)] = keep
    return arr


# ----------------------------------------------------------------------------
# O5  compact  (Sec. 4 Execution: keep R'_i, free the rest)
# ----------------------------------------------------------------------------
def copy_state(st):
    out = {}
    for key, val in st.items():
        out[key] = val.copy() if isinstance(val, np.ndarray) else val
    return out


def compact(st, k, sel):
    """Order-preserving in-place compaction of every changed node.

    Slot s of node i afterwards holds position R'_i[s]; its K/V rows (every
    layer and KV head) are copied bitwise from the slot that held that
    position.  The node keeps its first ceil(k_i/P) page-table entries; the
    pages it no longer needs are pushed on the free stack in (node, page)
    order; vacated slots and released pages get slot_pos = -1; unused
    page-table entries become -1; c_i = k_i.
    """
    P = st["page_size"]
    new = copy_state(st)
    top = int(st["free_top"])
    for i in range(len(st["parent"])):
        c = int(st["n_kept"][i])
        ki = int(k[i])
        if ki >= c:
            continue
        keep = sel[i]
        old = retained(st, i)
        slot_of = {pos: (page, r) for (_, page, r, pos) in old}
        po = int(st["page_off"][i])
        for s, pos in enumerate(keep):
            sp, sr = slot_of[pos]
            dp = int(st["page_table"][po + s // P])
            dr = s % P
            new["k"][:, dp, :, dr, :] = st["k"][:, sp, :, sr, :]
            new["v"][:, dp, :, dr, :] = st["v"][:, sp, :, sr, :]
            new["slot_pos"][dp, dr] = pos
        keep_pages = -(-ki // P)
        for s in range(ki, keep_pages * P):
            new["slot_pos"][int(st["page_table"][po + s // P]), s % P] = -1
        for q in range(keep_pages, -(-c // P)):
            page = int(st["page_table"][po + q])
            new["free_stack"][top] = page
            top += 1
            new["slot_pos"][page, :] = -1
            new["page_table"][po + q] = -1
        new["n_kept"][i] = ki
    new["free_top"] = np.int64(top)
    return new


# ----------------------------------------------------------------------------
# O6  rehydrate  (Sec. 4 lazy rehydration; Alg. 2 Transition)
# ----------------------------------------------------------------------------
def rehydrate(st, on_path, host_k, host_v):
    """Restore every Path* node with c_i < n_i to full retention, root first.

    The token span is never discarded; here its K/V record lives in a host
    store [N][L][Hkv][d], so restoring gives exactly the full-retention state.
    Pages come off the top of the free stack in (node, page) order; afterwards
    slot p holds position p.  Retained rows move bitwise; evicted rows are
    copied bitwise from the store.  Too few free pages: ENOPAGES and nothing
    changes.  Returns (state, status).
    """
    P = st["page_size"]
    todo = [i for i in range(len(st["parent"]))
            if on_path[i] and int(st["n_kept"][i]) < int(st["n_full"][i])]
    need = sum(-(-int(st["n_full"][i]) // P) - (-(-int(st["n_kept"][i]) // P)) for i in todo)
    if need > int(st["free_top"]):
        return copy_state(st), ENOPAGES
    new = copy_state(st)
    top = int(st["free_top"])
    for i in todo:
        n = int(st["n_full"][i])
        c = int(st["n_kept"][i])
        po = int(st["page_off"][i])
        old = retained(st, i)
        slot_of = {pos: (page, r) for (_, page, r, pos) in old}
        for q in range(-(-c // P), -(-n // P)):
            top -= 1
            new["page_table"][po + q] = int(st["free_stack"][top])
        base = int(st["tok_off"][i])
        for pos in range(n):
            dp = int(new["page_table"][po + pos // P])
            dr = pos % P
            if pos in slot_of:
                sp, sr = slot_of[pos]
                new["k"][:, dp, :, dr, :] = st["k"][:, sp, :, sr, :]
                new["v"][:, dp, :, dr, :] = st["v"][:, sp, :, sr, :]
            else:
                new["k"][:, dp, :, dr, :] = host_k[base + pos]
                new["v"][:, dp, :, dr, :] = host_v[base + pos]
            new["slot_pos"][dp, dr] = pos
        last = int(new["page_table"][po + (n - 1) // P])
        for r in range(n - ((n - 1) // P) * P, P):
            new["slot_pos"][last, r] = -1
        new["n_kept"][i] = n
    new["free_top"] = np.int64(top)
    return new, OK


# ----------------------------------------------------------------------------
# O7  tree decode attention  (Sec. 1/3: the next step depends on the chain)
# ----------------------------------------------------------------------------
def tree_decode_attn(st, leaves, layer_begin, layer_end, q, q_per_kv, softmax_scale=None):
    """o = softmax(scale q K^T) V over every retained key of the leaf's
    root-to-leaf chain, per leaf, layer in [layer_begin, layer_end) and query
    head (head h reads KV head h // G).  fp64; returns (o, lse) with
    lse = max z + ln sum exp(z - max z)."""
    K = st["k"]
    Vv = st["v"]
    L, _, Hkv, P, dh = K.shape
    G = int(q_per_kv)
    Hq = Hkv * G
    if softmax_scale is None:
        softmax_scale = 1.0 / math.sqrt(dh)
    Lr = layer_end - layer_begin
    o = np.zeros((len(leaves), Lr, Hq, dh), dtype=np.float64)
    lse = np.full((len(leaves), Lr, Hq), -np.inf, dtype=np.float64)
    for li, leaf in enumerate(leaves):
        pages, rs = [], []
        for a in chain(st["parent"], int(leaf)):
            for (_, page, r, _) in retained(st, a):
                pages.append(page)
                rs.append(r)
        if not pages:
            continue
        pages = np.array(pages)
        rs = np.array(rs)
        for lr in range(Lr):
            l = layer_begin + lr
            for h in range(Hq):
                g = h // G
                Kc = K[l, pages, g, rs, :].astype(np.float64)
                Vc = Vv[l, pages, g, rs, :].astype(np.float64)
                z = softmax_scale * (Kc @ q[li, lr, h].astype(np.float64))
                m = z.max()
                e = np.exp(z - m)
                o[li, lr, h] = (e @ Vc) / e.sum()
                lse[li, lr, h] = m + math.log(e.sum())
    return o, lse


# ----------------------------------------------------------------------------
# O8  decode-time credit of accumulated attention  (Sec. 4 Execution (iii))
# ----------------------------------------------------------------------------
def decode_credit(st, leaves, layer_begin, q, q_per_kv, slice_layers, A, rows_seen,
                  self_window=0, softmax_scale=None):
    """A_i(t) grown from the weights a decoding step already computes.

    The query of leaf l (one per layer of the call and query head, q laid out
    [leaf][layer - layer_begin][head][d]) sits at the leaf's newest position,
    after the end b_i of every proper ancestor i, so each of its attention
    weights on a token of a proper ancestor is a term of A_i(t) (the sum over
    u > b_i, over the slice layers and all heads).  The weights are the
    decode softmax over the whole retained chain, the leaf's own tokens
    included.  rows_seen_i grows by one per (leaf below i, slice layer, head).
    With self_window = 1 the leaf's own tokens before its newest position
    (p < n_l - 1) are credited too and the leaf counts its own rows.
    Returns (A_out fp32, rows_seen_out).
    """
    K = st["k"]
    L, _, Hkv, P, dh = K.shape
    G = int(q_per_kv)
    Hq = Hkv * G
    if softmax_scale is None:
        softmax_scale = 1.0 / math.sqrt(dh)
    contrib = np.zeros(len(A), dtype=np.float64)
    rows_seen = np.asarray(rows_seen, dtype=np.int64).copy()
    for li, leaf in enumerate(leaves):
        leaf = int(leaf)
        ch = chain(st["parent"], leaf)
        n_leaf = int(st["n_full"][leaf])
        toks, pages, rs, credit = [], [], [], []
        for a in ch:
            for (_, page, r, pos) in retained(st, a):
                toks.append(int(st["tok_off"][a]) + pos)
                pages.append(page)
                rs.append(r)
                credit.append(a != leaf or (self_window and pos < n_leaf - 1))
        for a in ch[:-1]:
            rows_seen[a] += len(slice_layers) * Hq
        if self_window:
            rows_seen[leaf] += len(slice_layers) * Hq
        if not toks:
            continue
        toks = np.array(toks)
        pages = np.array(pages)
        rs = np.array(rs)
        credit = np.array(credit, dtype=bool)
        for l in slice_layers:
            for h in range(Hq):
                g = h // G
                Kc = K[l, pages, g, rs, :].astype(np.float64)
                z = softmax_scale * (Kc @ q[li, l - layer_begin, h].astype(np.float64))
                e = np.exp(z - z.max())
                p = e / e.sum()
                np.add.at(contrib, toks[credit], p[credit])
    A_out = (np.asarray(A, dtype=np.float64) + contrib).astype(np.float32)
    return A_out, rows_seen


# ----------------------------------------------------------------------------
# O9  event-driven controller over a walk  (Alg. 2: Transition, Pressure)
# ----------------------------------------------------------------------------
def walk(st, targets, budget, s, A, rows_seen, p, host_k, host_v, pressure_margin=0,
         q_win=None, window=0, slice_layers=(), q_per_kv=1, v_sig=None, u_sig=None):
    """Alg. 2 for a sequence of Transition events, one per entry of targets.

    Each event: RootToLeaf and the keep-counts of every block for the new
    active leaf (allocate: Path* pinned or floored, every other block lowered
    only where its count drops); Path* blocks with evicted tokens are
    restored from the token-span record before the leaf is attended (lazy
    rehydration); the new leaf's window queries q_win[e] attend over its chain
    and grow A, rows_seen and s (score with that one observer; the reading
    taken here: the window stands in for the decoding at the new leaf, which
    follows the rehydration); the blocks whose count drops are evicted
    (select + compact).  Then, if the resident tokens M reach B - delta
    (RaisePressureEvent, delta = pressure_margin > 0), a Pressure event
    recomputes the counts for the budget B - delta and evicts again.
    Returns (state, A, rows_seen, s, stats, status) where stats has one row
    per event: [resident tokens after it, tokens restored from the record,
    tokens evicted, 1 if Pressure fired].  A negative status stops the walk.
    """
    rehyd = int(p.get("lazy_rehydration", 1)) != 0
    mode = int(p.get("select_mode", TAIL_HEAVY))
    n_sinks = int(p.get("n_sinks", 0))
    A = np.asarray(A, np.float32).copy()
    rows_seen = np.asarray(rows_seen, np.int64).copy()
    s = np.asarray(s, np.float32).copy()
    status = OK
    stats = []

    def note(code):
        nonlocal status
        if code < 0:
            status = code
        elif code > 0 and status == OK:
            status = code

    for e, leaf in enumerate(targets):
        n_full = st["n_full"]
        c = st["n_kept"]
        k, _, on_path, code = allocate(st["parent"], n_full, c, [int(leaf)], budget, s, p)
        note(code)
        if status < 0:
            break
        restored = sum(int(n_full[i]) - int(c[i]) for i in range(len(c))
                       if rehyd and on_path[i] and c[i] < n_full[i])
        row = [int(np.sum(k)), restored, int(np.sum(np.maximum(0, c - k))), 0]
        if rehyd:
            st, code = rehydrate(st, on_path, host_k, host_v)
            note(code)
            if status < 0:
                break
        if q_win is not None:
            A, rows_seen, _, s = score(st, [int(leaf)], q_win[e:e + 1], window, list(slice_layers),
                                       q_per_kv, v_sig, u_sig, A, rows_seen,
                                       theta=p.get("theta", (1.0, 1.0, 1.0)),
                                       self_window=int(p.get("score_self_window", 0)))
        sel, code = select(st, A, k, p["l_tail"], mode, n_sinks)
        note(code)
        if status < 0:
            break
        st = compact(st, k, sel)
        if pressure_margin > 0:
            bp = int(budget) - int(pressure_margin)
            if int(np.sum(st["n_kept"])) >= bp:
                c = st["n_kept"]
                k, _, _, code = allocate(st["parent"], st["n_full"], c, [int(leaf)], bp, s, p)
                note(code)
                if status < 0:
                    break
                row[0] = int(np.sum(k))
                row[2] += int(np.sum(np.maximum(0, c - k)))
                row[3] = 1
                sel, code = select(st, A, k, p["l_tail"], mode, n_sinks)
                note(code)
                if status < 0:
                    break
                st = compact(st, k, sel)
        stats.append(row)
    return st, A, rows_seen, s, np.array(stats, np.int64).reshape(-1, 4), status
