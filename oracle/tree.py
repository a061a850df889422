"""Oracle for the draft-tree calls (test infrastructure only).

Scores live in the natural-log domain: the paper's edge score p(u) and path
score s(v) = prod p(u) (Sec. 3.1) are stored as ``logp = log p`` and
``cum = log s`` (so s(root) = 1 becomes cum = 0).  Every float that decides a
selection is fp32 and is produced by exactly two IEEE fp32 operations per node:

    logp = fl(x - lse)          x = the token's logit, lse = the row's log-sum-exp
    cum  = fl(cum_parent + logp)

``lse`` itself is computed in fp64 and rounded once to fp32; callers may pass
the GPU's exported lse instead (``lse_override``) so that every later step runs
on identical fp32 operands.

Readings of the paper where it is silent (all applied identically here and in
the library):
  * Top_m over a logits row ranks tokens by (logit desc, token id asc).
  * Every node ranking (Top_W of a candidate pool) uses the key Alg. 3 fixes for
    pruning: (cum desc, depth asc, id asc); the root has id -1, cum 0, depth 0.
  * -0.0 ranks equal to +0.0; NaN and +inf logits are read as -inf and raise
    the NONFINITE error bit; a row whose logits are all -inf has lse = -inf
    and gives its children logp = -inf.
  * Expansion attaches every child of every frontier node (Alg. 1) and also
    returns the next step's frontier Top_W over those children.
  * Node ids are dense and topological: children get ids after their parent.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from .attention import path_of, sanitize_parent

F32 = np.float32
NEG_INF = F32(-np.inf)

# Device error word bits (same meaning as the library documents).
DERR_BAD_PARENT = 1
DERR_CAPACITY = 2
DERR_NONFINITE = 4
DERR_BAD_PREFIX = 8
DERR_BAD_NODE = 16

NO_NODE = -2  # padding for frontier outputs (-1 is the root)

# Variant flags of the middle step (the two ablations of Sec. 5.3 and a
# duplicate-sibling filter); 0 = TreeGraft as described in Sec. 3.2.
POOL_NEWONLY = 1    # w/o EG: the pool is the previous step's new nodes
GRAFT_OVERWRITE = 2  # w/o ND: grafting replaces the frontier nodes' subtrees
GRAFT_DEDUP = 4      # a child whose token an existing sibling has is skipped


@dataclass
class Tree:
    """Host copy of the caller-owned tree (one row of ``cap`` slots per batch)."""
    parent: np.ndarray
    token: np.ndarray
    depth: np.ndarray
    logp: np.ndarray
    cum: np.ndarray
    visited: np.ndarray
    root_visited: np.ndarray
    n_nodes: np.ndarray
    cap: int = field(default=0)

    @staticmethod
    def empty(B: int, cap: int) -> "Tree":
        return Tree(
            parent=np.full((B, cap), -1, np.int32),
            token=np.zeros((B, cap), np.int32),
            depth=np.zeros((B, cap), np.int32),
            logp=np.zeros((B, cap), np.float32),
            cum=np.zeros((B, cap), np.float32),
            visited=np.zeros((B, cap), np.uint8),
            root_visited=np.zeros(B, np.uint8),
            n_nodes=np.zeros(B, np.int32),
            cap=cap,
        )

    def copy(self) -> "Tree":
        return Tree(*(np.array(getattr(self, f), copy=True) for f in
                      ("parent", "token", "depth", "logp", "cum", "visited",
                       "root_visited", "n_nodes")), cap=self.cap)


# ---------------------------------------------------------------- logits rows

def clean_logits(x: np.ndarray):
    """(fp32 row with NaN/+inf read as -inf, whether any was seen)."""
    x = np.asarray(x, dtype=np.float32)
    bad = np.isnan(x) | (x == np.inf)
    return np.where(bad, NEG_INF, x).astype(np.float32), bool(bad.any())


def row_lse(x: np.ndarray) -> np.float32:
    """log sum_v exp(x_v) of one logits row: fp64, max-subtracted, rounded once."""
    xc, _ = clean_logits(x)
    x64 = xc.astype(np.float64)
    m = x64.max()
    if m == -np.inf:
        return NEG_INF
    return F32(m + np.log(np.sum(np.exp(x64 - m))))


def row_topk(x: np.ndarray, k: int):
    """Top_m of Alg. 1/2: the k tokens with the largest logits.

    Full sort of the row by (logit desc, token asc); returns (tokens, logits).
    """
    xc, _ = clean_logits(x)
    order = np.lexsort((np.arange(xc.shape[0]), -xc.astype(np.float64)))
    top = order[:k]
    return top.astype(np.int32), xc[top]


def edge_logp(x: np.float32, lse: np.float32) -> np.float32:
    """log p(u) = fl(x - lse); -inf when the row has no finite logit."""
    if lse == NEG_INF:
        return NEG_INF
    return F32(x) - F32(lse)


def node_key(cum, depth, nid):
    """Ranking key, best first: (cum desc, depth asc, id asc)."""
    return (-float(cum), int(depth), int(nid))


# ------------------------------------------------------------------- expand

def expand(tree: Tree, logits: np.ndarray, frontier: np.ndarray,
           n_frontier, K: int, N: int, lse_override=None):
    """One standard expansion step (Sec. 3.1; Alg. 1), applied to a copy.

    logits: [B, F, V] fp32, row f = the drafter's next-token logits at
    frontier node ``frontier[b, f]`` (-1 = root).  ``n_frontier[b]`` rows are
    live (None = all F).  Returns (tree', row_lse [B, F], next_frontier [B, N],
    n_next [B], err).  Rows beyond n_frontier keep row_lse = NaN.
    """
    B, F, V = logits.shape
    t = tree.copy()
    err = 0
    lse_out = np.full((B, F), np.nan, np.float32)
    nxt = np.full((B, N), NO_NODE, np.int32)
    n_next = np.zeros(B, np.int32)
    for b in range(B):
        Fb = F if n_frontier is None else int(n_frontier[b])
        nb = int(t.n_nodes[b])
        fr = [int(v) for v in frontier[b, :Fb]]
        for f in range(Fb):
            _, bad = clean_logits(logits[b, f])
            if bad:
                err |= DERR_NONFINITE
            lse_out[b, f] = row_lse(logits[b, f]) if lse_override is None \
                else F32(lse_override[b, f])
        if any(v < -1 or v >= nb for v in fr):
            err |= DERR_BAD_NODE
            continue
        if nb + Fb * K > t.cap:
            err |= DERR_CAPACITY
            continue
        kids = []
        for f, v in enumerate(fr):
            lse = lse_out[b, f]
            toks, vals = row_topk(logits[b, f], K)
            cum_v = F32(0.0) if v == -1 else t.cum[b, v]
            d_v = 0 if v == -1 else int(t.depth[b, v])
            for j in range(K):
                nid = nb + f * K + j
                lp = edge_logp(vals[j], lse)
                c = F32(cum_v + lp)
                t.parent[b, nid] = v
                t.token[b, nid] = toks[j]
                t.depth[b, nid] = d_v + 1
                t.logp[b, nid] = lp
                t.cum[b, nid] = c
                t.visited[b, nid] = 0
                kids.append(node_key(c, d_v + 1, nid))
        t.n_nodes[b] = nb + Fb * K
        kids.sort()
        sel = [k[2] for k in kids[:N]]
        nxt[b, :len(sel)] = sel
        n_next[b] = len(sel)
    return t, lse_out, nxt, n_next, err


# ------------------------------------------------------------ rescore + graft

def pool_of(tree: Tree, b: int, flags: int = 0, new_from=None):
    """Middle-drafter candidate pool (Sec. 3.2): C = V(T) minus P, i.e. the
    unvisited ids plus the root (-1) while the root is unvisited.  With
    POOL_NEWONLY (the w/o EG ablation, Sec. 5.3) C = N_k instead: the ids
    new_from[b] .. n_b - 1 made by the previous step, the root when
    new_from[b] == -1 (the first step, whose tree is the root alone)."""
    nb = int(tree.n_nodes[b])
    if flags & POOL_NEWONLY:
        lo = int(new_from[b])
        return list(range(max(lo, -1), nb))
    C = [v for v in range(nb) if not tree.visited[b, v]]
    if not tree.root_visited[b]:
        C = [-1] + C
    return C


def needed_rows(tree: Tree, b: int, flags: int = 0, new_from=None):
    """Logits rows a middle step reads: each pool node's own row (its children)
    and the row of each pool node's parent (its edge score)."""
    rows = set()
    for v in pool_of(tree, b, flags, new_from):
        rows.add(v + 1)
        if v != -1:
            rows.add(int(tree.parent[b, v]) + 1)
    return sorted(rows)


def overwrite_compact(t: Tree, b: int, F):
    """The w/o ND reading (Sec. 5.3): attaching under a frontier node
    overwrites its existing children, so every node with a strict ancestor in
    F is removed.  Frontier nodes inside a removed subtree are removed with
    it.  The surviving nodes keep their order and are renumbered densely
    (parents stay before children).  Returns (old -> new id map, surviving F
    in the order of F, new id)."""
    nb = int(t.n_nodes[b])
    inF = set(F)
    dead = np.zeros(nb, bool)
    for u in range(nb):           # ids are topological
        p = int(t.parent[b, u])
        dead[u] = (p in inF) or (p >= 0 and dead[p])
    newid = np.full(nb, -1, np.int64)
    keep = [u for u in range(nb) if not dead[u]]
    for i, u in enumerate(keep):
        newid[u] = i
    cols = {name: getattr(t, name)[b, :nb].copy()
            for name in ("parent", "token", "depth", "logp", "cum", "visited")}
    for name, col in cols.items():
        arr = getattr(t, name)
        for i, u in enumerate(keep):
            arr[b, i] = col[u]
    for i, u in enumerate(keep):
        p = int(cols["parent"][u])
        t.parent[b, i] = -1 if p < 0 else newid[p]
    t.n_nodes[b] = len(keep)
    Fs = [(-1 if v < 0 else int(newid[v])) for v in F if v < 0 or not dead[v]]
    Fold = [v for v in F if v < 0 or not dead[v]]
    return newid, Fold, Fs


def rescore_graft(tree: Tree, strong: np.ndarray, W: int, M: int,
                  lse_override=None, N: int = 0, flags: int = 0, new_from=None):
    """One middle-drafter step of Alg. 2, applied to a copy.

    strong: [B, R, V] fp32; row 0 = the middle drafter's logits at the root,
    row 1 + i = at node i (its cached next-token logits).  Steps, in the
    paper's order:
      1. C = unvisited nodes (+ root while unvisited).
      2. For every non-root v in C (ascending id = topological order):
         logp[v] = fl(x[pa(v)+1][token v] - lse[pa(v)+1]),
         cum[v]  = fl(cum[pa v] + logp[v])   (cum[root] = 0).
      3. F = Top_W(C) by (cum desc, depth asc, id asc).
      4. For each v in F (rank f) and each of its row's top-M tokens (rank j):
         attach a new child, id n_b + f*M + j, never touching existing nodes.
      5. P <- P u C: every pre-existing node and the root become visited.
    The grafted children are N_{k+1}, the pool of a following small step
    (Sec. 3.2: a small step's pool is the previous step's new nodes); with
    N > 0 their Top_N by (cum desc, depth asc, id asc) is also returned.
    Variant flags (Sec. 5.3 ablations; 0 = the paper's method):
      POOL_NEWONLY   step 1 uses C = N_k (ids >= new_from[b]; see pool_of);
      GRAFT_OVERWRITE before step 4 the frontier nodes' existing subtrees are
                     removed and the tree compacted (overwrite_compact); F
                     and the children then use the new ids;
      GRAFT_DEDUP    step 4 skips a child whose token an existing child of
                     the same parent already carries; the kept children take
                     dense ids in (slot, rank) order.  (With OVERWRITE a
                     frontier node has no children left, so nothing is
                     skipped.)
    The capacity check uses the upper bound n_b + |F|*M in every variant.
    Returns (tree', row_lse [B, R], graft_frontier [B, W], n_graft [B], err)
    and, when N > 0, also (next_frontier [B, N], n_next [B]).  row_lse holds
    NaN for rows that were not needed.
    """
    B, R, V = strong.shape
    t = tree.copy()
    err = 0
    lse_out = np.full((B, R), np.nan, np.float32)
    fr_out = np.full((B, W), NO_NODE, np.int32)
    n_graft = np.zeros(B, np.int32)
    nxt = np.full((B, max(N, 1)), NO_NODE, np.int32)
    n_next = np.zeros(B, np.int32)
    for b in range(B):
        nb = int(t.n_nodes[b])
        if nb + 1 > R:
            err |= DERR_BAD_NODE
            continue
        C = pool_of(t, b, flags, new_from)
        rows = needed_rows(t, b, flags, new_from)
        for r in rows:
            _, bad = clean_logits(strong[b, r])
            if bad:
                err |= DERR_NONFINITE
            lse_out[b, r] = row_lse(strong[b, r]) if lse_override is None \
                else F32(lse_override[b, r])
        nF = min(W, len(C))
        if nb + nF * M > t.cap:
            err |= DERR_CAPACITY
            continue
        # 2. rescoring, parents before children
        for v in C:
            if v == -1:
                continue
            p = int(t.parent[b, v])
            x, _ = clean_logits(strong[b, p + 1, t.token[b, v]:t.token[b, v] + 1])
            lp = edge_logp(x[0], lse_out[b, p + 1])
            cum_p = F32(0.0) if p == -1 else t.cum[b, p]
            t.logp[b, v] = lp
            t.cum[b, v] = F32(cum_p + lp)
        # 3. reselection
        cand = sorted(node_key(0.0, 0, -1) if v == -1 else
                      node_key(t.cum[b, v], t.depth[b, v], v) for v in C)
        Fsel = [k[2] for k in cand[:nF]]
        # 5 (first half). P <- P u C (all unvisited nodes for the paper's
        # pool; only N_k with POOL_NEWONLY)
        for v in C:
            if v == -1:
                t.root_visited[b] = 1
            else:
                t.visited[b, v] = 1
        # variant: overwrite the frontier nodes' subtrees
        Frows = list(Fsel)      # logits rows stay those of the old ids
        Fids = list(Fsel)
        if flags & GRAFT_OVERWRITE:
            _, Frows, Fids = overwrite_compact(t, b, Fsel)
        nb2 = int(t.n_nodes[b])
        # 4. grafting (non-destructive unless overwritten above)
        kids = []
        nid = nb2
        for f, (v_row, v) in enumerate(zip(Frows, Fids)):
            toks, vals = row_topk(strong[b, v_row + 1], M)
            lse = lse_out[b, v_row + 1]
            cum_v = F32(0.0) if v == -1 else t.cum[b, v]
            d_v = 0 if v == -1 else int(t.depth[b, v])
            sib = set()
            if flags & GRAFT_DEDUP:
                sib = {int(t.token[b, u]) for u in range(nb2) if int(t.parent[b, u]) == v}
            for j in range(M):
                if not (flags & (GRAFT_OVERWRITE | GRAFT_DEDUP)):
                    nid = nb2 + f * M + j
                elif int(toks[j]) in sib:
                    continue
                lp = edge_logp(vals[j], lse)
                t.parent[b, nid] = v
                t.token[b, nid] = toks[j]
                t.depth[b, nid] = d_v + 1
                t.logp[b, nid] = lp
                t.cum[b, nid] = F32(cum_v + lp)
                t.visited[b, nid] = 0
                kids.append(node_key(t.cum[b, nid], d_v + 1, nid))
                nid += 1
        kids.sort()
        sel = [k[2] for k in kids[:N]]
        nxt[b, :len(sel)] = sel
        n_next[b] = len(sel)
        t.n_nodes[b] = nb2 + len(kids)
        fr_out[b, :len(Fids)] = Fids
        n_graft[b] = len(Fids)
    if N > 0:
        return t, lse_out, fr_out, n_graft, err, nxt, n_next
    return t, lse_out, fr_out, n_graft, err


# ------------------------------------------------------------------- accept

def accept(parent: np.ndarray, token: np.ndarray, n_nodes: np.ndarray,
           greedy: np.ndarray, max_depth: int):
    """Greedy acceptance by brute force over every root-to-node path.

    greedy: [B, cap + 1], row 0 = the target's arg-max token at the root, row
    1 + i = at node i.  A node is acceptable iff every node u on its path
    carries the token the target emits after u's parent.  The accepted node is
    the deepest acceptable one (ties to the smallest id); nodes deeper than
    ``max_depth`` are not considered (CAPACITY bit if one would have been
    acceptable).  Returns (accept_len [B], accept_path [B, max_depth] padded
    -1, bonus [B], err).  accept_len counts draft nodes, not the bonus token.
    """
    B = parent.shape[0]
    err = 0
    A = np.zeros(B, np.int32)
    paths = np.full((B, max_depth), -1, np.int32)
    bonus = np.zeros(B, np.int32)
    for b in range(B):
        n = int(n_nodes[b])
        raw = np.asarray(parent[b, :n], dtype=np.int64)
        if np.any((raw < -1) | (raw >= np.arange(n))):
            err |= DERR_BAD_PARENT
        par = sanitize_parent(raw)
        best = None
        for v in range(n):
            path = path_of(par, v)
            if all(int(token[b, u]) == int(greedy[b, par[u] + 1]) for u in path):
                if len(path) > max_depth:
                    err |= DERR_CAPACITY
                    continue
                if best is None or len(path) > len(best):
                    best = path
        if best is None:
            bonus[b] = greedy[b, 0]
        else:
            A[b] = len(best)
            paths[b, :len(best)] = best
            bonus[b] = greedy[b, best[-1] + 1]
    return A, paths, bonus, err


def greedy_argmax(logits: np.ndarray, n_nodes: np.ndarray):
    """The target's greedy tokens (temperature 0, App. E) from its logits
    [B, R, V]: greedy[b, r] = arg-max of row r for r <= n_nodes[b] (ties to
    the smallest token id; NaN and +inf read as -inf, NONFINITE bit), -1 for
    rows past the tree (BAD_NODE when the tree needs a row past R).  Returns
    (greedy [B, R], err)."""
    B, R, V = logits.shape
    g = np.full((B, R), -1, np.int32)
    err = 0
    for b in range(B):
        if int(n_nodes[b]) + 1 > R:
            err |= DERR_BAD_NODE
        for r in range(min(R, int(n_nodes[b]) + 1)):
            x, bad = clean_logits(logits[b, r])
            if bad:
                err |= DERR_NONFINITE
            g[b, r] = int(np.argmax(x))   # first maximum = smallest token id
    return g, err


def accept_logits(parent, token, n_nodes, logits, max_depth: int):
    """Acceptance straight from the target's logits: greedy_argmax, then
    accept.  Returns (greedy [B, cap + 1] with -1 past the rows computed,
    accept_len, accept_path, bonus, err)."""
    g, e1 = greedy_argmax(logits, n_nodes)
    B, cap = parent.shape
    full = np.full((B, cap + 1), -1, np.int32)
    w = min(g.shape[1], cap + 1)
    full[:, :w] = g[:, :w]
    A, paths, bonus, e2 = accept(parent, token, n_nodes, full, max_depth)
    return full, A, paths, bonus, e1 | e2


# -------------------------------------------------------------- global prune

def global_prune(parent: np.ndarray, cum: np.ndarray, n: int, B_ver: int):
    """Alg. 3, step by step, for one tree of ``n`` non-root nodes.

    Returns dict with ``kept`` (original ids of kept non-root nodes, in the new
    order), ``parent`` (new parent array, -1 = root), ``mask`` ([M', M'] with the
    root as row/column 0), ``position_ids`` (depth, root 0) and
    ``retrieval`` (root-to-leaf paths in new indices incl. the root 0,
    padded with -1).  The kept nodes are re-indexed by (depth, original id),
    which puts parents before children as Alg. 3 requires.
    """
    par = sanitize_parent(np.asarray(parent[:n]))
    depth = np.array([len(path_of(par, v)) for v in range(n)], dtype=np.int64)
    M = B_ver + 1
    if n + 1 <= M:
        keep = set(range(n))
    else:
        ranked = sorted(range(n), key=lambda v: node_key(cum[v], depth[v], v))
        keep = set()
        size = 1  # the root
        for v in ranked:
            chain = []
            u = v
            while u != -1 and u not in keep:
                chain.append(u)
                u = int(par[u])
            if size + len(chain) <= M:
                keep.update(chain)
                size += len(chain)
            if size == M:
                break
    kept = sorted(keep, key=lambda v: (depth[v], v))
    new_id = {v: i + 1 for i, v in enumerate(kept)}   # verify index, root = 0
    nparent = np.array([-1 if par[v] == -1 else new_id[int(par[v])] - 1
                        for v in kept], dtype=np.int32)
    Mk = len(kept) + 1
    vpar = [-1] + [0 if par[v] == -1 else new_id[int(par[v])] for v in kept]
    mask = np.zeros((Mk, Mk), dtype=np.uint8)
    for u in range(Mk):
        w = u
        while w != -1:
            mask[u, w] = 1
            w = vpar[w]
    pos = np.array([0] + [int(depth[v]) for v in kept], dtype=np.int32)
    is_parent = set(vpar[1:])
    leaves = [u for u in range(Mk) if u not in is_parent]
    width = int(pos.max()) + 1
    retr = np.full((len(leaves), width), -1, dtype=np.int32)
    for r, u in enumerate(leaves):
        chain = []
        w = u
        while w != -1:
            chain.append(w)
            w = vpar[w]
        retr[r, :len(chain)] = chain[::-1]
    return dict(kept=np.array(kept, dtype=np.int32), parent=nparent, mask=mask,
                position_ids=pos, retrieval=retr)
