"""Oracle for the n-gram small drafter (test infrastructure only).

The small drafter of the paper's main experiments is a training-free lookup
(App. C.1, the small drafter's implementation):
  * at prefill, every context position i caches the target's top-m next
    tokens after x_<=i with their target probabilities;
  * at a small step, the suffix of each frontier node's prefix (context, then
    the draft tokens on the node's root path) is matched against the context
    with the longest n-gram available, shortening it on a miss; the cached
    candidates of the matched position become the node's children, their
    cached probabilities the edge scores p(u);
  * with no match at any length, the candidates cached at the position of the
    prompt's most frequent token are used.

Readings where the appendix is silent (applied identically in the library):
  * scores are natural logs: cand_logp = fl(x - lse) of the prefill row, the
    same two-operation fp32 rule as every other edge score;
  * the candidates of a position are its top-m by (logit desc, token asc);
  * several occurrences of the matched n-gram: the latest one (the largest
    end position j) wins;
  * n runs from n_max down to 1, and an n longer than the prefix is skipped;
    a match may end anywhere in the context, the last position included (the
    root's own prefix matches there, giving the target's prefill prediction);
  * "most frequent token": highest count in x_<ctx_len, ties to the smallest
    token id; its position = its last occurrence;
  * an empty context (ctx_len = 0) has nothing to propose: BAD_PREFIX, the
    tree is left unchanged; a fallback position outside the context raises
    BAD_NODE and the last context position is used.
Every node ranking uses (cum desc, depth asc, id asc), as in expand.
"""
from __future__ import annotations

import numpy as np

from . import tree as T

F32 = np.float32


def ngram_cache(logits: np.ndarray, context: np.ndarray, ctx_len: np.ndarray, m: int):
    """Prefill cache.  logits [B, L, V] (row i = target logits after x_<=i),
    context [B, L] tokens, ctx_len [B].  Returns (cand_tok [B, L, m],
    cand_logp [B, L, m], fallback_pos [B], err); every row is cached (rows at
    or past ctx_len are never looked up)."""
    B, L, V = logits.shape
    tok = np.zeros((B, L, m), np.int32)
    lp = np.zeros((B, L, m), np.float32)
    err = 0
    for b in range(B):
        for i in range(L):
            _, bad = T.clean_logits(logits[b, i])
            if bad:
                err |= T.DERR_NONFINITE
            lse = T.row_lse(logits[b, i])
            t, x = T.row_topk(logits[b, i], m)
            tok[b, i] = t
            lp[b, i] = [T.edge_logp(v, lse) for v in x]
    fb, e2 = fallback_position(context, ctx_len, V)
    return tok, lp, fb, err | e2


def fallback_position(context: np.ndarray, ctx_len: np.ndarray, V: int):
    """Last position of the most frequent context token (ties to the smallest
    token id; tokens outside [0, V) are skipped with BAD_NODE); -1 for an empty
    context.  Returns (fallback_pos [B], err)."""
    B = context.shape[0]
    fb = np.full(B, -1, np.int32)
    err = 0
    for b in range(B):
        n = int(ctx_len[b])
        ctx = [int(x) for x in context[b, :n]]
        if any(x < 0 or x >= V for x in ctx):
            err |= T.DERR_BAD_NODE
        ctx = [x for x in ctx if 0 <= x < V]
        if ctx:
            counts = {}
            for x in ctx:
                counts[x] = counts.get(x, 0) + 1
            best = min(counts, key=lambda x: (-counts[x], x))
            fb[b] = max(i for i in range(n) if int(context[b, i]) == best)
    return fb, err


def match_position(ctx, prefix, n_max: int):
    """Latest end position j in ctx of the longest suffix of `prefix` (length
    n_max down to 1) that occurs in ctx; -1 when none does."""
    for n in range(min(n_max, len(prefix)), 0, -1):
        suf = list(prefix[-n:])
        for j in range(len(ctx) - 1, n - 2, -1):
            if list(ctx[j - n + 1:j + 1]) == suf:
                return j
    return -1


def expand_ngram(tree: T.Tree, frontier: np.ndarray, n_frontier, context: np.ndarray,
                 ctx_len: np.ndarray, cand_tok: np.ndarray, cand_logp: np.ndarray,
                 fallback_pos: np.ndarray, K: int, N: int, n_max: int):
    """One small-drafter step with the n-gram drafter, applied to a copy:
    the Alg. 1 expansion with each frontier node's children read from the
    cache at its matched position (top-K of the m cached, K <= m).  Children
    get ids n_b + f*K + j, logp = the cached score, cum = fl(cum_v + logp).
    Returns (tree', match_pos [B, F] (-1 padded), next_frontier [B, N],
    n_next [B], err)."""
    B, F = frontier.shape
    t = tree.copy()
    err = 0
    pos_out = np.full((B, F), -1, np.int32)
    nxt = np.full((B, N), T.NO_NODE, np.int32)
    n_next = np.zeros(B, np.int32)
    for b in range(B):
        Fb = F if n_frontier is None else int(n_frontier[b])
        nb = int(t.n_nodes[b])
        fr = [int(v) for v in frontier[b, :Fb]]
        Lb = int(ctx_len[b])
        if any(v < -1 or v >= nb for v in fr):
            err |= T.DERR_BAD_NODE
            continue
        if Lb <= 0:
            err |= T.DERR_BAD_PREFIX
            continue
        if nb + Fb * K > t.cap:
            err |= T.DERR_CAPACITY
            continue
        ctx = [int(x) for x in context[b, :Lb]]
        par = t.parent[b, :nb].astype(np.int64)
        kids = []
        for f, v in enumerate(fr):
            path = [] if v < 0 else [int(t.token[b, u]) for u in T.path_of(par, v)]
            j = match_position(ctx, ctx + path, n_max)
            if j < 0:
                j = int(fallback_pos[b])
                if not 0 <= j < Lb:          # not a context position
                    err |= T.DERR_BAD_NODE
                    j = Lb - 1
            pos_out[b, f] = j
            cum_v = F32(0.0) if v == -1 else t.cum[b, v]
            d_v = 0 if v == -1 else int(t.depth[b, v])
            for k in range(K):
                nid = nb + f * K + k
                lp = F32(cand_logp[b, j, k])
                c = F32(cum_v + lp)
                t.parent[b, nid] = v
                t.token[b, nid] = cand_tok[b, j, k]
                t.depth[b, nid] = d_v + 1
                t.logp[b, nid] = lp
                t.cum[b, nid] = c
                t.visited[b, nid] = 0
                kids.append(T.node_key(c, d_v + 1, nid))
        t.n_nodes[b] = nb + Fb * K
        kids.sort()
        sel = [k[2] for k in kids[:N]]
        nxt[b, :len(sel)] = sel
        n_next[b] = len(sel)
    return t, pos_out, nxt, n_next, err
