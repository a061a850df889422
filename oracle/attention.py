"""Oracle for tree-verify attention (test infrastructure only).

Definition followed (Alg. 3, tree-attention mask; Sec. 3.1, root = verified
prefix): a draft node u attends to key v iff v is the root, an ancestor of u, or
u itself.  In the verify layout the root is the whole verified prefix (cache
positions [0, L_b)) and tree node j lives at cache position L_b + j.  So for
batch b, tree node i and query head h (KV head g = h // (Hq / Hkv)):

  keys    = K[b, g, 0:L_b]  followed by  K[b, g, L_b + a] for a on path(i)
  s_j     = sm_scale * <q, k_j>                (fp64)
  out     = sum_j softmax(s)_j v_j             (fp64, max-subtracted)

where path(i) = [a_1, ..., a_t = i] is the root-to-node list of tree nodes
(follow ``parent`` until -1).  No mask matrix is built here.

Reading of the paper where it is silent: parent -1 means "hangs under the
prefix end"; the softmax scale is a parameter; query head h uses KV head
h // (Hq / Hkv) (contiguous groups).  A parent outside [-1, i-1] is treated
as -1, the rule the library documents for that input error.
"""
from __future__ import annotations

import numpy as np


def sanitize_parent(parent: np.ndarray) -> np.ndarray:
    """parent[i] outside [-1, i-1] is read as -1 (documented error fallback)."""
    p = np.asarray(parent, dtype=np.int64).copy()
    idx = np.arange(len(p))
    p[(p < -1) | (p >= idx)] = -1
    return p


def path_of(parent: np.ndarray, i: int) -> list:
    """Root-to-node list of tree nodes ending at ``i``."""
    out = []
    v = int(i)
    while v != -1:
        out.append(v)
        v = int(parent[v])
    return out[::-1]


def tree_verify_attention(q, k_cache, v_cache, parent, prefix_len, sm_scale,
                          rows=None):
    """fp64 tree attention.

    q: [B, N, Hq, D]; k_cache, v_cache: [B, Hkv, S_max, D]; parent: [B, N];
    prefix_len: [B].  Inputs may be any real dtype; they are upcast exactly.

    rows=None computes every output and returns [B, N, Hq, D] fp64.  Otherwise
    ``rows`` is a list of (b, i, h) triples and the result is [len(rows), D].
    """
    q = np.asarray(q)
    B, N, Hq, D = q.shape
    Hkv = k_cache.shape[1]
    if Hq % Hkv:
        raise ValueError("Hq must be a multiple of Hkv")
    G = Hq // Hkv
    scale = float(sm_scale)

    def one_group(b, g, nodes, heads):
        """Outputs for the given (node, head) pairs of one (batch, KV head)."""
        L = int(prefix_len[b])
        par = sanitize_parent(parent[b])
        Kp = np.asarray(k_cache[b, g, :L], dtype=np.float64)
        Vp = np.asarray(v_cache[b, g, :L], dtype=np.float64)
        Kt = np.asarray(k_cache[b, g, L:L + N], dtype=np.float64)
        Vt = np.asarray(v_cache[b, g, L:L + N], dtype=np.float64)
        res = []
        for i, h in zip(nodes, heads):
            qi = np.asarray(q[b, i, h], dtype=np.float64)
            path = path_of(par, i)
            s = np.concatenate([Kp @ qi, Kt[path] @ qi]) * scale
            e = np.exp(s - s.max())
            p = e / e.sum()
            res.append(p[:L] @ Vp + p[L:] @ Vt[path])
        return res

    if rows is not None:
        out = np.empty((len(rows), D), dtype=np.float64)
        for r, (b, i, h) in enumerate(rows):
            out[r] = one_group(b, h // G, [i], [h])[0]
        return out

    out = np.empty((B, N, Hq, D), dtype=np.float64)
    for b in range(B):
        for g in range(Hkv):
            nodes = [i for i in range(N) for _ in range(G)]
            heads = [g * G + hh for _ in range(N) for hh in range(G)]
            for (i, h), o in zip(zip(nodes, heads), one_group(b, g, nodes, heads)):
                out[b, i, h] = o
    return out


def tree_verify_attention_fast(q, k_cache, v_cache, parent, prefix_len, sm_scale):
    """Same definition, with the prefix scores of a (batch, KV head) computed by
    one matrix product (a library primitive) instead of one per node.

    Nothing else changes: each row still concatenates its prefix scores with
    its own path scores and takes one softmax.  Used for the large parity cases
    where the per-node loop would take minutes.
    """
    q = np.asarray(q)
    B, N, Hq, D = q.shape
    Hkv = k_cache.shape[1]
    G = Hq // Hkv
    scale = float(sm_scale)
    out = np.empty((B, N, Hq, D), dtype=np.float64)
    for b in range(B):
        L = int(prefix_len[b])
        par = sanitize_parent(parent[b])
        paths = [path_of(par, i) for i in range(N)]
        for g in range(Hkv):
            Kp = np.asarray(k_cache[b, g, :L], dtype=np.float64)
            Vp = np.asarray(v_cache[b, g, :L], dtype=np.float64)
            Kt = np.asarray(k_cache[b, g, L:L + N], dtype=np.float64)
            Vt = np.asarray(v_cache[b, g, L:L + N], dtype=np.float64)
            Qg = np.asarray(q[b, :, g * G:(g + 1) * G], dtype=np.float64)  # [N, G, D]
            Sp = (Qg.reshape(N * G, D) @ Kp.T).reshape(N, G, L) * scale
            for i in range(N):
                path = paths[i]
                St = (Qg[i] @ Kt[path].T) * scale               # [G, t]
                s = np.concatenate([Sp[i], St], axis=1)         # [G, L + t]
                e = np.exp(s - s.max(axis=1, keepdims=True))
                p = e / e.sum(axis=1, keepdims=True)
                out[b, i, g * G:(g + 1) * G] = p[:, :L] @ Vp + p[:, L:] @ Vt[path]
    return out


def kv_compact(k_cache, v_cache, prefix_len, path, n_path):
    """Cache update after acceptance, as a plain gather (returns new arrays).

    The verified tokens become the next turn's prefix (Sec. 3.1: the root of
    the draft tree is the verified prefix).  In the verify layout tree slot a
    of sequence b holds the K/V of tree node a at cache row L_b + a; the
    accepted chain is given as tree slots path[b, 0:n_b] (the root's slot 0
    first when it carries a token, then the accepted nodes, parents before
    children).  Afterwards rows L_b + j, j < n_b, hold what rows
    L_b + path[b, j] held, the other rows are unchanged, and the prefix
    length becomes L_b + n_b.

    Reading where the paper is silent: the chain must be strictly increasing
    with path[b, j] >= j (it is, for a root-to-node path in a parents-first
    layout) and fit the cache (L_b + path[b, j] < S_max); a sequence that
    violates this is left untouched, keeps its length and raises
    DERR_BAD_NODE.
    """
    k2 = np.array(k_cache, copy=True)
    v2 = np.array(v_cache, copy=True)
    B, _, S_max, _ = k2.shape
    new_len = np.zeros(B, dtype=np.int32)
    err = 0
    for b in range(B):
        L, n = int(prefix_len[b]), int(n_path[b])
        new_len[b] = L
        p = [int(x) for x in path[b, :max(n, 0)]]
        ok = 0 <= n <= path.shape[1] and L >= 0
        ok = ok and all(p[j] >= j and (j == 0 or p[j] > p[j - 1]) for j in range(n))
        ok = ok and all(L + x < S_max for x in p)
        if not ok:
            err |= 16
            continue
        rows_k = [k_cache[b, :, L + x, :].copy() for x in p]
        rows_v = [v_cache[b, :, L + x, :].copy() for x in p]
        for j in range(n):
            k2[b, :, L + j, :] = rows_k[j]
            v2[b, :, L + j, :] = rows_v[j]
        new_len[b] = L + n
    return k2, v2, new_len, err
