"""Pins for the attention oracle (CPU only).

Each test checks the oracle against something other than itself: torch's CPU
scaled-dot-product attention with an explicit causal mask (a library routine),
a dense formulation through an ancestor mask matrix built by transitive
closure, closed forms (single visible key, constant keys) and invariances the
tree-attention mask of Alg. 3 fixes.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as Fnn

import workloads as W
from oracle.attention import (kv_compact, path_of, sanitize_parent, tree_verify_attention,
                              tree_verify_attention_fast)


def _inputs(seed, B, N, Hq, Hkv, D, L, extra=0):
    g = W.rng(seed)
    S = L + N + extra
    q = W.normal(g, (B, N, Hq, D))
    k = W.normal(g, (B, Hkv, S, D))
    v = W.normal(g, (B, Hkv, S, D))
    return q, k, v


def test_chain_tree_is_causal_attention():
    """A chain tree (parent[i] = i - 1) is ordinary causal attention over
    prefix + tree tokens; GQA uses contiguous head groups."""
    B, N, Hq, Hkv, D, L = 2, 9, 8, 2, 16, 7
    q, k, v = _inputs(1, B, N, Hq, Hkv, D, L)
    parent = np.tile(np.arange(-1, N - 1, dtype=np.int32), (B, 1))
    plen = np.array([L, L])
    scale = 0.37
    got = tree_verify_attention(q, k, v, parent, plen, scale)

    G = Hq // Hkv
    qt = torch.from_numpy(q).double().permute(0, 2, 1, 3)          # [B,Hq,N,D]
    kt = torch.from_numpy(k[:, :, :L + N]).double().repeat_interleave(G, dim=1)
    vt = torch.from_numpy(v[:, :, :L + N]).double().repeat_interleave(G, dim=1)
    qpos = torch.arange(N)[:, None] + L
    kpos = torch.arange(L + N)[None, :]
    mask = kpos <= qpos
    ref = Fnn.scaled_dot_product_attention(qt, kt, vt, attn_mask=mask, scale=scale)
    ref = ref.permute(0, 2, 1, 3).numpy()
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12)


def _ancestor_or_self(parent):
    """Boolean [N, N] closure of the parent relation (Warshall)."""
    N = len(parent)
    A = np.eye(N, dtype=bool)
    for i, p in enumerate(parent):
        if p >= 0:
            A[i, p] = True
    for m in range(N):
        A |= A[:, m:m + 1] & A[m:m + 1, :]
    return A


@pytest.mark.parametrize("seed", range(6))
def test_random_tree_matches_dense_masked_attention(seed):
    """Dense attention over all L + N keys with mask(u, v) = v in prefix or
    v ancestor-or-self of u equals the per-path definition."""
    g = W.rng(100 + seed)
    B, N, Hq, Hkv, D = 2, 13, 4, 2, 8
    plen = np.array([int(g.integers(0, 6)), int(g.integers(0, 6))])
    L = int(plen.max())
    q, k, v = _inputs(200 + seed, B, N, Hq, Hkv, D, L, extra=3)
    parent = np.stack([W.uniform_parents(g, N) for _ in range(B)])
    got = tree_verify_attention(q, k, v, parent, plen, 0.5)
    G = Hq // Hkv
    for b in range(B):
        Lb = plen[b]
        anc = _ancestor_or_self(parent[b])
        for h in range(Hq):
            Kb = k[b, h // G, :Lb + N].astype(np.float64)
            Vb = v[b, h // G, :Lb + N].astype(np.float64)
            s = (q[b, :, h].astype(np.float64) @ Kb.T) * 0.5     # [N, Lb+N]
            allowed = np.concatenate([np.ones((N, Lb), bool), anc], axis=1)
            s = np.where(allowed, s, -np.inf)
            p = np.exp(s - s.max(axis=1, keepdims=True))
            p /= p.sum(axis=1, keepdims=True)
            np.testing.assert_allclose(got[b, :, h], p @ Vb, rtol=0, atol=1e-12)


def test_fast_form_equals_per_row_form():
    g = W.rng(7)
    B, N, Hq, Hkv, D, L = 2, 17, 8, 2, 16, 11
    q, k, v = _inputs(8, B, N, Hq, Hkv, D, L)
    parent = np.stack([W.uniform_parents(g, N) for _ in range(B)])
    plen = np.array([L, 3])
    a = tree_verify_attention(q, k, v, parent, plen, 0.25)
    b = tree_verify_attention_fast(q, k, v, parent, plen, 0.25)
    np.testing.assert_allclose(a, b, rtol=0, atol=1e-12)


def test_empty_prefix_root_level_node_returns_its_value():
    """With L = 0 a node under the root sees only itself: softmax of one score
    is exactly 1, so the output is exactly V_self."""
    B, N, Hq, Hkv, D = 1, 5, 2, 2, 8
    q, k, v = _inputs(3, B, N, Hq, Hkv, D, 0)
    parent = np.array([[-1, 0, -1, 2, -1]], np.int32)
    got = tree_verify_attention(q, k, v, parent, np.array([0]), 1.0)
    for i in (0, 2, 4):
        for h in range(Hq):
            assert np.array_equal(got[0, i, h], v[0, h, i].astype(np.float64))


def test_constant_keys_give_mean_of_visible_values():
    B, N, Hq, Hkv, D, L = 1, 8, 2, 1, 4, 5
    q, _, v = _inputs(4, B, N, Hq, Hkv, D, L)
    k = np.ones((B, Hkv, L + N, D), np.float32) * 0.3
    parent = np.array([[-1, 0, 1, 0, -1, 4, 5, 2]], np.int32)
    got = tree_verify_attention(q, k, v, parent, np.array([L]), 0.9)
    for i in range(N):
        vis = list(range(L)) + [L + a for a in path_of(parent[0], i)]
        want = v[0, 0, vis].astype(np.float64).mean(axis=0)
        for h in range(Hq):
            np.testing.assert_allclose(got[0, i, h], want, rtol=0, atol=1e-14)


def test_poison_on_non_ancestors_changes_nothing():
    """Masked tree slots are never read: poisoning them is bitwise invisible."""
    g = W.rng(9)
    B, N, Hq, Hkv, D, L = 1, 12, 2, 1, 8, 6
    q, k, v = _inputs(10, B, N, Hq, Hkv, D, L)
    parent = W.uniform_parents(g, N)[None]
    base = tree_verify_attention(q, k, v, parent, np.array([L]), 0.5)
    for i in range(N):
        keep = set(path_of(parent[0], i))
        kp, vp = k.copy(), v.copy()
        for j in range(N):
            if j not in keep:
                kp[0, 0, L + j] = q[0, i, 0] * 1e3
                vp[0, 0, L + j] = 1e3
        pois = tree_verify_attention(q, kp, vp, parent, np.array([L]), 0.5)
        assert np.array_equal(pois[0, i], base[0, i])


def test_topology_preserving_relabel_permutes_outputs():
    g = W.rng(11)
    N, L, D = 10, 4, 8
    q, k, v = _inputs(12, 1, N, 2, 2, D, L)
    parent = W.uniform_parents(g, N)
    # random topological order: repeatedly pick any node whose parent is placed
    placed, order = {-1}, []
    while len(order) < N:
        ready = [i for i in range(N) if i not in order and parent[i] in placed]
        c = ready[g.integers(0, len(ready))]
        order.append(c)
        placed.add(c)
    new = {old: n for n, old in enumerate(order)}
    npar = np.array([-1 if parent[o] < 0 else new[parent[o]] for o in order], np.int32)
    q2 = q[:, order]
    k2, v2 = k.copy(), v.copy()
    k2[:, :, L:L + N] = k[:, :, L + np.array(order)]
    v2[:, :, L:L + N] = v[:, :, L + np.array(order)]
    a = tree_verify_attention(q, k, v, parent[None], np.array([L]), 0.4)
    b = tree_verify_attention(q2, k2, v2, npar[None], np.array([L]), 0.4)
    np.testing.assert_allclose(b, a[:, order], rtol=0, atol=1e-13)


def test_bad_parent_reads_as_root_child():
    parent = np.array([3, -5, 0, 2], np.int32)
    assert list(sanitize_parent(parent)) == [-1, -1, 0, 2]
    q, k, v = _inputs(13, 1, 4, 1, 1, 4, 2)
    a = tree_verify_attention(q, k, v, parent[None], np.array([2]), 1.0)
    b = tree_verify_attention(q, k, v, np.array([[-1, -1, 0, 2]]), np.array([2]), 1.0)
    assert np.array_equal(a, b)


def test_sampled_rows_equal_full():
    g = W.rng(14)
    q, k, v = _inputs(15, 2, 6, 4, 2, 8, 5)
    parent = np.stack([W.uniform_parents(g, 6) for _ in range(2)])
    plen = np.array([5, 2])
    full = tree_verify_attention(q, k, v, parent, plen, 0.3)
    rows = [(1, 5, 3), (0, 0, 0), (1, 2, 1)]
    part = tree_verify_attention(q, k, v, parent, plen, 0.3, rows=rows)
    for r, (b, i, h) in enumerate(rows):
        assert np.array_equal(part[r], full[b, i, h])


# ---------------------------------------------------------------- kv compact

def _accepted_chain(parent, leaf):
    """Tree slots of the root-to-leaf chain (parents first)."""
    return path_of(sanitize_parent(parent), leaf)


@pytest.mark.parametrize("seed", range(4))
def test_kv_compact_turns_the_accepted_chain_into_causal_prefix(seed):
    """After compaction, the accepted leaf's output equals plain causal
    attention over the new prefix: the node attends to the old prefix plus
    its root-to-node chain, exactly the rows the compaction lines up at
    [L, L + n).  Pins the gather against the attention definition."""
    g = W.rng(700 + seed)
    B, N, Hq, Hkv, D = 2, 12, 4, 2, 16
    L = [5, 9]
    S = max(L) + N + 3
    parent = np.stack([W.uniform_parents(g, N) for _ in range(B)]).astype(np.int32)
    q = W.normal(g, (B, N, Hq, D))
    k = W.normal(g, (B, Hkv, S, D))
    v = W.normal(g, (B, Hkv, S, D))
    leaves = [int(g.integers(0, N)) for _ in range(B)]
    paths = [_accepted_chain(parent[b], leaves[b]) for b in range(B)]
    width = max(len(p) for p in paths) + 2
    path = np.full((B, width), -7, np.int32)
    n_path = np.array([len(p) for p in paths], np.int32)
    for b in range(B):
        path[b, :len(paths[b])] = paths[b]
    before = tree_verify_attention(q, k, v, parent, np.array(L), 0.3)
    k2, v2, new_len, err = kv_compact(k, v, np.array(L), path, n_path)
    assert err == 0 and list(new_len) == [L[b] + n_path[b] for b in range(B)]
    for b in range(B):
        n = int(n_path[b])
        chain = np.arange(-1, n - 1, dtype=np.int32)[None]      # 0 <- 1 <- ... <- n-1
        qb = q[b:b + 1, leaves[b]:leaves[b] + 1]
        qq = np.zeros((1, n, Hq, D))
        qq[0, n - 1] = qb[0, 0]
        after = tree_verify_attention(qq, k2[b:b + 1], v2[b:b + 1], chain, np.array([L[b]]), 0.3)
        assert np.allclose(after[0, n - 1], before[b, leaves[b]], rtol=1e-12, atol=1e-12)


def test_kv_compact_identity_and_errors():
    g = W.rng(710)
    B, Hkv, S, D = 3, 2, 20, 4
    k = W.normal(g, (B, Hkv, S, D))
    v = W.normal(g, (B, Hkv, S, D))
    L = np.array([4, 6, 2])
    path = np.array([[0, 1, 2, 3], [0, 2, 1, 5], [0, 3, 9, 18]], np.int32)
    n = np.array([4, 3, 4], np.int32)
    k2, v2, new_len, err = kv_compact(k, v, L, path, n)
    assert np.array_equal(k2[0], k[0]) and new_len[0] == 8          # identity chain
    assert np.array_equal(k2[1], k[1]) and new_len[1] == 6          # not increasing
    assert np.array_equal(k2[2], k[2]) and new_len[2] == 2          # 2 + 18 >= 20
    assert err == 16
    _, _, nl, e0 = kv_compact(k, v, L, path, np.zeros(3, np.int32))
    assert e0 == 0 and list(nl) == list(L)


def test_self_parent_reads_as_root_child():
    """parent[i] == i (a node its own parent) is outside [-1, i-1] too."""
    assert list(sanitize_parent(np.array([0, 1, 1, 3]))) == [-1, -1, 1, -1]


@pytest.mark.parametrize("fast", [False, True])
def test_widely_spread_scores_keep_the_dominant_value(fast):
    """Scores 2000 apart: the softmax is one-hot on the larger (closed form),
    which only a max-shifted exponent computes without overflow."""
    D = 4
    q = np.zeros((1, 1, 1, D)); q[0, 0, 0, 0] = 1.0
    k = np.zeros((1, 1, 3, D)); k[0, 0, 1, 0] = 2000.0        # prefix key 1 dominates
    v = np.arange(12, dtype=np.float64).reshape(1, 1, 3, D)
    f = tree_verify_attention_fast if fast else tree_verify_attention
    out = f(q, k, v, np.array([[-1]]), np.array([2]), 1.0)
    assert np.array_equal(out[0, 0, 0], v[0, 0, 1])


def test_kv_compact_edges():
    """The input is left as it was; an empty prefix is valid; a chain that
    repeats or decreases a slot, or is longer than the path array, is not."""
    g = W.rng(711)
    B, Hkv, S, D = 1, 1, 8, 2
    k = W.normal(g, (B, Hkv, S, D)); v = W.normal(g, (B, Hkv, S, D))
    k0, v0 = k.copy(), v.copy()
    k2, v2, nl, err = kv_compact(k, v, np.array([0]), np.array([[0, 2, 5]], np.int32),
                                 np.array([3], np.int32))
    assert err == 0 and int(nl[0]) == 3
    assert np.array_equal(k, k0) and np.array_equal(v, v0)
    assert np.array_equal(k2[0, 0, :3], k0[0, 0, [0, 2, 5]])
    assert np.array_equal(k2[0, 0, 3:], k0[0, 0, 3:])
    for path, n in [([1, 1, 4], 3), ([2, 1, 4], 3), ([0, 1, 2], 4)]:
        k3, _, nl3, e3 = kv_compact(k, v, np.array([2]), np.array([path], np.int32),
                                    np.array([n], np.int32))
        assert e3 == 16 and int(nl3[0]) == 2 and np.array_equal(k3, k0)
