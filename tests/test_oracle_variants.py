"""Pins for the oracle's middle-step variants (Sec. 5.3 ablations: w/o EG,
w/o ND; a duplicate-sibling filter) and the target arg-max (App. E,
temperature 0).  CPU only.

What fixes them:
  * w/o ND vs TreeGraft (App. G): a branch the target accepts survives a
    non-destructive graft and is lost when the graft overwrites it;
  * overwrite removes exactly the nodes with a strict ancestor in F (checked
    by walking each node's root path), keeps the others in order;
  * w/o EG never grafts at a historical position (Sec. 5.3 reports 0% for
    it); when N_k equals the unvisited set it is the paper's method;
  * dedup never adds a child whose token an existing sibling carries, and
    skips exactly those (brute force over siblings);
  * arg-max: first maximum, NaN read as -inf (brute force).
"""
import math

import numpy as np

import workloads as W
from oracle import tree as T
from oracle.attention import path_of

F32 = np.float32


def _hand_tree(cap, nodes, root_visited=1):
    """nodes: list of (parent, token, visited); logp/cum left 0 (rescored)."""
    t = T.Tree.empty(1, cap)
    for i, (p, tok, vis) in enumerate(nodes):
        t.parent[0, i] = p
        t.token[0, i] = tok
        t.depth[0, i] = 1 if p < 0 else int(t.depth[0, p]) + 1
        t.visited[0, i] = vis
    t.n_nodes[0] = len(nodes)
    t.root_visited[0] = root_visited
    return t


def _rows(R, V, spec):
    """Logits rows: spec {row: {token: logit}}, everything else -20."""
    x = np.full((1, R, V), -20.0, np.float32)
    for r, d in spec.items():
        for tok, val in d.items():
            x[0, r, tok] = val
    return x


def _greedy_by_rule(t, rule):
    """greedy[0, i+1] = rule(token path of node i); greedy[0, 0] = rule(())."""
    n = int(t.n_nodes[0])
    par = t.parent[0, :n].astype(np.int64)
    g = np.zeros((1, t.cap + 1), np.int32)
    g[0, 0] = rule(())
    for i in range(n):
        toks = tuple(int(t.token[0, u]) for u in path_of(par, i))
        g[0, i + 1] = rule(toks)
    return g


# -------------------------------------------------------------- w/o ND

def test_overwrite_loses_the_accepted_branch_that_nd_keeps():
    """App. G in miniature: the middle step grafts at a historical node whose
    existing subtree holds the continuation the target accepts."""
    V, cap = 8, 32
    #      root -> 0(tok 1) -> 1(tok 2) -> 2(tok 3);  root -> 3(tok 4)
    t = _hand_tree(cap, [(-1, 1, 0), (0, 2, 0), (1, 3, 0), (-1, 4, 0)])
    strong = _rows(5, V, {0: {1: 5.0, 4: 1.0},      # root row: node 0 ranks first
                          1: {5: 4.0, 6: 3.0, 2: 0.0},  # node 0's row: new tokens 5, 6
                          2: {3: 4.0}, 3: {7: 4.0}, 4: {0: 4.0}})
    rule = {(): 1, (1,): 2, (1, 2): 3, (1, 2, 3): 7}
    target = lambda toks: rule.get(toks, 0)
    out = {}
    for flags in (0, T.GRAFT_OVERWRITE):
        t2, _, fr, ng, err = T.rescore_graft(t, strong, W=1, M=2, flags=flags)
        assert err == 0 and int(ng[0]) == 1
        g = _greedy_by_rule(t2, target)
        A, path, bonus, err = T.accept(t2.parent, t2.token, t2.n_nodes, g, 8)
        assert err == 0
        out[flags] = (t2, fr, int(A[0]), path[0])
    t_nd, fr_nd, A_nd, _ = out[0]
    t_ow, fr_ow, A_ow, _ = out[T.GRAFT_OVERWRITE]
    assert fr_nd[0, 0] == 0 and fr_ow[0, 0] == 0          # the historical node 0
    assert A_nd == 3                                     # 1, 2, 3 accepted
    assert A_ow == 1                                     # subtree 1 -> 2 is gone
    assert int(t_nd.n_nodes[0]) == 6 and int(t_ow.n_nodes[0]) == 4
    assert list(t_ow.token[0, :4]) == [1, 4, 5, 6]
    assert list(t_ow.parent[0, :4]) == [-1, -1, 0, 0]


def _grown_tree(seed, V=50, steps=3, width=3, K=3, cap=256):
    t = T.Tree.empty(1, cap)
    fr = np.full((1, 1), -1, np.int32)
    nf = np.ones(1, np.int32)
    for s in range(steps):
        lg = W.normal(W.rng([seed, s]), (1, fr.shape[1], V), 2.0)
        t, _, fr, nf, err = T.expand(t, lg, fr, nf, K, width)
        assert err == 0
    return t


def test_overwrite_removes_exactly_the_strict_descendants_of_f():
    for seed in range(6):
        t = _grown_tree(700 + seed)
        n = int(t.n_nodes[0])
        strong = W.normal(W.rng([710, seed]), (1, n + 1, 50), 3.0)
        Wsel, M = 3 + seed % 3, 2
        ref, _, fr_nd, ng_nd, _ = T.rescore_graft(t, strong, Wsel, M)
        t2, _, fr, ng, err = T.rescore_graft(t, strong, Wsel, M, flags=T.GRAFT_OVERWRITE)
        assert err == 0
        F_old = [int(v) for v in fr_nd[0, :int(ng_nd[0])]]   # same reselection
        par = t.parent[0, :n].astype(np.int64)
        dead = [any(a in F_old for a in path_of(par, u)[:-1]) or
                (-1 in F_old) for u in range(n)]
        keep = [u for u in range(n) if not dead[u]]
        n2 = len(keep)
        assert int(t2.n_nodes[0]) == n2 + M * len([v for v in F_old if v < 0 or not dead[v]])
        newid = {u: i for i, u in enumerate(keep)}
        for i, u in enumerate(keep):
            p = int(t.parent[0, u])
            assert int(t2.parent[0, i]) == (-1 if p < 0 else newid[p])
            assert int(t2.token[0, i]) == int(t.token[0, u])
            assert int(t2.depth[0, i]) == int(t.depth[0, u])
            assert t2.cum[0, i].view(np.uint32) == ref.cum[0, u].view(np.uint32)
        surv = [v for v in F_old if v < 0 or not dead[v]]
        assert [int(x) for x in fr[0, :int(ng[0])]] == [(-1 if v < 0 else newid[v]) for v in surv]
        for c in range(n2, int(t2.n_nodes[0])):
            assert int(t2.parent[0, c]) in [(-1 if v < 0 else newid[v]) for v in surv]
            assert int(t2.parent[0, c]) < c
        assert (t2.visited[0, :n2] == 1).all() and (t2.visited[0, n2:int(t2.n_nodes[0])] == 0).all()


def test_overwrite_at_the_root_leaves_only_the_new_children():
    t = _hand_tree(16, [(-1, 1, 0), (0, 2, 0)], root_visited=0)
    strong = _rows(3, 6, {0: {3: 9.0, 4: 8.0}, 1: {5: 1.0}, 2: {5: 1.0}})
    t2, _, fr, ng, err = T.rescore_graft(t, strong, W=1, M=2, flags=T.GRAFT_OVERWRITE)
    assert err == 0 and list(fr[0, :1]) == [-1]
    assert int(t2.n_nodes[0]) == 2
    assert list(t2.parent[0, :2]) == [-1, -1] and list(t2.token[0, :2]) == [3, 4]


# -------------------------------------------------------------- w/o EG

def test_newonly_equals_the_paper_pool_when_n_k_is_the_unvisited_set():
    """Two middle steps in a row: the second one's unvisited nodes are exactly
    the first one's grafts (N_k), so both pools coincide."""
    V = 40
    t = T.Tree.empty(1, 128)
    s1 = W.normal(W.rng(720), (1, 1, V), 3.0)
    t1, *_ = T.rescore_graft(t, s1, W=1, M=4)
    n1 = int(t1.n_nodes[0])
    s2 = W.normal(W.rng(721), (1, n1 + 1, V), 3.0)
    a = T.rescore_graft(t1, s2, W=3, M=3, N=5)
    b = T.rescore_graft(t1, s2, W=3, M=3, N=5, flags=T.POOL_NEWONLY,
                        new_from=np.array([0], np.int32))
    for x, y in zip(a[1:], b[1:]):
        np.testing.assert_array_equal(np.asarray(x), np.asarray(y))
    for f in ("parent", "token", "depth", "visited"):
        np.testing.assert_array_equal(getattr(a[0], f), getattr(b[0], f))
    # first step: N_1 = {root}, the same pool too
    c = T.rescore_graft(t, s1, W=1, M=4, flags=T.POOL_NEWONLY,
                        new_from=np.array([-1], np.int32))
    np.testing.assert_array_equal(c[0].token, t1.token)


def test_newonly_never_grafts_at_a_historical_position():
    hist = 0
    for seed in range(8):
        t = _grown_tree(730 + seed, steps=2)
        n_before = int(t.n_nodes[0])
        # one more small step makes N_k = ids >= n_before
        fr = np.arange(min(3, n_before), dtype=np.int32)[None, :]
        lg = W.normal(W.rng([731, seed]), (1, fr.shape[1], 50), 2.0)
        t, _, _, _, err = T.expand(t, lg, fr, np.array([fr.shape[1]], np.int32), 3, 3)
        n = int(t.n_nodes[0])
        strong = W.normal(W.rng([732, seed]), (1, n + 1, 50), 3.0)
        _, _, fr_p, ng_p, _ = T.rescore_graft(t, strong, 4, 2)
        t2, _, fr_e, ng_e, err = T.rescore_graft(t, strong, 4, 2, flags=T.POOL_NEWONLY,
                                                 new_from=np.array([n_before], np.int32))
        assert err == 0
        assert all(int(v) >= n_before for v in fr_e[0, :int(ng_e[0])])
        hist += sum(int(v) < n_before for v in fr_p[0, :int(ng_p[0])])
        # visited: only the pool (N_k) joins P, older unvisited nodes stay unvisited
        assert (t2.visited[0, n_before:n] == 1).all()
        np.testing.assert_array_equal(t2.visited[0, :n_before], t.visited[0, :n_before])
    assert hist > 0   # the paper's pool does pick historical positions here


# ---------------------------------------------------------------- dedup

def test_dedup_skips_the_token_an_existing_sibling_has():
    t = _hand_tree(16, [(-1, 5, 1), (-1, 2, 1)], root_visited=0)
    strong = _rows(3, 8, {0: {5: 9.0, 6: 8.0, 2: 7.0}, 1: {1: 1.0}, 2: {1: 1.0}})
    t_nd, *_ = T.rescore_graft(t, strong, W=1, M=3)
    t_dd, _, fr, ng, err = T.rescore_graft(t, strong, W=1, M=3, flags=T.GRAFT_DEDUP)
    assert err == 0 and list(fr[0, :1]) == [-1]
    assert int(t_nd.n_nodes[0]) == 5 and list(t_nd.token[0, 2:5]) == [5, 6, 2]
    assert int(t_dd.n_nodes[0]) == 3 and list(t_dd.token[0, 2:3]) == [6]
    assert t_dd.cum[0, 2] == t_nd.cum[0, 3]


def test_dedup_counts_match_brute_force():
    for seed in range(6):
        t = _grown_tree(740 + seed, V=6, K=3)   # small vocab: many repeats
        n = int(t.n_nodes[0])
        strong = W.normal(W.rng([741, seed]), (1, n + 1, 6), 3.0)
        _, _, fr, ng, _ = T.rescore_graft(t, strong, 4, 3)
        t2, _, fr2, ng2, err = T.rescore_graft(t, strong, 4, 3, flags=T.GRAFT_DEDUP)
        assert err == 0 and np.array_equal(fr, fr2)
        expect = 0
        for v in fr[0, :int(ng[0])]:
            v = int(v)
            sib = {int(t.token[0, u]) for u in range(n) if int(t.parent[0, u]) == v}
            toks, _ = T.row_topk(strong[0, v + 1], 3)
            expect += sum(int(x) not in sib for x in toks)
        assert int(t2.n_nodes[0]) == n + expect
        for c in range(n, int(t2.n_nodes[0])):
            p = int(t2.parent[0, c])
            old_sibs = {int(t.token[0, u]) for u in range(n) if int(t.parent[0, u]) == p}
            assert int(t2.token[0, c]) not in old_sibs


# -------------------------------------------------------------- arg-max

def test_greedy_argmax_brute_force_ties_nan_and_padding():
    g = W.rng(750)
    x = np.round(W.normal(g, (2, 6, 9), 1.0)).astype(np.float32)  # many ties
    x[0, 1, 3] = np.nan
    x[1, 2, :] = -np.inf
    x[1, 3, 0] = np.inf                      # +inf reads as -inf
    n_nodes = np.array([5, 3], np.int32)
    got, err = T.greedy_argmax(x, n_nodes)
    assert err == T.DERR_NONFINITE
    for b in range(2):
        for r in range(6):
            if r > n_nodes[b]:
                assert got[b, r] == -1
                continue
            vals = [(-math.inf if (math.isnan(v) or v == math.inf) else v) for v in x[b, r]]
            best = max(vals)
            assert got[b, r] == vals.index(best)
