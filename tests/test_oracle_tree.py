"""Pins for the draft-tree oracle (CPU only).

The oracle is checked against hand-derived closed-form cases (tests/golden),
library routines (scipy's logsumexp / log_softmax), brute force over tiny
inputs (full enumeration of orders, paths and subsets) and invariants that the
paper's definitions fix (Sec. 3.1 score, Sec. 3.2 pool and visited rule,
Alg. 2 non-destructive attach, Alg. 3 prune, temperature-0 acceptance).
"""
import itertools
import json
import math
import os

import numpy as np
import pytest
from scipy.special import log_softmax, logsumexp

import workloads as W
from oracle import tree as T
from oracle.attention import path_of

GOLD = os.path.join(os.path.dirname(__file__), "golden")
F32 = np.float32


def _gold(name):
    with open(os.path.join(GOLD, name)) as f:
        return json.load(f)


def _row(weights):
    """Natural-log logits of integer weights; '-' is a -inf logit."""
    return np.array([-np.inf if w == "-" else math.log(w) for w in weights],
                    dtype=np.float32)


# ------------------------------------------------------------- logits rows

def test_lse_matches_scipy_within_one_ulp():
    g = W.rng(1)
    for std in (0.1, 2.0, 3.0, 30.0):
        x = W.normal(g, (5000,), std)
        want = F32(logsumexp(x.astype(np.float64)))
        got = T.row_lse(x)
        assert abs(float(got) - float(want)) <= abs(float(np.spacing(want)))


def test_lse_closed_form_and_special_rows():
    assert abs(float(T.row_lse(_row([1, 2, 3, 4]))) - math.log(10)) < 1e-6
    assert T.row_lse(_row([1, "-", "-"])) == F32(0.0)
    assert T.row_lse(_row(["-", "-"])) == T.NEG_INF
    x = np.array([0.0, np.nan, np.inf, 0.0], np.float32)     # NaN/+inf -> -inf
    assert abs(float(T.row_lse(x)) - math.log(2)) < 1e-7
    assert T.clean_logits(x)[1] is True


def _topk_bruteforce(x, k):
    xs = [(-np.inf if (np.isnan(v) or v == np.inf) else float(v)) for v in x]
    order = sorted(range(len(xs)), key=lambda t: (-xs[t], t))
    return order[:k]


@pytest.mark.parametrize("seed", range(8))
def test_topk_matches_python_sort_with_ties(seed):
    g = W.rng(10 + seed)
    V = int(g.integers(5, 300))
    x = g.integers(-4, 4, size=V).astype(np.float32)          # many exact ties
    x[g.integers(0, V, size=3)] = -0.0
    x[g.integers(0, V, size=2)] = -np.inf
    if seed % 2:
        x[g.integers(0, V)] = np.nan
    k = int(g.integers(1, min(V, 64) + 1))
    toks, vals = T.row_topk(x, k)
    assert list(toks) == _topk_bruteforce(x, k)
    xc, _ = T.clean_logits(x)
    assert np.array_equal(vals, xc[toks])


def test_negative_zero_ranks_equal_to_zero():
    x = np.array([-0.0, 0.0, -1.0], np.float32)
    assert list(T.row_topk(x, 2)[0]) == [0, 1]
    x = np.array([0.0, -0.0, -1.0], np.float32)
    assert list(T.row_topk(x, 2)[0]) == [0, 1]


# ------------------------------------------------------------------ expand

def _run_gold_expand(case):
    tree = T.Tree.empty(1, case["cap"])
    for step in case["steps"]:
        rows = np.stack([_row(w) for w in step["weights"]])[None]
        fr = np.array([step["frontier"]], np.int32)
        n0 = int(tree.n_nodes[0])
        tree, lse, nxt, nn, err = T.expand(tree, rows, fr, None, step["K"], step["N"])
        e = step["expect"]
        assert err == 0
        new = slice(n0, int(tree.n_nodes[0]))
        assert list(tree.parent[0, new]) == e["parent"]
        assert list(tree.token[0, new]) == e["token"]
        assert list(tree.depth[0, new]) == e["depth"]
        np.testing.assert_allclose(np.exp(tree.cum[0, new].astype(np.float64)),
                                   e["prob"], rtol=2e-6)
        np.testing.assert_allclose(np.exp(lse[0].astype(np.float64)), e["lse"], rtol=2e-6)
        assert int(nn[0]) == e["n_next"]
        assert list(nxt[0, :e["n_next"]]) == e["next_frontier"]
        assert all(v == T.NO_NODE for v in nxt[0, e["n_next"]:])


@pytest.mark.parametrize("idx", [0, 1])
def test_expand_golden(idx):
    _run_gold_expand(_gold("expand_closed_form.json")["cases"][idx])


def _scored_tree(seed, B, V, steps, W_, K, std=2.0, cap=4096):
    """Tree built from the root by repeated expansion; rows drawn per node."""
    tree = T.Tree.empty(B, cap)
    fr = np.full((B, 1), -1, np.int32)
    nf = np.ones(B, np.int32)
    for _ in range(steps):
        F = fr.shape[1]
        rows = np.stack([np.stack([W.node_logits(seed, b * 100000 + max(int(v), -1) + 1, V, std)
                                   for v in fr[b]]) for b in range(B)])
        tree, _, nxt, nn, err = T.expand(tree, rows, fr, nf, K, W_)
        assert err == 0
        fr, nf = nxt, nn
    return tree


def test_expand_scores_equal_path_sums_and_log_softmax():
    """cum(v) recomputed by summing logp along the enumerated root path (fp32,
    root first) equals the incrementally stored cum; logp equals scipy's
    log_softmax at the token within one fp32 rounding."""
    B, V = 2, 50
    tree = _scored_tree(3, B, V, steps=4, W_=3, K=3)
    for b in range(B):
        n = int(tree.n_nodes[b])
        for v in range(n):
            acc = F32(0.0)
            for u in path_of(tree.parent[b], v):
                acc = F32(acc + tree.logp[b, u])
            assert acc == tree.cum[b, v]
            p = int(tree.parent[b, v])
            x = W.node_logits(3, b * 100000 + p + 1, V, 2.0)
            want = log_softmax(x.astype(np.float64))[tree.token[b, v]]
            assert abs(float(tree.logp[b, v]) - want) <= _logp_bound(x, want)
            assert tree.depth[b, v] == len(path_of(tree.parent[b], v))
            if p >= 0:
                assert tree.cum[b, v] <= tree.cum[b, p]      # logp <= 0


def _logp_bound(x, want):
    """fl(x - fl(lse)) is off the exact log-softmax by at most half an ulp of
    lse (its rounding) plus half an ulp of the result (the subtraction)."""
    lse = F32(logsumexp(x.astype(np.float64)))
    return 0.5 * abs(float(np.spacing(lse))) + 0.5 * abs(float(np.spacing(F32(want)))) + 1e-12


def _beats(a, b):
    """Explicit comparison form of the ranking (cum desc, depth asc, id asc)."""
    ca, da, ia = a
    cb, db, ib = b
    if ca != cb:
        return ca > cb
    if da != db:
        return da < db
    return ia < ib


@pytest.mark.parametrize("seed", range(5))
def test_expand_next_frontier_by_pairwise_counting(seed):
    """The next frontier equals the N children with the fewest better children,
    counted pair by pair (a different method than the oracle's sort)."""
    g = W.rng(40 + seed)
    B, V, K = 2, 40, int(g.integers(1, 5))
    tree = _scored_tree(50 + seed, B, V, steps=2, W_=4, K=3)
    F = 4
    fr = np.stack([g.choice(int(tree.n_nodes[b]), F, replace=False) for b in range(B)]).astype(np.int32)
    fr[0, 0] = -1
    # quantised logits force exact cum ties across frontier rows
    logits = np.round(W.normal(g, (B, F, V), 2.0) * 2) / 2
    N = int(g.integers(1, F * K + 3))
    n0 = tree.n_nodes.copy()
    t2, lse, nxt, nn, err = T.expand(tree, logits.astype(np.float32), fr, None, K, N)
    assert err == 0
    for b in range(B):
        kids = list(range(int(n0[b]), int(t2.n_nodes[b])))
        assert len(kids) == F * K
        keys = {v: (float(t2.cum[b, v]), int(t2.depth[b, v]), v) for v in kids}
        rank = {v: sum(_beats(keys[u], keys[v]) for u in kids) for v in kids}
        want = sorted(kids, key=lambda v: rank[v])[:min(N, F * K)]
        assert list(nxt[b, :nn[b]]) == want
        # per-row top-K tokens by brute force
        for f in range(F):
            ch = [n0[b] + f * K + j for j in range(K)]
            assert list(t2.token[b, ch]) == _topk_bruteforce(logits[b, f], K)
            assert all(t2.parent[b, c] == fr[b, f] for c in ch)


def test_expand_error_paths():
    tree = T.Tree.empty(2, 8)
    logits = np.zeros((2, 2, 5), np.float32)
    fr = np.array([[-1, 3], [-1, -1]], np.int32)               # node 3 does not exist
    t2, _, _, nn, err = T.expand(tree, logits, fr, None, 2, 4)
    assert err & T.DERR_BAD_NODE and t2.n_nodes[0] == 0 and nn[0] == 0
    assert t2.n_nodes[1] == 4
    fr = np.array([[-1, -1], [-1, -1]], np.int32)
    t3, _, _, nn, err = T.expand(tree, logits, fr, None, 5, 4)   # 10 > cap 8
    assert err & T.DERR_CAPACITY and (t3.n_nodes == 0).all() and (nn == 0).all()
    logits[1, 0, 2] = np.nan
    _, _, _, _, err = T.expand(tree, logits, fr, None, 2, 4)
    assert err & T.DERR_NONFINITE


def test_expand_all_minus_inf_row():
    tree = T.Tree.empty(1, 8)
    logits = np.full((1, 1, 4), -np.inf, np.float32)
    t2, lse, nxt, nn, err = T.expand(tree, logits, np.array([[-1]], np.int32), None, 2, 2)
    assert lse[0, 0] == T.NEG_INF and list(t2.token[0, :2]) == [0, 1]
    assert np.all(t2.logp[0, :2] == T.NEG_INF) and np.all(t2.cum[0, :2] == T.NEG_INF)
    assert list(nxt[0]) == [0, 1]


# --------------------------------------------------------- rescore + graft

def _gold_tree(spec, cap):
    n = len(spec["parent"])
    t = T.Tree.empty(1, cap)
    t.parent[0, :n] = spec["parent"]
    t.token[0, :n] = spec["token"]
    t.depth[0, :n] = spec["depth"]
    t.visited[0, :n] = spec["visited"]
    t.root_visited[0] = spec["root_visited"]
    t.n_nodes[0] = n
    t.logp[0, :n] = -5.0        # weak scores: all overwritten by the first call
    t.cum[0, :n] = -9.0
    return t


def test_rescore_graft_golden():
    gd = _gold("rescore_graft_closed_form.json")
    t = _gold_tree(gd["initial_tree"], gd["cap"])
    rows = np.stack([_row(w) for w in gd["rows"]])[None]
    for call in gd["calls"]:
        e = call["expect"]
        n0 = int(t.n_nodes[0])
        old = (t.parent[0, :n0].copy(), t.token[0, :n0].copy(), t.depth[0, :n0].copy())
        t, lse, fr, ng, err, nx, nn = T.rescore_graft(t, rows, call["W"], call["M"],
                                                      N=call["N"])
        assert err == 0
        assert list(nx[0, :nn[0]]) == e["next_frontier"]
        assert all(v == T.NO_NODE for v in nx[0, nn[0]:])
        np.testing.assert_allclose(np.exp(t.cum[0, :n0].astype(np.float64)),
                                   e["prob_existing"], rtol=3e-6)
        assert int(ng[0]) == e["n_graft"]
        assert list(fr[0, :ng[0]]) == e["graft_frontier"]
        assert all(v == T.NO_NODE for v in fr[0, ng[0]:])
        new = slice(n0, int(t.n_nodes[0]))
        assert int(t.n_nodes[0]) == e["n_nodes"]
        assert list(t.parent[0, new]) == e["new_parent"]
        assert list(t.token[0, new]) == e["new_token"]
        assert list(t.depth[0, new]) == e["new_depth"]
        np.testing.assert_allclose(np.exp(t.cum[0, new].astype(np.float64)),
                                   e["new_prob"], rtol=3e-6)
        assert list(t.visited[0, :e["n_nodes"]]) == e["visited"]
        assert int(t.root_visited[0]) == e["root_visited"]
        got_rows = [r for r in range(rows.shape[1]) if not np.isnan(lse[0, r])]
        assert got_rows == e["lse_rows"]
        np.testing.assert_allclose(np.exp(lse[0, got_rows].astype(np.float64)),
                                   e["lse"], rtol=2e-6)
        # existing nodes keep parent, token and depth (non-destructive)
        assert np.array_equal(t.parent[0, :n0], old[0])
        assert np.array_equal(t.token[0, :n0], old[1])
        assert np.array_equal(t.depth[0, :n0], old[2])


def _rows_for_tree(seed, tree, b, V, std):
    """Row 0 = root, row 1+i = node i, from the same per-node stream the
    scored-tree builder used (index b*100000 + node + 1)."""
    n = int(tree.n_nodes[b])
    return np.stack([W.node_logits(seed, b * 100000 + r, V, std) for r in range(n + 1)])


def test_rescore_with_identical_drafter_is_a_noop_on_scores():
    """rho = 1: rescoring with the very logits that created the tree reproduces
    every stored logp and cum bit for bit (checks the parent-row/token gather)."""
    B, V = 2, 60
    tree = _scored_tree(7, B, V, steps=3, W_=3, K=3)
    R = int(tree.n_nodes.max()) + 1
    rows = np.full((B, R, V), -np.inf, np.float32)
    for b in range(B):
        rr = _rows_for_tree(7, tree, b, V, 2.0)
        rows[b, :len(rr)] = rr
    t2, _, _, _, err = T.rescore_graft(tree, rows, 4, 2)
    assert err == 0
    for b in range(B):
        n = int(tree.n_nodes[b])
        assert np.array_equal(t2.logp[b, :n], tree.logp[b, :n])
        assert np.array_equal(t2.cum[b, :n], tree.cum[b, :n])


def test_rescore_all_visited_is_noop():
    tree = _scored_tree(8, 1, 30, steps=2, W_=2, K=2)
    tree.visited[0, :] = 1
    tree.root_visited[0] = 1
    rows = W.normal(W.rng(1), (1, int(tree.n_nodes[0]) + 1, 30), 3.0)
    t2, lse, fr, ng, err = T.rescore_graft(tree, rows, 5, 3)
    assert err == 0 and ng[0] == 0 and np.all(np.isnan(lse))
    for f in ("parent", "token", "depth", "logp", "cum", "visited", "n_nodes"):
        assert np.array_equal(getattr(t2, f), getattr(tree, f))
    assert all(v == T.NO_NODE for v in fr[0])


@pytest.mark.parametrize("seed", range(6))
def test_rescore_graft_invariants(seed):
    g = W.rng(60 + seed)
    B, V = 2, 40
    tree = _scored_tree(70 + seed, B, V, steps=3, W_=3, K=3)
    # mark a random ancestor-closed subset as visited (what earlier middle steps leave)
    for b in range(B):
        n = int(tree.n_nodes[b])
        for v in range(n):
            p = int(tree.parent[b, v])
            par_vis = bool(tree.root_visited[b]) if p < 0 else bool(tree.visited[b, p])
            if par_vis or (p < 0 and g.random() < 0.5):
                tree.root_visited[b] = 1
                tree.visited[b, v] = int(g.random() < 0.5)
    R = int(tree.n_nodes.max()) + 1
    strong = W.normal(g, (B, R, V), 3.0)
    Wsel, M = int(g.integers(1, 8)), int(g.integers(1, 4))
    before = tree.copy()
    Nn = int(g.integers(1, 20))
    t2, lse, fr, ng, err, nx, nn = T.rescore_graft(tree, strong, Wsel, M, N=Nn)
    assert err == 0
    for b in range(B):
        n = int(before.n_nodes[b])
        C = [v for v in range(n) if not before.visited[b, v]]
        C_all = ([-1] if not before.root_visited[b] else []) + C
        assert T.pool_of(before, b) == C_all
        assert ng[b] == min(Wsel, len(C_all))
        assert t2.n_nodes[b] == n + ng[b] * M
        # preservation: existing structure untouched; scores outside C untouched
        for f in ("parent", "token", "depth"):
            assert np.array_equal(getattr(t2, f)[b, :n], getattr(before, f)[b, :n])
        out = [v for v in range(n) if before.visited[b, v]]
        assert np.array_equal(t2.cum[b, out], before.cum[b, out])
        # visited' = visited u C; new nodes unvisited
        assert np.all(t2.visited[b, :n] == 1) and np.all(t2.visited[b, n:t2.n_nodes[b]] == 0)
        assert t2.root_visited[b] == 1
        # rescored cum = fp32 sum of the new logp along the path
        for v in C:
            acc = F32(0.0)
            for u in path_of(t2.parent[b], v):
                acc = F32(acc + t2.logp[b, u])
            assert acc == t2.cum[b, v]
            p = int(before.parent[b, v])
            want = log_softmax(strong[b, p + 1].astype(np.float64))[before.token[b, v]]
            assert abs(float(t2.logp[b, v]) - want) <= _logp_bound(strong[b, p + 1], want)
        # frontier = best |F| of C by pairwise counting; closed under parent-in-C
        keys = {v: (0.0 if v < 0 else float(t2.cum[b, v]),
                    0 if v < 0 else int(t2.depth[b, v]), v) for v in C_all}
        rank = {v: sum(_beats(keys[u], keys[v]) for u in C_all) for v in C_all}
        want = sorted(C_all, key=lambda v: rank[v])[:ng[b]]
        assert list(fr[b, :ng[b]]) == want
        Fs = set(want)
        for v in want:
            p = -1 if v < 0 else int(before.parent[b, v])
            if v >= 0 and p in set(C_all):
                assert p in Fs
        # next frontier: best Nn grafted children, by pairwise counting
        kids = list(range(n, int(t2.n_nodes[b])))
        kk = {v: (float(t2.cum[b, v]), int(t2.depth[b, v]), v) for v in kids}
        krank = {v: sum(_beats(kk[u], kk[v]) for u in kids) for v in kids}
        assert list(nx[b, :nn[b]]) == sorted(kids, key=lambda v: krank[v])[:Nn]
        # grafted children: rank-j token of the frontier node's own row
        for f, v in enumerate(want):
            toks = _topk_bruteforce(strong[b, v + 1], M)
            for j in range(M):
                c = n + f * M + j
                assert t2.parent[b, c] == v and t2.token[b, c] == toks[j]
                d = 0 if v < 0 else int(t2.depth[b, v])
                assert t2.depth[b, c] == d + 1


def test_rescore_capacity_and_rows_errors():
    tree = _scored_tree(9, 1, 20, steps=1, W_=2, K=2)   # 2 nodes
    rows = W.normal(W.rng(2), (1, 3, 20), 1.0)
    small = tree.copy()
    small.cap = 3
    t2, _, _, ng, err = T.rescore_graft(small, rows, 3, 1)   # 2 + 3*1 > 3
    assert err & T.DERR_CAPACITY and ng[0] == 0
    assert np.array_equal(t2.cum, small.cum) and np.array_equal(t2.visited, small.visited)
    _, _, _, ng, err = T.rescore_graft(tree, rows[:, :2], 3, 1)  # R < n + 1
    assert err & T.DERR_BAD_NODE and ng[0] == 0


# ------------------------------------------------------------------ accept

def test_accept_golden_nd_vs_overwrite():
    gd = _gold("accept_nd_example.json")
    for key in ("nd", "overwrite"):
        c = gd[key]
        par = np.array([c["parent"]], np.int32)
        tok = np.array([c["token"]], np.int32)
        A, path, bonus, err = T.accept(par, tok, np.array([len(c["parent"])]),
                                       np.array([c["greedy"]], np.int32), c["max_depth"])
        assert err == 0
        assert A[0] == c["expect"]["A"]
        assert list(path[0]) == c["expect"]["path"]
        assert bonus[0] == c["expect"]["bonus"]


def test_accept_chain_all_match_and_no_match():
    n = 7
    par = np.arange(-1, n - 1, dtype=np.int32)[None]
    tok = np.arange(100, 100 + n, dtype=np.int32)[None]
    greedy = np.concatenate([tok[0], [5]]).astype(np.int32)[None]
    A, path, bonus, _ = T.accept(par, tok, np.array([n]), greedy, n)
    assert A[0] == n and list(path[0]) == list(range(n)) and bonus[0] == 5
    greedy2 = np.full((1, n + 1), 3, np.int32)
    A, path, bonus, _ = T.accept(par, tok, np.array([n]), greedy2, n)
    assert A[0] == 0 and np.all(path[0] == -1) and bonus[0] == 3
    # max_depth below the matching depth: deeper nodes are not considered
    A, path, bonus, err = T.accept(par, tok, np.array([n]), greedy, 3)
    assert A[0] == 3 and list(path[0]) == [0, 1, 2] and bonus[0] == greedy[0, 3]
    assert err & T.DERR_CAPACITY


def test_accept_duplicate_siblings_prefers_deeper_then_smaller_id():
    # nodes 0 and 1 are siblings with the same token; only node 1 has a matching child
    par = np.array([[-1, -1, 1, 0]], np.int32)
    tok = np.array([[5, 5, 6, 9]], np.int32)
    greedy = np.array([[5, 6, 6, 1, 0]], np.int32)
    A, path, bonus, _ = T.accept(par, tok, np.array([4]), greedy, 4)
    assert A[0] == 2 and list(path[0][:2]) == [1, 2] and bonus[0] == greedy[0, 3]
    greedy = np.array([[5, 7, 7, 1, 0]], np.int32)           # neither has a matching child
    A, path, bonus, _ = T.accept(par, tok, np.array([4]), greedy, 4)
    assert A[0] == 1 and path[0][0] == 0 and bonus[0] == 7


def _toy_target(seq):
    """Deterministic toy target: next token = a hash of the whole prefix."""
    h = 2166136261
    for t in seq:
        h = ((h ^ int(t)) * 16777619) & 0xFFFFFFFF
    return h % 50


def test_accept_preserves_the_target_greedy_sequence():
    """Distribution preservation at temperature 0 (Sec. 3.2): whatever draft
    tree is proposed, accepted path + bonus token reproduce exactly the
    target's own greedy autoregressive continuation."""
    g = W.rng(77)
    prompt = [1, 2, 3]
    seq = list(prompt)
    while len(seq) < 200:
        n = int(g.integers(1, 30))
        par = W.uniform_parents(g, n)
        tok = g.integers(0, 50, size=n).astype(np.int32)
        # plant the true continuation on a random chain with probability 1/2
        if g.random() < 0.5:
            v, ctx = -1, list(seq)
            for i in range(n):
                if par[i] == v:
                    tok[i] = _toy_target(ctx)
                    ctx.append(int(tok[i]))
                    v = i
        ctxs = []
        for i in range(n):
            ctxs.append(seq + [int(tok[u]) for u in path_of(par, i)])
        greedy = np.array([_toy_target(seq)] + [_toy_target(c) for c in ctxs], np.int32)
        A, path, bonus, err = T.accept(par[None], tok[None], np.array([n]), greedy[None], n)
        assert err == 0
        seq += [int(tok[u]) for u in path[0, :A[0]]] + [int(bonus[0])]
    ref = list(prompt)
    while len(ref) < len(seq):
        ref.append(_toy_target(ref))
    assert seq == ref


def test_accept_bruteforce_over_all_token_assignments():
    """Tiny trees, every binary token assignment: the accepted length equals
    the longest root path along which each token is the target's choice."""
    par = np.array([-1, 0, 0, 1, -1, 4], np.int32)
    greedy = np.array([1, 0, 1, 1, 0, 1, 0], np.int32)
    for bits in itertools.product([0, 1], repeat=len(par)):
        tok = np.array(bits, np.int32)
        A, path, _, _ = T.accept(par[None], tok[None], np.array([6]), greedy[None], 6)
        best = 0
        for v in range(len(par)):
            p = path_of(par, v)
            if all(tok[u] == greedy[par[u] + 1] for u in p):
                best = max(best, len(p))
        assert A[0] == best


def test_accept_bad_parent_flag():
    par = np.array([[-1, 5, 0]], np.int32)
    tok = np.array([[1, 2, 3]], np.int32)
    greedy = np.array([[1, 3, 9, 9]], np.int32)
    A, path, bonus, err = T.accept(par, tok, np.array([3]), greedy, 3)
    assert err & T.DERR_BAD_PARENT
    assert A[0] == 2 and list(path[0][:2]) == [0, 2]


# -------------------------------------------------------------------- prune

@pytest.mark.parametrize("idx", [0, 1, 2])
def test_prune_golden(idx):
    gd = _gold("prune_alg3.json")
    c = gd["cases"][idx]
    par = np.array(gd["parent"], np.int32)
    cum = np.array(gd["cum"], np.float32)
    out = T.global_prune(par, cum, len(par), c["B_ver"])
    assert list(out["kept"]) == c["kept"]
    assert list(out["parent"]) == c["new_parent"]
    assert list(out["position_ids"]) == c["position_ids"]
    assert out["mask"].tolist() == c["mask"]
    assert out["retrieval"].tolist() == c["retrieval"]


@pytest.mark.parametrize("seed", range(5))
def test_prune_closed_form_on_scored_trees(seed):
    """With cum non-increasing along paths (logp <= 0) a parent always ranks
    before its child, so Alg. 3 keeps exactly the root plus the first B_ver
    ranked nodes; the result is ancestor-closed and within budget."""
    tree = _scored_tree(90 + seed, 1, 40, steps=5, W_=4, K=4)
    n = int(tree.n_nodes[0])
    par, cum = tree.parent[0, :n], tree.cum[0, :n]
    depth = tree.depth[0, :n]
    for B_ver in (1, 7, 31, n - 1, n, n + 5):
        out = T.global_prune(par, cum, n, B_ver)
        ranked = sorted(range(n), key=lambda v: (-float(cum[v]), int(depth[v]), v))
        assert set(out["kept"]) == set(ranked[:min(B_ver, n)])
        kept = set(out["kept"])
        assert all(par[v] == -1 or par[v] in kept for v in kept)
        # new order puts parents first; position id = depth
        assert all(p < i for i, p in enumerate(out["parent"]))
        assert list(out["position_ids"][1:]) == [int(depth[v]) for v in out["kept"]]
        # mask = ancestor-or-self closure in the new index (root = 0)
        vp = np.concatenate([[-1], out["parent"] + 1])
        for u in range(len(vp)):
            anc = set()
            w = u
            while w != -1:
                anc.add(w)
                w = vp[w]
            assert set(np.nonzero(out["mask"][u])[0]) == anc


def test_prune_bruteforce_tiny_against_subset_search():
    """For tiny trees, enumerate all subsets: Alg. 3's kept set is the
    lexicographically best ancestor-closed set built greedily in rank order,
    and is always ancestor-closed and of size min(n, B_ver)."""
    g = W.rng(5)
    for _ in range(30):
        n = int(g.integers(1, 7))
        par = W.uniform_parents(g, n)
        cum = (-g.integers(0, 4, size=n)).astype(np.float32)      # ties, non-monotone
        B_ver = int(g.integers(1, n + 1))
        out = T.global_prune(par, cum, n, B_ver)
        kept = set(int(v) for v in out["kept"])
        assert all(par[v] == -1 or par[v] in kept for v in kept)
        assert len(kept) <= B_ver
        # simulate the loop by explicit subset bookkeeping
        depth = W.node_depths(par)
        ranked = sorted(range(n), key=lambda v: (-float(cum[v]), int(depth[v]), v))
        K = set()
        for v in ranked:
            chain = set(path_of(par, v)) - K
            if len(K) + len(chain) <= B_ver:
                K |= chain
            if len(K) == B_ver:
                break
        assert kept == K


def test_expand_frontier_id_equal_to_the_node_count_and_exact_capacity():
    """A frontier id equal to n_b is not a node (BAD_NODE, tree unchanged);
    F*K children that fill the tree exactly are appended."""
    t = T.Tree.empty(1, 6)
    t.parent[0, :2], t.token[0, :2], t.depth[0, :2], t.n_nodes[0] = [-1, 0], [1, 2], [1, 2], 2
    logits = np.zeros((1, 2, 5), np.float32)
    t1, _, _, nn, err = T.expand(t, logits, np.array([[1, 2]], np.int32), None, 2, 4)
    assert err == T.DERR_BAD_NODE and int(nn[0]) == 0 and int(t1.n_nodes[0]) == 2
    t2, _, _, nn, err = T.expand(t, logits, np.array([[0, 1]], np.int32), None, 2, 4)
    assert err == 0 and int(t2.n_nodes[0]) == 6 and list(t2.depth[0, 2:6]) == [2, 2, 3, 3]


def test_greedy_argmax_needs_the_rows_through_n_nodes():
    """Rows 0..n_nodes are read: n_nodes = R - 1 fits, n_nodes = R does not."""
    x = np.zeros((1, 4, 3), np.float32)
    x[0, :, 2] = 1.0
    g, err = T.greedy_argmax(x, np.array([3]))
    assert err == 0 and list(g[0]) == [2, 2, 2, 2]
    g, err = T.greedy_argmax(x, np.array([4]))
    assert err == T.DERR_BAD_NODE and list(g[0]) == [2, 2, 2, 2]
