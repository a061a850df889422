"""GPU parity of tg_tree_expand_topk, tg_tree_rescore_graft and tg_tree_accept.

Float work that decides integers is checked with the split check:
  (i)   each exported row log-sum-exp is within 1e-5 * max(1, |lse|) of the
        oracle's fp64-then-rounded value;
  (ii)  the oracle re-run with the GPU's lse substituted must agree BIT FOR BIT
        on every integer output and on every stored fp32 logp / cum (after
        lse, each is one IEEE fp32 op on identical operands);
  (iii) the free oracle (its own lse) must give the same selections whenever
        the gaps at its selection boundaries exceed twice the largest score
        discrepancy the two lse sets cause.
Acceptance is integer-only and compared bit for bit.
"""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import tree as OT
from tests import _cases as C

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _d(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a))
    return t.to(DEV) if dtype is None else t.to(DEV).to(dtype)


def _lse_close(got, want):
    live = ~np.isnan(want)
    g, w = got[live].astype(np.float64), want[live].astype(np.float64)
    fin = np.isfinite(w)
    assert np.array_equal(np.isfinite(g), fin)
    assert np.all(g[~fin] == w[~fin])
    tol = 1e-5 * np.maximum(1.0, np.abs(w[fin]))
    assert np.all(np.abs(g[fin] - w[fin]) <= tol), float(np.abs(g[fin] - w[fin]).max())


def _boundary_ok(keys, n_sel, delta):
    """True when the first n_sel+1 sorted keys are separated by > 2*delta."""
    c = np.array([k[0] for k in keys[:n_sel + 1]])
    if len(c) < 2:
        return True
    gaps = np.abs(np.diff(c))
    return bool(np.all(gaps > 2 * delta))


# ------------------------------------------------------------------ expand

def run_expand(tg, tree_h, logits, fr, nf, K, N, check_free=True):
    ts = C.tree_to_dev(tg, tree_h)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    lse, nxt, nn = tg.expand_topk(ts, _d(logits), _d(fr, torch.int32),
                                  None if nf is None else _d(nf, torch.int32), K, N, d_err=err)
    torch.cuda.synchronize()
    lse_g, nxt_g, nn_g = lse.cpu().numpy(), nxt.cpu().numpy(), nn.cpu().numpy()
    got = C.tree_from_dev(ts)
    B, F = fr.shape
    nfv = np.full(B, F) if nf is None else np.asarray(nf)
    live = np.zeros((B, F), bool)
    for b in range(B):
        live[b, :nfv[b]] = True
    # (ii) oracle with the GPU's lse
    want, _, nxt_o, nn_o, err_o = OT.expand(tree_h, logits, fr, nf, K, N, lse_override=lse_g)
    C.assert_tree_equal(got, want, "expand")
    assert np.array_equal(nxt_g, nxt_o) and np.array_equal(nn_g, nn_o)
    assert int(err.item()) == err_o
    if check_free:
        # (i) + (iii) against the free oracle
        free, lse_f, nxt_f, nn_f, _ = OT.expand(tree_h, logits, fr, nf, K, N)
        lse_g_live = np.where(live, lse_g, np.nan)
        _lse_close(lse_g_live, lse_f)
        for b in range(B):
            n0, n1 = int(tree_h.n_nodes[b]), int(free.n_nodes[b])
            for f in ("parent", "token", "depth"):
                assert np.array_equal(getattr(free, f)[b, n0:n1], getattr(got, f)[b, n0:n1])
            if n1 == n0:
                continue
            delta = float(np.max(np.abs(free.cum[b, n0:n1].astype(np.float64) -
                                        got.cum[b, n0:n1].astype(np.float64)), initial=0.0))
            keys = sorted(OT.node_key(free.cum[b, v], free.depth[b, v], v) for v in range(n0, n1))
            if _boundary_ok(keys, int(nn_f[b]), delta):
                assert np.array_equal(nxt_f[b], nxt_g[b])
    return got, lse_g, nxt_g, nn_g, int(err.item())


def _tiny_scored_tree():
    """Tiny workload's 16-node tree with scores: node i takes, as its token,
    rank j (its rank among its siblings in id order) of its parent's logits
    row, so siblings are distinct; logp / cum by the oracle's expansion
    arithmetic (Sec. 3.1)."""
    cfg = W.CONFIGS["tiny"]
    g = W.rng(cfg["seed"])
    N, V = cfg["N"], cfg["vocab"]
    parent = W.uniform_parents(g, N)
    rows = W.normal(g, (N + 1, V), cfg["logit_std"])    # row 0 root, 1+i node i
    t = OT.Tree.empty(1, 64)
    kids = W.children_lists(parent)
    for r, ks in enumerate(kids):
        if not ks:
            continue
        toks, vals = OT.row_topk(rows[r], len(ks))
        lse = OT.row_lse(rows[r])
        for j, c in enumerate(ks):
            p = r - 1
            t.parent[0, c] = p
            t.token[0, c] = toks[j]
            t.depth[0, c] = 1 if p < 0 else t.depth[0, p] + 1
            lp = OT.edge_logp(vals[j], lse)
            t.logp[0, c] = lp
            t.cum[0, c] = np.float32((0.0 if p < 0 else t.cum[0, p]) + lp) if p < 0 else \
                np.float32(t.cum[0, p] + lp)
    t.n_nodes[0] = N
    return t, rows, parent


def test_tiny_config_expand(tg):
    """Tiny workload: V=1000, frontier = the 8 best nodes by (cum, depth, id),
    K=4 children each, next frontier N=8."""
    t, rows, _ = _tiny_scored_tree()
    keys = sorted(OT.node_key(t.cum[0, v], t.depth[0, v], v) for v in range(16))
    fr = np.array([[k[2] for k in keys[:8]]], np.int32)
    logits = np.stack([rows[v + 1] for v in fr[0]])[None]
    run_expand(tg, t, logits, fr, None, 4, 8)


CASES = [
    # B, F, V, K, N, note
    (1, 1, 1000, 4, 8, "root only"),
    (2, 8, 1000, 4, 8, "tiny-sized"),
    (3, 5, 4099, 7, 40, "ragged vocab (scalar tail), N > F*K"),
    (2, 16, 2047, 1, 5, "K = 1, odd vocab"),
    (2, 4, 5000, 64, 200, "K = 64 (max)"),
    (1, 3, 64, 64, 17, "K = V"),
    (4, 32, 30000, 10, 60, "many rows"),
    (1, 64, 128256, 10, 60, "one full-vocab tree"),
    (2, 40, 3000, 10, 10, "N = 10 of 400 children (selection)"),
    (1, 205, 700, 5, 60, "F*K = 1025: sorted selection"),
    (2, 256, 600, 8, 300, "F*K = 2048: sorted selection"),
]


@pytest.mark.parametrize("case", CASES, ids=[c[-1] for c in CASES])
def test_expand_shapes(tg, case):
    B, F, V, K, N, _ = case
    g = W.rng(B * 1000 + F * 10 + K)
    base, _ = C.scored_tree(F + V, B, 50, steps=2, width=4, K=4, cap=4096)
    fr = np.stack([g.choice(np.arange(-1, int(base.n_nodes[b])), F, replace=F > int(base.n_nodes[b]) + 1)
                   for b in range(B)]).astype(np.int32)
    nf = np.array([F] + [int(g.integers(0, F + 1)) for _ in range(B - 1)], np.int32)
    logits = W.normal(g, (B, F, V), 3.0)
    run_expand(tg, base, logits, fr, nf, K, N)


@pytest.mark.parametrize("F,K", [(64, 64), (512, 8)])
def test_expand_fills_capacity_with_4096_children(tg, F, K):
    """F*K = 4096 children under the root of an empty tree of capacity 4096
    (the largest tree): the sorted selection path, appending exactly to the
    capacity, with duplicated frontier entries (every row is the root)."""
    g = W.rng(F * 100 + K)
    base = OT.Tree.empty(1, 4096)
    fr = np.full((1, F), -1, np.int32)
    logits = W.normal(g, (1, F, 300), 3.0)
    got, _, _, nn, err = run_expand(tg, base, logits, fr, None, K, 500)
    assert err == 0 and int(got.n_nodes[0]) == 4096 and int(nn[0]) == 500


def test_expand_8192_children_overflow(tg):
    """F*K = 8192 (the documented maximum) can never fit a tree of capacity
    4096: the call reports CAPACITY, appends nothing and returns n_next = 0,
    next to a tree whose 1025 children do fit."""
    g = W.rng(8192)
    base = OT.Tree.empty(2, 4096)
    F, K = 128, 64
    fr = np.full((2, F), -1, np.int32)
    nf = np.array([F, 17], np.int32)             # 17 * 64 = 1088 children fit
    logits = W.normal(g, (2, F, 200), 3.0)
    got, _, _, nn, err = run_expand(tg, base, logits, fr, nf, K, 64)
    assert err & OT.DERR_CAPACITY
    assert int(got.n_nodes[0]) == 0 and int(nn[0]) == 0
    assert int(got.n_nodes[1]) == 17 * 64 and int(nn[1]) == 64


def test_expand_ties_and_special_values(tg):
    """Quantised logits force exact ties in logits and in cum across rows;
    -0.0, -inf entries and an all -inf row exercise the key canonicalisation."""
    g = W.rng(3)
    B, F, V, K, N = 2, 6, 300, 5, 12
    base, _ = C.scored_tree(4, B, 40, steps=2, width=3, K=3)
    fr = np.stack([g.choice(int(base.n_nodes[b]), F, replace=False) for b in range(B)]).astype(np.int32)
    fr[:, 1] = fr[:, 0]              # the same node twice: identical cum, ties by id
    logits = (np.round(W.normal(g, (B, F, V), 1.0) * 2) / 2).astype(np.float32)
    logits[:, 1] = logits[:, 0]
    logits[0, 2, ::7] = -0.0
    logits[0, 3, ::3] = -np.inf
    logits[1, 4] = -np.inf
    run_expand(tg, base, logits, fr, None, K, N)


ROW_CASES = [
    # F, V, K, note
    (3, 20000, 10, "heavy ties, several grains"),
    (3, 20001, 64, "heavy ties, scalar rows, K = 64"),
    (2, 600000, 16, "two grains per chunk"),
]


@pytest.mark.parametrize("case", ROW_CASES, ids=[c[-1] for c in ROW_CASES])
def test_expand_row_selection_ties(tg, case):
    """Rows where hundreds or thousands of logits tie at the top of a grain
    (a constant row, a row clipped at 1.0) or where fewer than K are finite
    (the rest -inf), next to a continuous row: the per-grain selection must
    still return the K best by (logit desc, token asc)."""
    F, V, K, _ = case
    g = W.rng(V + K)
    base, _ = C.scored_tree(5, 1, 30, steps=1, width=3, K=3)
    fr = np.array([[-1, 0, 1][:F]], np.int32)
    logits = W.normal(g, (1, F, V), 3.0)
    logits[0, 1] = 0.0
    if F > 2:
        logits[0, 2] = np.minimum(np.round(logits[0, 2] / 3.0), 1.0)
        logits[0, 2, : V // 2] = -np.inf
        logits[0, 2, g.choice(V // 2, 5, replace=False)] = 2.0
    run_expand(tg, base, logits, fr, None, K, 3 * K)


def test_expand_nonfinite_capacity_and_bad_node(tg):
    g = W.rng(4)
    base, _ = C.scored_tree(5, 3, 30, steps=1, width=3, K=3, cap=20)
    logits = W.normal(g, (3, 4, 100), 2.0)
    logits[0, 1, 5] = np.nan
    logits[0, 2, 9] = np.inf
    fr = np.array([[-1, 0, 1, 2], [-1, 0, 1, 7], [-1, 0, 1, 2]], np.int32)   # node 7 missing
    got, _, _, nn, err = run_expand(tg, base, logits, fr, None, 5, 6)  # 3 + 20 > cap 20
    assert err & OT.DERR_NONFINITE and err & OT.DERR_BAD_NODE and err & OT.DERR_CAPACITY
    assert list(nn) == [0, 0, 0]
    assert list(got.n_nodes) == list(base.n_nodes)
    got, _, _, nn, err = run_expand(tg, base, np.ascontiguousarray(logits[:, :3]),
                                    np.ascontiguousarray(fr[:, :3]), None, 4, 6)
    assert err & OT.DERR_NONFINITE and not err & OT.DERR_CAPACITY
    assert nn[0] == 6 and got.n_nodes[0] == 3 + 12


def test_llama8b_expand_chain(tg):
    """Llama-3-8B-shaped drafting: 6 chained steps from the root (frontier 10,
    top-8 children, vocab 128256, N(0,3) logits per node); each call's
    next_frontier feeds the next call on the GPU."""
    cfg = W.CONFIGS["llama8b"]
    V, K, Wd = cfg["vocab"], cfg["topk"], cfg["frontier"]
    tree_h = OT.Tree.empty(1, 512)
    ts = C.tree_to_dev(tg, tree_h)
    fr = torch.full((1, Wd), -1, dtype=torch.int32, device=DEV)
    nf = torch.ones(1, dtype=torch.int32, device=DEV)
    for step in range(6):
        fr_h, nf_h = fr.cpu().numpy(), nf.cpu().numpy()
        logits = np.full((1, Wd, V), -np.inf, np.float32)
        for f in range(int(nf_h[0])):
            logits[0, f] = W.node_logits(cfg["seed"], int(fr_h[0, f]) + 1, V, cfg["logit_std"])
        lse, nxt, nn = tg.expand_topk(ts, _d(logits), fr, nf, K, Wd)
        torch.cuda.synchronize()
        want, _, nxt_o, nn_o, _ = OT.expand(tree_h, logits, fr_h, nf_h, K, Wd,
                                            lse_override=lse.cpu().numpy())
        got = C.tree_from_dev(ts)
        C.assert_tree_equal(got, want, f"step {step}")
        assert np.array_equal(nxt.cpu().numpy(), nxt_o) and np.array_equal(nn.cpu().numpy(), nn_o)
        _, lse_f, nxt_f, _, _ = OT.expand(tree_h, logits, fr_h, nf_h, K, Wd)
        _lse_close(np.where(np.arange(Wd)[None] < nf_h[:, None], lse.cpu().numpy(), np.nan), lse_f)
        assert np.array_equal(nxt_f, nxt_o)
        tree_h, fr, nf = want, nxt, nn
    assert int(tree_h.n_nodes[0]) == 8 + 64 + 4 * 80


def twodrafter_setup(B=8):
    """Two-drafter workload: per tree a 256-node tree pruned (Alg. 3) from a
    weak top-10 / frontier-10 expansion of 5 steps (410 nodes); weak rows
    N(0,3); strong = 0.8 * weak + 0.6 * N(0,3) (rho = 0.8); rows re-indexed
    with the kept nodes (row 0 root, 1 + i node i)."""
    cfg = W.CONFIGS["twodrafter"]
    V, seed = cfg["vocab"], cfg["seed"]
    big, rows = C.scored_tree(seed, B, V, steps=5, width=10, K=10, std=3.0, cap=512)
    trees, weak, strong = [], np.empty((B, 257, V), np.float32), np.empty((B, 257, V), np.float32)
    for b in range(B):
        assert int(big.n_nodes[b]) == 410
        kept, npar = C.prune_tree(big, b, 256)
        assert len(kept) == 256
        trees.append(C.subtree(big, b, kept, npar, cap=2048))
        orig = [-1] + [int(v) for v in kept]
        for r, v in enumerate(orig):
            weak[b, r] = C.row_for(rows[b], v, seed, b, V, 3.0)
            noise = W.node_logits(seed + 77, b * 1_000_000 + v + 1, V, 3.0)
            strong[b, r] = (np.float32(0.8) * weak[b, r] + np.float32(0.6) * noise)
    return C.stack_trees(trees, 2048), weak, strong


@pytest.fixture(scope="module")
def twodrafter():
    return twodrafter_setup()


def test_twodrafter_expand(tg, twodrafter):
    """Two-drafter workload, call 1: expand the 64 best leaves (K=10, N=60)."""
    tree, weak, _ = twodrafter
    B = tree.parent.shape[0]
    fr = np.empty((B, 64), np.int32)
    for b in range(B):
        n = int(tree.n_nodes[b])
        has_kid = set(int(p) for p in tree.parent[b, :n])
        leaves = [v for v in range(n) if v not in has_kid]
        keys = sorted(OT.node_key(tree.cum[b, v], tree.depth[b, v], v) for v in leaves)
        fr[b] = [k[2] for k in keys[:64]]
    logits = np.stack([weak[b, fr[b] + 1] for b in range(B)])
    run_expand(tg, tree, logits, fr, None, 10, 60)


# ----------------------------------------------------------- rescore + graft

def run_rescore(tg, tree_h, strong, Wsel, M, check_free=True, N=7):
    ts = C.tree_to_dev(tg, tree_h)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    lse, gf, ng, nx, nn = tg.rescore_graft(ts, _d(strong), Wsel, M, N=N, d_err=err)
    torch.cuda.synchronize()
    lse_g, gf_g, ng_g = lse.cpu().numpy(), gf.cpu().numpy(), ng.cpu().numpy()
    got = C.tree_from_dev(ts)
    want, lse_o, gf_o, ng_o, err_o, nx_o, nn_o = OT.rescore_graft(
        tree_h, strong, Wsel, M, lse_override=np.nan_to_num(lse_g, nan=0.0), N=N)
    C.assert_tree_equal(got, want, "rescore")
    assert np.array_equal(gf_g, gf_o) and np.array_equal(ng_g, ng_o)
    assert np.array_equal(nx.cpu().numpy(), nx_o) and np.array_equal(nn.cpu().numpy(), nn_o)
    assert int(err.item()) == err_o
    # rows written exactly where the oracle reads them
    assert np.array_equal(np.isnan(lse_g), np.isnan(lse_o))
    if check_free:
        free, lse_f, gf_f, ng_f, _ = OT.rescore_graft(tree_h, strong, Wsel, M)
        _lse_close(lse_g, lse_f)
        assert np.array_equal(ng_f, ng_g)
        for b in range(len(ng_f)):
            n0 = int(tree_h.n_nodes[b])
            C_ = OT.pool_of(tree_h, b)
            delta = float(np.max(np.abs(free.cum[b, :n0].astype(np.float64) -
                                        got.cum[b, :n0].astype(np.float64)), initial=0.0))
            keys = sorted(OT.node_key(0.0, 0, -1) if v < 0 else
                          OT.node_key(free.cum[b, v], free.depth[b, v], v) for v in C_)
            if _boundary_ok(keys, int(ng_f[b]), delta):
                assert np.array_equal(gf_f[b], gf_g[b])
    return got, lse_g, gf_g, ng_g, int(err.item())


def test_rescore_graft_golden(tg):
    """The hand-derived two-call case of tests/golden (closed-form softmaxes)."""
    import json
    import math
    import os
    gd = json.load(open(os.path.join(os.path.dirname(__file__), "golden",
                                     "rescore_graft_closed_form.json")))
    t = OT.Tree.empty(1, gd["cap"])
    it = gd["initial_tree"]
    n = len(it["parent"])
    t.parent[0, :n], t.token[0, :n], t.depth[0, :n] = it["parent"], it["token"], it["depth"]
    t.logp[0, :n], t.cum[0, :n] = -5.0, -9.0
    t.n_nodes[0] = n
    rows = np.array([[math.log(w) for w in r] for r in gd["rows"]], np.float32)[None]
    for call in gd["calls"]:
        e = call["expect"]
        n0 = int(t.n_nodes[0])
        t, lse, gf, ng, err = run_rescore(tg, t, rows, call["W"], call["M"], N=call["N"])
        assert err == 0
        assert list(gf[0, :ng[0]]) == e["graft_frontier"]
        assert list(t.token[0, n0:int(t.n_nodes[0])]) == e["new_token"]
        np.testing.assert_allclose(np.exp(t.cum[0, :n0].astype(np.float64)),
                                   e["prob_existing"], rtol=3e-6)


@pytest.mark.parametrize("seed", range(8))
def test_rescore_random_small(tg, seed):
    g = W.rng(500 + seed)
    B = int(g.integers(1, 4))
    V = int([60, 1000, 4099, 20000][seed % 4])
    tree, _ = C.scored_tree(600 + seed, B, V, steps=int(g.integers(1, 4)), width=4, K=3,
                            cap=512)
    C.mark_visited_closed(g, tree)
    R = int(tree.n_nodes.max()) + 1 + int(g.integers(0, 3))
    strong = W.normal(g, (B, R, V), 3.0)
    Wsel, M = int(g.integers(1, 12)), int(g.integers(1, min(V, 64) + 1))
    run_rescore(tg, tree, strong, Wsel, M)


def test_rescore_identical_drafter_and_all_visited(tg):
    """GPU tree built by GPU expansion, then rescored with the very rows that
    built it: every stored logp / cum is reproduced bit for bit.  A second call
    with everything visited is a no-op."""
    V, B = 3000, 2
    ts = tg.TreeState(B, 256, DEV)
    fr = torch.full((B, 4), -1, dtype=torch.int32, device=DEV)
    nf = torch.ones(B, dtype=torch.int32, device=DEV)
    rows = {}
    for _ in range(3):
        fr_h, nf_h = fr.cpu().numpy(), nf.cpu().numpy()
        lg = np.full((B, 4, V), -np.inf, np.float32)
        for b in range(B):
            for f in range(int(nf_h[b])):
                v = int(fr_h[b, f])
                rows[(b, v)] = W.node_logits(9, b * 1000 + v + 1, V, 3.0)
                lg[b, f] = rows[(b, v)]
        _, fr, nf = tg.expand_topk(ts, _d(lg), fr, nf, 3, 4)
    before = C.tree_from_dev(ts)
    R = int(before.n_nodes.max()) + 1
    strong = np.stack([np.stack([rows.get((b, r - 1), np.zeros(V, np.float32))
                                 for r in range(R)]) for b in range(B)])
    tg.rescore_graft(ts, _d(strong), 4, 2)
    torch.cuda.synchronize()
    after = C.tree_from_dev(ts)
    for b in range(B):
        n = int(before.n_nodes[b])
        assert np.array_equal(after.logp[b, :n].view(np.uint32), before.logp[b, :n].view(np.uint32))
        assert np.array_equal(after.cum[b, :n].view(np.uint32), before.cum[b, :n].view(np.uint32))
    snap = C.tree_from_dev(ts)
    R2 = int(snap.n_nodes.max()) + 1
    strong2 = W.normal(W.rng(1), (B, R2, V), 3.0)
    # mark everything visited, then a middle step must change nothing
    ts.visited.fill_(1)
    ts.root_visited.fill_(1)
    snap = C.tree_from_dev(ts)
    lse, gf, ng = tg.rescore_graft(ts, _d(strong2), 4, 2)
    torch.cuda.synchronize()
    C.assert_tree_equal(C.tree_from_dev(ts), snap, "all visited")
    assert list(ng.cpu().numpy()) == [0, 0]
    assert np.all(np.isnan(lse.cpu().numpy()))


def test_rescore_deep_pool_chains(tg):
    """Pool paths deeper than the rescore kernel's per-thread walk (16 pool
    levels above a node): a 45-node chain and a 20-node branch hanging from
    its sixth node, the first three chain nodes visited (the rest and the
    branch form the pool), plus a second tree whose pool is shallow."""
    g = W.rng(91)
    V, cap = 400, 256
    t = OT.Tree.empty(2, cap)
    par = [[-1] + list(range(0, 44)) + [5] + list(range(45, 64)),
           [-1, -1, 0, 0, 1, 2, 3, 3, 5, 6]]
    for b, pb in enumerate(par):
        n = len(pb)
        t.parent[b, :n] = pb
        for v, p in enumerate(pb):
            t.depth[b, v] = 1 if p < 0 else t.depth[b, p] + 1
            t.token[b, v] = int(g.integers(0, V))
            t.logp[b, v] = np.float32(-g.random() * 4.0)
            t.cum[b, v] = t.logp[b, v] if p < 0 else np.float32(t.cum[b, p] + t.logp[b, v])
        t.n_nodes[b] = n
        t.root_visited[b] = 1
    t.visited[0, :3] = 1
    t.visited[1, :2] = 1
    R = int(t.n_nodes.max()) + 1
    strong = W.normal(g, (2, R, V), 3.0)
    got, _, _, ng, err = run_rescore(tg, t, strong, 5, 3)
    assert err == 0 and list(ng) == [5, 5]


def test_rescore_capacity_and_rows_errors(tg):
    tree, _ = C.scored_tree(8, 2, 50, steps=2, width=3, K=3, cap=20)  # 3 + 9 = 12 nodes
    strong = W.normal(W.rng(2), (2, 13, 50), 2.0)
    got, _, gf, ng, err = run_rescore(tg, tree, strong, 4, 3)         # 12 + 4*3 > 20
    assert err & OT.DERR_CAPACITY and list(ng) == [0, 0]
    got, _, gf, ng, err = run_rescore(tg, tree, strong[:, :12], 2, 2)  # R < n + 1
    assert err & OT.DERR_BAD_NODE and list(ng) == [0, 0]


def test_twodrafter_rescore(tg, twodrafter):
    """Two-drafter workload, call 2: middle-drafter step on the initial
    256-node trees (nothing visited: pool = 256 nodes + root, 257 rows),
    W = 60, M = 10."""
    tree, _, strong = twodrafter
    got, lse, gf, ng, err = run_rescore(tg, tree, strong, 60, 10)
    assert err == 0 and list(ng) == [60] * 8
    assert list(got.n_nodes) == [256 + 600] * 8


def test_twodrafter_chained_expand_then_rescore(tg, twodrafter):
    """Expand (weak, 64 leaves) then rescore + graft (strong) on the result:
    pool = 256 + 640 nodes + root; oracle chained with the GPU lse."""
    tree, weak, strong = twodrafter
    tree = OT.Tree(*(getattr(tree, f)[:2].copy() for f in
                     ("parent", "token", "depth", "logp", "cum", "visited", "root_visited",
                      "n_nodes")), cap=tree.cap)
    B, V = 2, weak.shape[2]
    fr = np.stack([np.argsort(-tree.cum[b, :256], kind="stable")[:64] for b in range(B)]).astype(np.int32)
    logits = np.stack([weak[b, fr[b] + 1] for b in range(B)])
    mid, *_ = run_expand(tg, tree, logits, fr, None, 10, 60, check_free=False)
    g = W.rng(99)
    R = 256 + 640 + 1
    strong2 = np.empty((B, R, V), np.float32)
    strong2[:, :257] = strong[:B]
    strong2[:, 257:] = W.normal(g, (B, R - 257, V), 3.0)
    run_rescore(tg, mid, strong2, 60, 10, check_free=False)


# ------------------------------------------------------------------ accept

def run_accept(tg, parent, token, n, greedy, max_depth):
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    A, path, bonus = tg.accept(_d(parent, torch.int32), _d(token, torch.int32),
                               _d(n, torch.int32), _d(greedy, torch.int32), max_depth,
                               d_err=err)
    torch.cuda.synchronize()
    rA, rpath, rbonus, rerr = OT.accept(parent, token, n, greedy, max_depth)
    assert np.array_equal(A.cpu().numpy(), rA)
    assert np.array_equal(path.cpu().numpy(), rpath)
    assert np.array_equal(bonus.cpu().numpy(), rbonus)
    assert int(err.item()) == rerr
    return rA


@pytest.mark.parametrize("seed", range(10))
def test_accept_random(tg, seed):
    g = W.rng(700 + seed)
    B, cap = 4, 300
    parent = np.full((B, cap), -1, np.int32)
    token = np.zeros((B, cap), np.int32)
    greedy = np.zeros((B, cap + 1), np.int32)
    n = np.zeros(B, np.int32)
    for b in range(B):
        nb = int(g.integers(0, cap + 1))
        n[b] = nb
        par = W.uniform_parents(g, nb) if seed % 2 else W.level_tree(g, max(nb, 12), 12, 8)[:nb]
        if nb and seed % 2 == 0:
            par = W.level_tree(g, nb, min(12, nb), 8) if nb >= 12 else W.uniform_parents(g, nb)
        parent[b, :nb] = par
        V = 5 if seed % 3 == 0 else 1000        # tiny vocab: duplicate siblings
        tok = (g.integers(0, V, size=nb) if V == 5 else W.distinct_sibling_tokens(g, par, V))
        token[b, :nb] = tok
        greedy[b] = W.greedy_match_random_child(g, np.concatenate([par, np.full(cap - nb, -1)]),
                                                np.concatenate([tok, np.zeros(cap - nb)]).astype(np.int32),
                                                V + 1, 0.8)
    run_accept(tg, parent, token, n, greedy, 16)


def test_accept_tiny_and_llama8b_configs(tg):
    cfg = W.CONFIGS["tiny"]
    g = W.rng(cfg["seed"] + 5)
    par = W.uniform_parents(g, 16)
    tok = W.distinct_sibling_tokens(g, par, cfg["vocab"])
    greedy = W.greedy_match_random_child(g, par, tok, cfg["vocab"], 0.5)
    run_accept(tg, par[None], tok[None], np.array([16]), greedy[None], 16)
    cfg = W.CONFIGS["llama8b"]
    g = W.rng(cfg["seed"] + 5)
    par = W.expansion_shaped_tree(g, 63, 6, 8, 10)
    tok = W.distinct_sibling_tokens(g, par, cfg["vocab"])
    for s in range(20):
        greedy = W.greedy_match_first_child(W.rng([cfg["seed"], s]), par, tok, cfg["vocab"], 0.7)
        run_accept(tg, par[None], tok[None], np.array([63]), greedy[None], 6)


def test_accept_deep_chain_and_depth_limit(tg):
    n = 4096
    par = np.arange(-1, n - 1, dtype=np.int32)[None]
    tok = np.arange(n, dtype=np.int32)[None] % 7
    greedy = np.concatenate([tok[0], [3]]).astype(np.int32)[None]
    assert run_accept(tg, par, tok, np.array([n]), greedy, n)[0] == n
    greedy2 = greedy.copy()
    greedy2[0, 3000] = 99           # breaks the match at node 3000
    assert run_accept(tg, par, tok, np.array([n]), greedy2, n)[0] == 3000
    assert run_accept(tg, par, tok, np.array([n]), greedy, 100)[0] == 100   # CAPACITY bit


def test_accept_bad_parent(tg):
    par = np.array([[-1, 5, 0, 1]], np.int32)
    tok = np.array([[1, 2, 3, 4]], np.int32)
    greedy = np.array([[1, 3, 9, 9, 9]], np.int32)
    run_accept(tg, par, tok, np.array([4]), greedy, 4)


def test_accept_nd_example(tg):
    import json
    import os
    gd = json.load(open(os.path.join(os.path.dirname(__file__), "golden",
                                     "accept_nd_example.json")))
    for key in ("nd", "overwrite"):
        c = gd[key]
        n = len(c["parent"])
        A = run_accept(tg, np.array([c["parent"]], np.int32), np.array([c["token"]], np.int32),
                       np.array([n]), np.array([c["greedy"]], np.int32), c["max_depth"])
        assert A[0] == c["expect"]["A"]


def test_expand_frontier_id_equal_to_the_node_count(tg):
    """Frontier id n_b is one past the last node: BAD_NODE, tree unchanged;
    ids n_b - 1 fill the tree to its capacity exactly."""
    t = OT.Tree.empty(1, 6)
    t.parent[0, :2], t.token[0, :2], t.depth[0, :2], t.n_nodes[0] = [-1, 0], [1, 2], [1, 2], 2
    logits = W.normal(W.rng(41), (1, 2, 50), 2.0)
    got, _, _, nn, err = run_expand(tg, t, logits, np.array([[1, 2]], np.int32), None, 2, 4)
    assert err & OT.DERR_BAD_NODE and int(nn[0]) == 0 and int(got.n_nodes[0]) == 2
    got, _, _, nn, err = run_expand(tg, t, logits, np.array([[0, 1]], np.int32), None, 2, 4)
    assert err == 0 and int(got.n_nodes[0]) == 6
