"""GPU parity of tg_tree_signals (scheduler tree signals and margin
predictor) against the oracle.  Signals are means of small integers or of
fp32 scores: compared to 1e-5 relative; NaN where the oracle has NaN; the
action is compared wherever the margin is not within 1e-4 of zero."""
from __future__ import annotations

import json
import os

import numpy as np
import pytest

import workloads as W
from oracle import signals as OS
from oracle import tree as OT
from tests import _cases as C

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu
DEV = "cuda"
GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _d(a, dtype=torch.int32):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV).to(dtype)


def run(tg, tree_h, frontier, nf, Wd, L, context=None, params=None):
    ts = C.tree_to_dev(tg, tree_h)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    sig, mg, act = tg.tree_signals(ts, _d(frontier), None if nf is None else _d(nf), Wd, L,
                                   None if context is None else _d(context, torch.float32),
                                   None if params is None else _d(params, torch.float32),
                                   d_err=err)
    torch.cuda.synchronize()
    return (sig.cpu().numpy(), None if mg is None else mg.cpu().numpy(),
            None if act is None else act.cpu().numpy(), int(err.item()))


def close(a, b):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    both_nan = np.isnan(a) & np.isnan(b)
    return bool(np.all(both_nan | np.isclose(a, b, rtol=1e-5, atol=1e-6)))


def test_signals_golden(tg):
    gd = json.load(open(os.path.join(GOLD, "tree_signals.json")))
    for c in gd["cases"]:
        t = OT.Tree.empty(1, 8)
        n = len(gd["parent"])
        t.parent[0, :n] = gd["parent"]
        t.depth[0, :n] = gd["depth"]
        t.cum[0, :n] = [float(x) for x in c["cum"]]
        t.n_nodes[0] = n
        fr = np.array([c["frontier"]], np.int32)
        sig, _, _, err = run(tg, t, fr, None, c["W"], c["L"])
        assert err == 0
        assert np.allclose(sig[0], c["signals"], rtol=0, atol=1e-6)


@pytest.mark.parametrize("seed", range(3))
def test_signals_grown_trees(tg, seed):
    """Trees grown by expansion; the frontier is the last step's Top_W of new
    children (what the scheduler sees before the next step), plus random
    frontiers with the root and older nodes."""
    tree, _ = C.scored_tree(900 + seed, 4, 60, steps=5, width=8, K=4, cap=1024)
    g = W.rng(910 + seed)
    B, F = 4, 12
    fr = np.full((B, F), -1, np.int32)
    nf = np.zeros(B, np.int32)
    for b in range(B):
        n = int(tree.n_nodes[b])
        k = int(g.integers(1, F + 1))
        fr[b, :k] = g.choice(np.arange(-1, n), size=k, replace=False)
        nf[b] = k
    for Wd, L in ((1, 0), (8, 5), (60, 2), (500, 9)):
        sig, _, _, err = run(tg, tree, fr, nf, Wd, L)
        assert err == 0
        for b in range(B):
            n = int(tree.n_nodes[b])
            want, _ = OS.tree_signals(tree.parent[b], tree.depth[b], tree.cum[b], n,
                                      list(fr[b, :nf[b]]), Wd, L)
            assert close(sig[b], want), (b, Wd, L, sig[b], want)


def test_signals_larger_grown_trees_select_the_preview(tg):
    """552-node grown trees: the preview frontier Top_W(R) of a few hundred
    candidates takes the selection paths (a per-wave bound, then counting
    among the keys above it) for W up to 16 and up to 64."""
    tree, _ = C.scored_tree(940, 2, 60, steps=7, width=12, K=8, cap=1024)
    g = W.rng(941)
    B, F = 2, 12
    fr = np.full((B, F), -1, np.int32)
    nf = np.zeros(B, np.int32)
    for b in range(B):
        n = int(tree.n_nodes[b])
        assert n > 512
        fr[b] = g.choice(np.arange(-1, n), size=F, replace=False)
        nf[b] = F
    for Wd, L in ((1, 0), (10, 5), (16, 9), (17, 9), (60, 9)):
        sig, _, _, err = run(tg, tree, fr, nf, Wd, L)
        assert err == 0
        for b in range(B):
            n = int(tree.n_nodes[b])
            want, _ = OS.tree_signals(tree.parent[b], tree.depth[b], tree.cum[b], n,
                                      list(fr[b, :nf[b]]), Wd, L)
            assert close(sig[b], want), (b, Wd, L, sig[b], want)


def test_signals_full_tree_with_infinite_scores_and_margin(tg):
    """4096-node random trees with -inf scores, and the predictor on top."""
    g = W.rng(920)
    B, cap = 3, 4096
    t = OT.Tree.empty(B, cap)
    for b in range(B):
        n = cap - 7 * b
        par = W.uniform_parents(g, n)
        t.parent[b, :n] = par
        t.depth[b, :n] = W.node_depths(par)
        cum = -np.abs(W.normal(g, (n,), 3.0))
        cum[g.random(n) < 0.05] = -np.inf
        t.cum[b, :n] = cum
        t.n_nodes[b] = n
    F = 60
    fr = np.stack([g.choice(np.arange(-1, int(t.n_nodes[b])), size=F, replace=False)
                   for b in range(B)]).astype(np.int32)
    params = W.normal(g, (OS.N_PARAMS,), 0.3)
    ctx = W.normal(g, (B, 11), 1.0)
    sig, mg, act, err = run(tg, t, fr, None, 60, 5, ctx, params)
    assert err == 0
    for b in range(B):
        want, _ = OS.tree_signals(t.parent[b], t.depth[b], t.cum[b], int(t.n_nodes[b]),
                                  list(fr[b]), 60, 5)
        assert close(sig[b], want)
        y, a = OS.margin(ctx[b], sig[b].astype(np.float64), params)
        assert abs(mg[b] - y) <= 1e-5 * max(1.0, abs(y))
        if abs(y) > 1e-4:
            assert act[b] == a


def test_signals_errors_and_empty_frontier(tg):
    tree, _ = C.scored_tree(930, 3, 30, steps=2, width=3, K=3)
    fr = np.array([[0, 1], [0, 999], [2, 3]], np.int32)
    nf = np.array([2, 2, 0], np.int32)
    sig, _, _, err = run(tg, tree, fr, nf, 4, 5)
    assert err & OT.DERR_BAD_NODE
    assert np.isnan(sig[1]).all()                       # bad frontier id
    want, _ = OS.tree_signals(tree.parent[2], tree.depth[2], tree.cum[2],
                              int(tree.n_nodes[2]), [], 4, 5)
    assert close(sig[2], want)                          # empty frontier: NaN means
    want0, _ = OS.tree_signals(tree.parent[0], tree.depth[0], tree.cum[0],
                               int(tree.n_nodes[0]), [0, 1], 4, 5)
    assert close(sig[0], want0)
