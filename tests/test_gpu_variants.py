"""GPU parity of the middle-step variants of tg_tree_rescore_graft (the Sec.
4.4 ablations w/o EG and w/o ND, and the duplicate-sibling filter) and of
tg_tree_accept_logits (the target's arg-max fused with acceptance).

As for the paper's variant, the oracle re-run with the GPU's exported lse
must agree bit for bit on every integer output and every stored fp32 score.
"""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import tree as OT
from tests import _cases as C

pytestmark = pytest.mark.gpu
DEV = "cuda"

NEW, OVW, DED = OT.POOL_NEWONLY, OT.GRAFT_OVERWRITE, OT.GRAFT_DEDUP
FLAG_SETS = [NEW, OVW, DED, OVW | DED, NEW | OVW, NEW | DED, NEW | OVW | DED]


def _d(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def run_variant(tg, tree_h, strong, Wsel, M, flags, new_from=None, N=7):
    ts = C.tree_to_dev(tg, tree_h)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    nf = _d(new_from.astype(np.int32)) if new_from is not None else None
    lse, gf, ng, nx, nn = tg.rescore_graft(ts, _d(strong), Wsel, M, N=N, d_err=err,
                                           flags=flags, new_from=nf)
    torch.cuda.synchronize()
    lse_g = lse.cpu().numpy()
    got = C.tree_from_dev(ts)
    want, lse_o, gf_o, ng_o, err_o, nx_o, nn_o = OT.rescore_graft(
        tree_h, strong, Wsel, M, lse_override=np.nan_to_num(lse_g, nan=0.0), N=N,
        flags=flags, new_from=new_from)
    C.assert_tree_equal(got, want, f"flags {flags}")
    assert np.array_equal(gf.cpu().numpy(), gf_o) and np.array_equal(ng.cpu().numpy(), ng_o)
    assert np.array_equal(nx.cpu().numpy(), nx_o) and np.array_equal(nn.cpu().numpy(), nn_o)
    assert int(err.item()) == err_o
    assert np.array_equal(np.isnan(lse_g), np.isnan(lse_o))
    return got, gf.cpu().numpy(), ng.cpu().numpy()


@pytest.mark.parametrize("flags", FLAG_SETS)
@pytest.mark.parametrize("seed", range(3))
def test_variants_random_trees(tg, flags, seed):
    g = W.rng([800, flags, seed])
    B = int(g.integers(1, 4))
    V = [8, 60, 1000][seed]               # small vocabularies give duplicate siblings
    tree, _ = C.scored_tree(810 + seed, B, V, steps=3, width=4, K=3, cap=512)
    C.mark_visited_closed(g, tree)
    R = int(tree.n_nodes.max()) + 1
    strong = W.normal(g, (B, R, V), 3.0)
    new_from = np.array([int(g.integers(-1, int(n) + 1)) for n in tree.n_nodes], np.int32)
    Wsel, M = int(g.integers(1, 10)), int(g.integers(1, min(V, 6) + 1))
    run_variant(tg, tree, strong, Wsel, M, flags, new_from)


def test_overwrite_large_tree(tg):
    """A 2048-slot tree (the largest the variants hold) with ~1100 nodes,
    frontier spread over many depths."""
    g = W.rng(820)
    tree, _ = C.scored_tree(821, 1, 500, steps=6, width=40, K=5, cap=2048)
    R = int(tree.n_nodes[0]) + 1
    strong = W.normal(g, (1, R, 500), 3.0)
    got, gf, ng = run_variant(tg, tree, strong, 40, 4, OVW | DED)
    assert int(got.n_nodes[0]) < int(tree.n_nodes[0]) + 40 * 4


def test_overwrite_vs_nd_accepted_branch(tg):
    """App. G end to end on the GPU: grafting at a historical node keeps the
    branch the target accepts (length 3) unless the graft overwrites it
    (length 1)."""
    V, cap = 8, 32
    t = OT.Tree.empty(1, cap)
    for i, (p, tok) in enumerate([(-1, 1), (0, 2), (1, 3), (-1, 4)]):
        t.parent[0, i], t.token[0, i] = p, tok
        t.depth[0, i] = 1 if p < 0 else int(t.depth[0, p]) + 1
    t.n_nodes[0], t.root_visited[0] = 4, 1
    strong = np.full((1, 5, V), -20.0, np.float32)
    strong[0, 0, 1], strong[0, 0, 4] = 5.0, 1.0
    strong[0, 1, 5], strong[0, 1, 6], strong[0, 1, 2] = 4.0, 3.0, 0.0
    strong[0, 2, 3], strong[0, 3, 7], strong[0, 4, 0] = 4.0, 4.0, 4.0
    rule = {(): 1, (1,): 2, (1, 2): 3, (1, 2, 3): 7}
    lens = {}
    for flags in (0, OVW):
        ts = C.tree_to_dev(tg, t)
        tg.rescore_graft(ts, _d(strong), 1, 2, flags=flags)
        got = C.tree_from_dev(ts)
        n = int(got.n_nodes[0])
        # the target's greedy token after each node's token path
        logits = np.full((1, cap + 1, V), 0.0, np.float32)
        paths = {}
        for i in range(n):
            p = int(got.parent[0, i])
            paths[i] = (paths[p] if p >= 0 else ()) + (int(got.token[0, i]),)
        logits[0, 0, rule[()]] = 9.0
        for i in range(n):
            logits[0, i + 1, rule.get(paths[i], 0)] = 9.0
        greedy, A, path, bonus = tg.accept_logits(ts.parent, ts.token, ts.n_nodes,
                                                  _d(logits), 8)
        lens[flags] = int(A.item())
    assert lens == {0: 3, OVW: 1}


@pytest.mark.parametrize("seed", range(4))
def test_accept_logits_matches_oracle(tg, seed):
    g = W.rng(830 + seed)
    B = int(g.integers(1, 4))
    V = [17, 1000, 4096, 32003][seed]
    tree, _ = C.scored_tree(831 + seed, B, 50, steps=3, width=4, K=3, cap=128)
    R = int(tree.n_nodes.max()) + 1 + (0 if seed != 2 else -2)   # seed 2: rows missing
    logits = np.round(W.normal(g, (B, max(R, 1), V), 1.5)).astype(np.float32)  # ties
    logits[0, 0, min(3, V - 1)] = np.nan
    # make some paths acceptable: the arg-max after a node's parent is its token
    for b in range(B):
        for v in range(int(tree.n_nodes[b])):
            p = int(tree.parent[b, v])
            if p + 1 < logits.shape[1] and g.random() < 0.6:
                logits[b, p + 1, int(tree.token[b, v]) % V] = 50.0
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    ts = C.tree_to_dev(tg, tree)
    greedy, A, path, bonus = tg.accept_logits(ts.parent, ts.token, ts.n_nodes, _d(logits), 6,
                                              d_err=err)
    torch.cuda.synchronize()
    g_o, A_o, path_o, bonus_o, err_o = OT.accept_logits(tree.parent, tree.token,
                                                        tree.n_nodes, logits, 6)
    gg = greedy.cpu().numpy()
    Rw = min(logits.shape[1], tree.cap + 1)
    assert np.array_equal(gg[:, :Rw], g_o[:, :Rw])
    assert (gg[:, Rw:] == -1).all()
    assert np.array_equal(A.cpu().numpy(), A_o)
    assert np.array_equal(path.cpu().numpy(), path_o)
    assert np.array_equal(bonus.cpu().numpy(), bonus_o)
    assert int(err.item()) == err_o


@pytest.mark.parametrize("extra", [0, -1])
def test_accept_logits_row_bound(tg, extra):
    """Rows 0..n_nodes are read: R = n_nodes + 1 fits, R = n_nodes does not
    (BAD_NODE; the missing row reads as no match)."""
    g = W.rng(840)
    tree, _ = C.scored_tree(841, 1, 40, steps=2, width=3, K=2, cap=32)
    R = int(tree.n_nodes[0]) + 1 + extra
    logits = np.round(W.normal(g, (1, R, 300), 1.5)).astype(np.float32)
    for v in range(int(tree.n_nodes[0])):
        p = int(tree.parent[0, v])
        if p + 1 < R:
            logits[0, p + 1, int(tree.token[0, v])] = 50.0
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    ts = C.tree_to_dev(tg, tree)
    greedy, A, path, bonus = tg.accept_logits(ts.parent, ts.token, ts.n_nodes, _d(logits), 6,
                                              d_err=err)
    torch.cuda.synchronize()
    g_o, A_o, path_o, bonus_o, err_o = OT.accept_logits(tree.parent, tree.token,
                                                        tree.n_nodes, logits, 6)
    assert int(err.item()) == err_o == (0 if extra == 0 else OT.DERR_BAD_NODE)
    Rw = min(R, tree.cap + 1)
    assert np.array_equal(greedy.cpu().numpy()[:, :Rw], g_o[:, :Rw])
    assert np.array_equal(A.cpu().numpy(), A_o) and np.array_equal(bonus.cpu().numpy(), bonus_o)
    assert np.array_equal(path.cpu().numpy(), path_o)
