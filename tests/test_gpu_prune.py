"""GPU parity of tg_tree_global_prune (Alg. 3 and its verification buffers)
and tg_kv_compact (cache update after acceptance) against the oracle.
Integer outputs are compared bit for bit."""
from __future__ import annotations

import json
import os

import numpy as np
import pytest

import workloads as W
from oracle import attention as OA
from oracle import tree as OT
from tests import _cases as C

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu
DEV = "cuda"
GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _bits(mask_rows, M):
    """[M, M] 0/1 matrix -> [M, ceil(M/32)] uint32 bitsets (bit v of word v/32)."""
    W_ = (M + 31) // 32
    out = np.zeros((M, W_), np.uint32)
    for u in range(mask_rows.shape[0]):
        for v in np.nonzero(mask_rows[u])[0]:
            out[u, v >> 5] |= np.uint32(1 << (int(v) & 31))
    return out


def run_prune(tg, tree_h, B_ver, max_path=None):
    ts = C.tree_to_dev(tg, tree_h)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    out = tg.global_prune(ts, B_ver, max_path, d_err=err)
    torch.cuda.synchronize()
    got = {k: v.cpu().numpy() for k, v in out.items()}
    got["mask"] = got["mask"].view(np.uint32)
    return got, int(err.item())


def check_tree(got, tree_h, b, B_ver, max_path):
    """Tree b of a prune result against the oracle's Alg. 3."""
    n = int(tree_h.n_nodes[b])
    M = B_ver + 1
    want = OT.global_prune(tree_h.parent[b, :n], tree_h.cum[b, :n], n, B_ver)
    nk = len(want["kept"])
    assert got["n_keep"][b] == nk
    assert list(got["kept"][b, :nk]) == list(want["kept"])
    assert (got["kept"][b, nk:] == -1).all()
    assert list(got["vparent"][b, :nk]) == list(want["parent"])
    assert list(got["vtoken"][b, :nk]) == list(tree_h.token[b, want["kept"]])
    assert list(got["position_ids"][b, :nk + 1]) == list(want["position_ids"])
    assert (got["position_ids"][b, nk + 1:] == -1).all()
    wb = _bits(want["mask"], M)
    assert np.array_equal(got["mask"][b, :nk + 1], wb[:nk + 1])
    assert (got["mask"][b, nk + 1:] == 0).all()
    retr = want["retrieval"]
    nl, width = retr.shape
    assert got["n_leaves"][b] == nl
    assert np.array_equal(got["retrieval"][b, :nl, :width], retr)
    assert (got["retrieval"][b, :nl, width:] == -1).all()
    assert (got["retrieval"][b, nl:] == -1).all()


def test_prune_golden_non_monotone_scores(tg):
    """Hand-derived Alg. 3 cases where a chain adds two nodes (the literal
    loop, not the closed form)."""
    gd = json.load(open(os.path.join(GOLD, "prune_alg3.json")))
    par = np.array(gd["parent"], np.int32)
    cum = np.array(gd["cum"], np.float32)
    for c in gd["cases"]:
        t = OT.Tree.empty(1, 16)
        n = len(par)
        t.parent[0, :n] = par
        t.cum[0, :n] = cum
        t.token[0, :n] = np.arange(100, 100 + n)
        t.n_nodes[0] = n
        got, err = run_prune(tg, t, c["B_ver"], 8)
        assert err == 0
        nk = len(c["kept"])
        assert list(got["kept"][0, :nk]) == c["kept"]
        assert list(got["vparent"][0, :nk]) == c["new_parent"]
        assert list(got["position_ids"][0, :nk + 1]) == c["position_ids"]
        M = c["B_ver"] + 1
        assert np.array_equal(got["mask"][0, :nk + 1], _bits(np.array(c["mask"]), M)[:nk + 1])
        r = np.array(c["retrieval"])
        assert np.array_equal(got["retrieval"][0, :r.shape[0], :r.shape[1]], r)


@pytest.mark.parametrize("seed", range(3))
def test_prune_scored_trees(tg, seed):
    """Trees grown by expansion (cum never increases along a path): budgets
    below, at and above the node count."""
    tree, _ = C.scored_tree(500 + seed, 3, 60, steps=5, width=6, K=4, cap=1024)
    for B_ver in (1, 7, 31, 63, int(tree.n_nodes.max()), 200):
        got, err = run_prune(tg, tree, B_ver, B_ver + 1)
        assert err == 0
        for b in range(3):
            check_tree(got, tree, b, B_ver, B_ver + 1)


@pytest.mark.parametrize("seed", range(4))
def test_prune_random_trees_with_ties_and_inversions(tg, seed):
    """Uniform random parents with integer scores (ties in cum, children
    scoring above parents): exercises the literal loop and the tie-break."""
    g = W.rng(520 + seed)
    B, cap = 4, 300
    t = OT.Tree.empty(B, cap)
    for b in range(B):
        n = int(g.integers(1, cap + 1))
        t.parent[b, :n] = W.uniform_parents(g, n)
        t.cum[b, :n] = -g.integers(0, 6, size=n).astype(np.float32)
        t.token[b, :n] = g.integers(0, 1000, size=n)
        t.n_nodes[b] = n
    for B_ver in (1, 10, 64, 299):
        got, err = run_prune(tg, t, B_ver, cap + 1)
        assert err == 0
        for b in range(B):
            check_tree(got, t, b, B_ver, cap + 1)


def test_prune_full_capacity_chain_and_path_limit(tg):
    """A 4096-node chain (deepest tree the library holds): depths by pointer
    jumping; a retrieval width below the kept depth raises CAPACITY and
    leaves that tree's paths empty."""
    cap = 4096                                           # TG_MAX_CAP
    t = OT.Tree.empty(2, cap)
    t.parent[0, :cap] = np.arange(-1, cap - 1)
    t.cum[0, :cap] = -np.arange(cap, dtype=np.float32) * 0.01
    t.n_nodes[0] = cap
    g = W.rng(530)
    t.parent[1, :cap] = W.uniform_parents(g, cap)
    t.cum[1, :cap] = -np.abs(W.normal(g, (cap,), 1.0))
    t.n_nodes[1] = cap
    got, err = run_prune(tg, t, 63, 64)
    assert err == 0
    check_tree(got, t, 0, 63, 64)
    check_tree(got, t, 1, 63, 64)
    got, err = run_prune(tg, t, 63, 10)
    assert err & OT.DERR_CAPACITY
    assert (got["retrieval"][0] == -1).all()
    assert got["n_keep"][0] == 63 and list(got["kept"][0, :63]) == list(range(63))


def test_prune_large_budget_sorts(tg):
    """Budgets and trees past 1024 nodes take the sorting paths for both the
    rank and the re-index (a 4096-node random tree, 1500 kept)."""
    cap = 4096
    t = OT.Tree.empty(1, cap)
    g = W.rng(531)
    t.parent[0, :cap] = W.uniform_parents(g, cap)
    t.cum[0, :cap] = -np.abs(W.normal(g, (cap,), 1.0))
    t.token[0, :cap] = np.arange(cap, dtype=np.int32) * 7 % 32000
    t.n_nodes[0] = cap
    got, err = run_prune(tg, t, 1500, 64)
    assert err == 0
    check_tree(got, t, 0, 1500, 64)


def test_prune_bad_tree_and_parent(tg):
    t = OT.Tree.empty(2, 8)
    t.parent[0, :3] = [-1, 5, 0]     # node 1's parent is not earlier: read as the root
    t.cum[0, :3] = [-1.0, -2.0, -3.0]
    t.n_nodes[0] = 3
    t.n_nodes[1] = 9                 # more than cap
    got, err = run_prune(tg, t, 4, 5)
    assert err & OT.DERR_BAD_PARENT and err & OT.DERR_BAD_NODE
    check_tree(got, t, 0, 4, 5)
    assert got["n_keep"][1] == 0 and got["n_leaves"][1] == 0
    assert (got["kept"][1] == -1).all() and (got["retrieval"][1] == -1).all()


def test_prune_then_verify_tree_is_ancestor_closed(tg):
    """A two-drafter-shaped tree (256 nodes) pruned to 63: every kept node's
    parent is kept and earlier, position ids are depths, and each mask row
    is exactly the ancestor chain (the layout tg_tree_verify_attention takes
    after prepending the root)."""
    tree, _ = C.scored_tree(540, 2, 80, steps=4, width=8, K=8, cap=1024)
    got, err = run_prune(tg, tree, 63, 64)
    assert err == 0
    for b in range(2):
        nk = got["n_keep"][b]
        vp = got["vparent"][b, :nk]
        assert all(p < j for j, p in enumerate(vp))
        check_tree(got, tree, b, 63, 64)


# ---------------------------------------------------------------- kv compact

@pytest.mark.parametrize("dtype,D", [(torch.bfloat16, 128), (torch.float32, 64),
                                     (torch.bfloat16, 64)])
def test_kv_compact_matches_oracle(tg, dtype, D):
    g = W.rng(550 + D)
    B, Hkv, N = 4, 3, 40
    L = np.array([0, 17, 100, 33])
    S = int(L.max()) + N + 5
    k = W.normal(g, (B, Hkv, S, D))
    v = W.normal(g, (B, Hkv, S, D))
    maxp = 12
    path = np.full((B, maxp), -1, np.int32)
    n = np.zeros(B, np.int32)
    for b in range(B):
        par = W.uniform_parents(g, N)
        leaf = int(g.integers(0, N))
        chain = [0] + [a + 1 for a in OA.path_of(par, leaf)]   # root slot, then nodes
        chain = chain[:maxp]
        path[b, :len(chain)] = chain
        n[b] = len(chain)
    n[3] = 0
    kd = torch.from_numpy(k).to(DEV).to(dtype)
    vd = torch.from_numpy(v).to(DEV).to(dtype)
    k_in = kd.float().cpu().numpy()
    v_in = vd.float().cpu().numpy()
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    nl = tg.kv_compact(kd, vd, torch.from_numpy(L.astype(np.int32)).to(DEV),
                       torch.from_numpy(path).to(DEV), torch.from_numpy(n).to(DEV), d_err=err)
    torch.cuda.synchronize()
    k2, v2, nl_o, err_o = OA.kv_compact(k_in, v_in, L, path, n)
    assert int(err.item()) == err_o == 0
    assert list(nl.cpu().numpy()) == list(nl_o)
    assert np.array_equal(kd.float().cpu().numpy(), k2)
    assert np.array_equal(vd.float().cpu().numpy(), v2)


def test_kv_compact_rejects_bad_paths(tg):
    g = W.rng(560)
    B, Hkv, S, D = 3, 2, 24, 64
    k = torch.from_numpy(W.normal(g, (B, Hkv, S, D))).to(DEV)
    v = torch.from_numpy(W.normal(g, (B, Hkv, S, D))).to(DEV)
    k0, v0 = k.clone(), v.clone()
    L = torch.tensor([4, 6, 2], dtype=torch.int32, device=DEV)
    path = torch.tensor([[0, 1, 2, 3], [0, 2, 1, 5], [0, 3, 9, 22]], dtype=torch.int32,
                        device=DEV)
    n = torch.tensor([4, 3, 4], dtype=torch.int32, device=DEV)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    nl = tg.kv_compact(k, v, L, path, n, d_err=err)
    torch.cuda.synchronize()
    assert int(err.item()) & OT.DERR_BAD_NODE
    assert list(nl.cpu().numpy()) == [8, 6, 2]
    assert torch.equal(k, k0) and torch.equal(v, v0)   # row 0 identity, rows 1-2 rejected


@pytest.mark.parametrize("n", [257, 300, 513, 1024])
def test_prune_selects_kept_set_of_monotone_trees(tg, n):
    """Trees whose scores never rise from parent to child (as expansion builds
    them): the kept set is the budget's largest keys, selected without ranking
    the rest; past 256 nodes this takes the per-wave bound paths for budgets
    up to 16 and up to 64.  Quantised log-probabilities make ties in cum
    (broken by depth, then id)."""
    g = W.rng([560, n])
    B, cap = 2, 1024
    t = OT.Tree.empty(B, cap)
    for b in range(B):
        par = W.uniform_parents(g, n)
        lp = (-np.round(np.abs(W.normal(g, (n,), 1.0)) * 4) / 4).astype(np.float32)
        cum = np.zeros(n, np.float32)
        for i in range(n):
            cum[i] = (cum[par[i]] if par[i] >= 0 else np.float32(0.0)) + lp[i]
        t.parent[b, :n] = par
        t.cum[b, :n] = cum
        t.token[b, :n] = g.integers(0, 1000, size=n)
        t.n_nodes[b] = n
    for B_ver in (1, 10, 16, 17, 40, 64):
        got, err = run_prune(tg, t, B_ver, cap + 1)
        assert err == 0
        for b in range(B):
            check_tree(got, t, b, B_ver, cap + 1)


def test_kv_compact_edges(tg):
    """An empty prefix is valid; a chain that repeats or decreases a slot, or
    that is longer than the path array, leaves its sequence untouched."""
    g = W.rng(561)
    B, Hkv, S, D = 4, 2, 16, 64
    k = torch.from_numpy(W.normal(g, (B, Hkv, S, D))).to(DEV)
    v = torch.from_numpy(W.normal(g, (B, Hkv, S, D))).to(DEV)
    k_in, v_in = k.cpu().numpy(), v.cpu().numpy()
    L = np.array([0, 2, 2, 2], np.int32)
    path = np.array([[0, 2, 5], [1, 1, 4], [2, 1, 4], [0, 1, 2]], np.int32)
    n = np.array([3, 3, 3, 4], np.int32)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    nl = tg.kv_compact(k, v, torch.from_numpy(L).to(DEV), torch.from_numpy(path).to(DEV),
                       torch.from_numpy(n).to(DEV), d_err=err)
    torch.cuda.synchronize()
    k2, v2, nl_o, err_o = OA.kv_compact(k_in, v_in, L, path, n)
    assert int(err.item()) == err_o and err_o & OT.DERR_BAD_NODE
    assert list(nl.cpu().numpy()) == list(nl_o) == [3, 2, 2, 2]
    assert np.array_equal(k.cpu().numpy(), k2) and np.array_equal(v.cpu().numpy(), v2)
