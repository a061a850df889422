"""Test inputs for the GPU parity tests.

Structures and random values come from ``workloads``; scored trees (edge and
path scores) are built with the oracle, so no expected value ever comes from
the GPU path.  Each builder states which workload it follows.
"""
from __future__ import annotations

import numpy as np

import workloads as W
from oracle import tree as OT

F32 = np.float32


# ----------------------------------------------------------------- trees

def scored_tree(seed, B, V, steps, width, K, std=2.0, cap=1024, row_seed=None):
    """Tree grown from the root by `steps` expansion steps (frontier `width`,
    `K` children per node), each frontier node's logits row drawn from the
    counter stream (row_seed, b * 1_000_000 + creation index + 1).
    Returns (tree, rows) with rows[b] = {node id: logits row} (-1 = root)."""
    row_seed = seed if row_seed is None else row_seed
    tree = OT.Tree.empty(B, cap)
    rows = [dict() for _ in range(B)]
    fr = np.full((B, 1), -1, np.int32)
    nf = np.ones(B, np.int32)
    for _ in range(steps):
        F = fr.shape[1]
        lg = np.full((B, F, V), -np.inf, np.float32)
        for b in range(B):
            for f in range(int(nf[b])):
                v = int(fr[b, f])
                r = W.node_logits(row_seed, b * 1_000_000 + v + 1, V, std)
                rows[b][v] = r
                lg[b, f] = r
        tree, _, nxt, nn, err = OT.expand(tree, lg, fr, nf, K, width)
        assert err == 0
        fr, nf = nxt, nn
    return tree, rows


def row_for(rows_b, v, seed, b, V, std):
    """The logits row of node v (drawn now if the node was never expanded)."""
    if v in rows_b:
        return rows_b[v]
    return W.node_logits(seed, b * 1_000_000 + v + 1, V, std)


def prune_tree(tree: OT.Tree, b: int, B_ver: int):
    """Alg. 3 prune of tree b; returns (kept original ids, new parent array)."""
    n = int(tree.n_nodes[b])
    out = OT.global_prune(tree.parent[b, :n], tree.cum[b, :n], n, B_ver)
    return out["kept"], out["parent"]


def subtree(tree: OT.Tree, b: int, kept, new_parent, cap):
    """Copy the kept nodes of tree b into a fresh single-tree Tree (new ids)."""
    t = OT.Tree.empty(1, cap)
    n = len(kept)
    t.parent[0, :n] = new_parent
    t.token[0, :n] = tree.token[b, kept]
    t.depth[0, :n] = tree.depth[b, kept]
    t.logp[0, :n] = tree.logp[b, kept]
    t.cum[0, :n] = tree.cum[b, kept]
    t.n_nodes[0] = n
    return t


def stack_trees(trees, cap):
    B = len(trees)
    out = OT.Tree.empty(B, cap)
    for b, t in enumerate(trees):
        for f in ("parent", "token", "depth", "logp", "cum", "visited"):
            getattr(out, f)[b] = getattr(t, f)[0, :cap]
        out.root_visited[b] = t.root_visited[0]
        out.n_nodes[b] = t.n_nodes[0]
    return out


def mark_visited_closed(g, tree: OT.Tree, p_root=0.5, p_node=0.5):
    """Random visited set closed under ancestors (what earlier middle steps
    leave behind: a node can only have entered a pool after its parent)."""
    for b in range(tree.parent.shape[0]):
        tree.root_visited[b] = int(g.random() < p_root)
        for v in range(int(tree.n_nodes[b])):
            p = int(tree.parent[b, v])
            par_vis = bool(tree.root_visited[b]) if p < 0 else bool(tree.visited[b, p])
            tree.visited[b, v] = int(par_vis and g.random() < p_node)
    return tree


# ------------------------------------------------------------- tolerances

def attn_close_f32(got, want, rel=1e-5):
    """fp32 bar: per output row, max |g - r| <= rel * max |r|."""
    g = got.reshape(-1, got.shape[-1]).astype(np.float64)
    r = want.reshape(-1, want.shape[-1])
    err = np.abs(g - r).max(axis=1)
    bound = rel * np.abs(r).max(axis=1)
    bad = np.nonzero(err > bound)[0]
    assert bad.size == 0, f"{bad.size} rows over the fp32 bar; worst {float((err / np.maximum(bound, 1e-300)).max()):.3g}x"


def attn_close_bf16(got, want, abs_tol=2e-2, rel_fro=1e-2):
    """bf16 bar: max abs error <= 2e-2 and tensor-relative Frobenius error <= 1e-2."""
    g = got.astype(np.float64)
    e_abs = float(np.abs(g - want).max())
    e_rel = float(np.linalg.norm(g - want) / max(np.linalg.norm(want), 1e-300))
    assert e_abs <= abs_tol, f"abs error {e_abs:.3g}"
    assert e_rel <= rel_fro, f"relative Frobenius error {e_rel:.3g}"
    return e_abs, e_rel


# ------------------------------------------------------------ device I/O

def tree_to_dev(tg, t: OT.Tree, device="cuda"):
    return tg.TreeState.from_host({f: getattr(t, f) for f in tg.TreeState.FIELDS},
                                  t.cap, device)


def tree_from_dev(ts) -> OT.Tree:
    h = ts.to_host()
    return OT.Tree(h["parent"], h["token"], h["depth"], h["logp"], h["cum"], h["visited"],
                   h["root_visited"], h["n_nodes"], cap=ts.cap)


def assert_tree_equal(got: OT.Tree, want: OT.Tree, what=""):
    """Bit-exact equality of every live slot and of the counters."""
    assert np.array_equal(got.n_nodes, want.n_nodes), f"{what} n_nodes"
    assert np.array_equal(got.root_visited, want.root_visited), f"{what} root_visited"
    for b in range(len(want.n_nodes)):
        n = int(want.n_nodes[b])
        for f in ("parent", "token", "depth", "visited"):
            assert np.array_equal(getattr(got, f)[b, :n], getattr(want, f)[b, :n]), \
                f"{what} tree {b} field {f}"
        for f in ("logp", "cum"):
            a = getattr(got, f)[b, :n].view(np.uint32)
            c = getattr(want, f)[b, :n].view(np.uint32)
            assert np.array_equal(a, c), f"{what} tree {b} field {f} (bitwise)"
