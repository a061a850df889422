"""Seeded synthetic inputs for the tree-verify and tree-expand workloads.

This module is shared by the tests, the benchmark and the smoke check.  It holds
random draws and tree *structures* only: no softmax, no score arithmetic, no
selection and no pruning.  Scores (edge log-probabilities, cumulative path
scores) are never produced here; whoever needs a scored tree builds it with the
method itself (the GPU path in the benchmark, the oracle in the tests).

Conventions shared with the library:
  * a draft tree of ``n`` nodes is a parent array ``parent[i] in [-1, i-1]``;
    ``-1`` means the node hangs directly under the root (the verified prefix);
  * nodes are numbered so that a parent always precedes its children;
  * logits rows are indexed ``0`` = root, ``1 + i`` = node ``i``.

Every generator takes an explicit ``numpy.random.Generator`` (PCG64) or a seed.
"""
from __future__ import annotations

import numpy as np

__all__ = [
    "rng",
    "normal",
    "node_logits",
    "uniform_parents",
    "level_tree",
    "expansion_shaped_tree",
    "children_lists",
    "node_depths",
    "distinct_sibling_tokens",
    "greedy_match_random_child",
    "greedy_match_first_child",
    "verify_layout_with_root",
    "token_stream",
    "CONFIGS",
]


def rng(seed) -> np.random.Generator:
    """PCG64 generator; ``seed`` may be an int or a sequence of ints."""
    return np.random.Generator(np.random.PCG64(seed))


def normal(g: np.random.Generator, shape, std: float = 1.0) -> np.ndarray:
    """fp32 array of i.i.d. N(0, std^2) draws (std = standard deviation)."""
    return (g.standard_normal(size=shape, dtype=np.float64) * std).astype(np.float32)


def node_logits(seed: int, index: int, vocab: int, std: float) -> np.ndarray:
    """One logits row from a counter-based stream keyed by (seed, index).

    The same (seed, index) always gives the same row, independent of the order
    in which rows are requested, so a tree built on the GPU and one built on
    the CPU can draw identical rows for identical node creation indices.
    """
    g = rng([int(seed), int(index)])
    return normal(g, (vocab,), std)


def uniform_parents(g: np.random.Generator, n: int) -> np.ndarray:
    """parent[i] uniform in [-1, i-1] (the 'tiny' workload's random forest)."""
    return np.array([g.integers(-1, i) for i in range(n)], dtype=np.int32)


def level_tree(g: np.random.Generator, n_nodes: int, n_levels: int,
               max_children: int) -> np.ndarray:
    """Random tree with exactly ``n_levels`` levels below the root.

    Level sizes are a seeded random composition of ``n_nodes`` (every level has
    at least one node, the root and every node have at most ``max_children``
    children).  Each node picks its parent uniformly among the previous level's
    nodes that still have room.  Nodes are numbered level by level; level-1 nodes
    have parent -1.
    """
    if n_levels < 1 or n_nodes < n_levels:
        raise ValueError("need n_nodes >= n_levels >= 1")
    for _ in range(10000):
        cuts = np.sort(g.choice(np.arange(1, n_nodes), size=n_levels - 1, replace=False))
        sizes = np.diff(np.concatenate([[0], cuts, [n_nodes]])).astype(int)
        ok = sizes[0] <= max_children and all(
            sizes[k + 1] <= sizes[k] * max_children for k in range(n_levels - 1))
        if ok:
            break
    else:  # pragma: no cover - only for infeasible arguments
        raise ValueError("could not draw a feasible level composition")
    parent = np.empty(n_nodes, dtype=np.int32)
    start = 0
    prev = [-1]
    for size in sizes:
        room = {p: max_children for p in prev}
        level = list(range(start, start + size))
        for v in level:
            open_ = [p for p in prev if room[p] > 0]
            p = open_[g.integers(0, len(open_))]
            room[p] -= 1
            parent[v] = p
        prev = level
        start += size
    return parent


def expansion_shaped_tree(g: np.random.Generator, n_nodes: int, n_levels: int,
                          branching: int, frontier: int) -> np.ndarray:
    """Tree shaped like a pruned top-``branching`` / frontier-``frontier`` expansion.

    Level 1 holds at most ``branching`` children of the root.  Only the first
    ``frontier`` nodes of a level (the ones an expansion would have picked) may
    have children, at most ``branching`` each.  Level sizes shrink with depth, as
    a score-pruned tree's do.  Structure only; nodes numbered level by level.
    """
    first = min(branching, n_nodes - (n_levels - 1))
    for _ in range(10000):
        w = 0.65 ** np.arange(n_levels - 1)
        rest = 1 + g.multinomial(n_nodes - first - (n_levels - 1), w / w.sum())
        sizes = np.concatenate([[first], rest]).astype(int)
        ok = True
        for k in range(n_levels - 1):
            cap = min(frontier, sizes[k]) * branching
            ok = ok and sizes[k + 1] <= cap
        if ok:
            break
    else:  # pragma: no cover
        raise ValueError("could not draw a feasible level composition")
    parent = np.empty(n_nodes, dtype=np.int32)
    start = 0
    prev = [-1]
    for size in sizes:
        room = {p: branching for p in prev}
        level = list(range(start, start + size))
        for v in level:
            open_ = [p for p in prev if room[p] > 0]
            p = open_[g.integers(0, len(open_))]
            room[p] -= 1
            parent[v] = p
        prev = level[:frontier]
        start += size
    return parent


def children_lists(parent: np.ndarray):
    """children[v+1] = ids of v's children in id order (index 0 = root)."""
    ch = [[] for _ in range(len(parent) + 1)]
    for i, p in enumerate(parent):
        ch[int(p) + 1].append(i)
    return ch


def node_depths(parent: np.ndarray) -> np.ndarray:
    """Depth of each node (root = 0, so a node with parent -1 has depth 1)."""
    d = np.zeros(len(parent), dtype=np.int32)
    for i, p in enumerate(parent):
        d[i] = 1 if p < 0 else d[p] + 1
    return d


def distinct_sibling_tokens(g: np.random.Generator, parent: np.ndarray,
                            vocab: int) -> np.ndarray:
    """A token per node, distinct among siblings, uniform over the vocabulary."""
    tok = np.empty(len(parent), dtype=np.int32)
    for kids in children_lists(parent):
        if kids:
            tok[kids] = g.choice(vocab, size=len(kids), replace=False)
    return tok


def _other_token(g, vocab, avoid):
    while True:
        t = int(g.integers(0, vocab))
        if t not in avoid:
            return t


def greedy_match_random_child(g: np.random.Generator, parent: np.ndarray,
                              token: np.ndarray, vocab: int, p: float) -> np.ndarray:
    """Target greedy tokens, rows 0 = root and 1 + i = node i.

    For a node with children, with probability ``p`` the greedy token is the
    token of a uniformly chosen child, otherwise a uniform token that none of
    its children carries.  Leaves get a uniform token.
    """
    kids = children_lists(parent)
    out = np.empty(len(parent) + 1, dtype=np.int32)
    for r, ks in enumerate(kids):
        toks = {int(token[c]) for c in ks}
        if ks and g.random() < p:
            out[r] = token[ks[g.integers(0, len(ks))]]
        else:
            out[r] = _other_token(g, vocab, toks)
    return out


def greedy_match_first_child(g: np.random.Generator, parent: np.ndarray,
                             token: np.ndarray, vocab: int, p: float,
                             preferred=None) -> np.ndarray:
    """Target greedy tokens that agree with one designated child per node.

    ``preferred[r]`` is the designated child of row ``r`` (0 = root, 1 + i =
    node i); by default it is the first child in id order.  With probability
    ``p`` the greedy token is that child's token, otherwise a uniform token
    different from it.  Leaves get a uniform token.
    """
    kids = children_lists(parent)
    out = np.empty(len(parent) + 1, dtype=np.int32)
    for r, ks in enumerate(kids):
        if not ks:
            out[r] = g.integers(0, vocab)
            continue
        c = ks[0] if preferred is None else int(preferred[r])
        if g.random() < p:
            out[r] = token[c]
        else:
            out[r] = _other_token(g, vocab, {int(token[c])})
    return out


def verify_layout_with_root(parent: np.ndarray) -> np.ndarray:
    """Verify-call layout with the root as node 0: draft node i -> verify node i+1."""
    vp = np.empty(len(parent) + 1, dtype=np.int32)
    vp[0] = -1
    vp[1:] = parent + 1
    return vp


def token_stream(g: np.random.Generator, length: int, vocab: int, n_phrases: int = 32,
                 phrase_len=(2, 8), p_phrase: float = 0.6) -> np.ndarray:
    """Synthetic prompt: a bank of random phrases (lengths in phrase_len) that
    recur through the stream, interleaved with single random tokens, so that
    n-grams of every length repeat as in real prompts.  int32 [length]."""
    lo, hi = phrase_len
    bank = [g.integers(0, vocab, int(g.integers(lo, hi + 1))) for _ in range(n_phrases)]
    out = []
    while len(out) < length:
        if g.random() < p_phrase:
            out.extend(int(x) for x in bank[int(g.integers(0, n_phrases))])
        else:
            out.append(int(g.integers(0, vocab)))
    return np.asarray(out[:length], dtype=np.int32)


# Shapes of the five workloads (the sizes the paper's setting implies; see the
# recipes above for how each input is drawn).
CONFIGS = {
    "tiny": dict(B=1, Hq=4, Hkv=4, D=64, L=128, N=16, dtype="f32", vocab=1000,
                 logit_std=2.0, topk=4, frontier=8, seed=1001),
    "llama8b": dict(B=1, Hq=32, Hkv=8, D=128, L=2048, N=64, dtype="bf16",
                    vocab=128256, logit_std=3.0, topk=8, frontier=10, depth=6,
                    qkv_scale=1.0 / np.sqrt(128.0), seed=1002),
    "longctx": dict(B=4, Hq=32, Hkv=8, D=128, L=8192, N=128, dtype="bf16",
                    depth=10, branching=8, seed=1003),
    "twodrafter": dict(B=8, vocab=128256, logit_std=3.0, frontier_rows=64,
                       topk=10, N=60, tree_nodes=256, rho=0.8, seed=1004),
    "llama70b": dict(B=8, Hq=64, Hkv=8, D=128, L=32768, N=256, dtype="bf16",
                     depth=12, branching=8, seed=1005),
}
