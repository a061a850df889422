"""Invariants of the hot path checked on the GPU, beyond the oracle parity of
each call:

  * relabelling equivariance of tree-verify attention (Alg. 3 mask): any
    parents-first renumbering of the draft nodes, applied to the parent array,
    the query rows and the tree's key/value slots, permutes the outputs the
    same way (both bf16 kernels and the fp32 one);
  * distribution preservation at temperature 0 (Sec. 3.2): rounds of
    accept + bonus on the GPU, over random draft trees that sometimes contain
    the target's continuation, reproduce exactly a deterministic toy target's
    own greedy sequence;
  * many seeds: 100 seeded random cases each for expand, rescore + graft and
    accept, bit-exact against the oracle by the split check.
"""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import tree as OT
from oracle.attention import path_of, tree_verify_attention_fast
from tests import _cases as C
from tests.test_gpu_tree import run_accept, run_expand, run_rescore

pytestmark = pytest.mark.gpu
DEV = "cuda"


# ------------------------------------------------------- relabelling

def _topo_relabel(g, parent):
    """A random parents-first order of the nodes: perm[new] = old."""
    n = len(parent)
    kids = W.children_lists(parent)
    ready, perm = list(kids[0]), []
    while ready:
        v = ready.pop(int(g.integers(0, len(ready))))
        perm.append(v)
        ready += kids[v + 1]
    assert sorted(perm) == list(range(n))
    return np.array(perm)


@pytest.mark.parametrize("case", ["mfma", "pingpong", "f32"])
def test_attention_relabelling_equivariance(tg, case):
    g = W.rng({"mfma": 61, "pingpong": 62, "f32": 63}[case])
    if case == "pingpong":      # >= 256 rows per KV head and >= 4096 prefix rows
        B, N, Hq, Hkv, D, L = 2, 90, 16, 2, 128, 4100
    else:
        B, N, Hq, Hkv, D, L = 2, 90, 8, 2, 64, 300
    dt = torch.float32 if case == "f32" else torch.bfloat16
    S = L + N + 4
    parent = np.stack([W.uniform_parents(g, N) for _ in range(B)])
    q = torch.from_numpy(W.normal(g, (B, N, Hq, D))).to(DEV).to(dt)
    k = torch.from_numpy(W.normal(g, (B, Hkv, S, D))).to(DEV).to(dt)
    v = torch.from_numpy(W.normal(g, (B, Hkv, S, D))).to(DEV).to(dt)
    plen = torch.full((B,), L, dtype=torch.int32, device=DEV)
    base = tg.verify_attention(q, k, v, torch.from_numpy(parent).to(DEV), plen, D ** -0.5)
    # relabel each tree: new node j = old node perm[j]
    q2, k2, v2 = q.clone(), k.clone(), v.clone()
    par2 = np.empty_like(parent)
    perms = []
    for b in range(B):
        perm = _topo_relabel(g, parent[b])
        inv = np.empty(N, np.int64)
        inv[perm] = np.arange(N)
        par2[b] = [-1 if parent[b, o] < 0 else inv[parent[b, o]] for o in perm]
        assert all(par2[b, j] < j for j in range(N))
        idx = torch.from_numpy(perm).to(DEV)
        q2[b] = q[b, idx]
        k2[b, :, L:L + N] = k[b, :, L + idx]
        v2[b, :, L:L + N] = v[b, :, L + idx]
        perms.append(idx)
    out2 = tg.verify_attention(q2, k2, v2, torch.from_numpy(par2.astype(np.int32)).to(DEV), plen,
                               D ** -0.5)
    torch.cuda.synchronize()
    back = torch.stack([out2[b][torch.argsort(perms[b])] for b in range(B)])
    a, b_ = base.float().cpu().numpy(), back.float().cpu().numpy()
    want = tree_verify_attention_fast(q.float().cpu().numpy(), k.float().cpu().numpy(),
                                      v.float().cpu().numpy(), parent, np.full(B, L), D ** -0.5)
    if case == "f32":
        C.attn_close_f32(b_, want)
        C.attn_close_f32(a, want)
        np.testing.assert_allclose(b_, a, rtol=0, atol=1e-5 * float(np.abs(a).max()))
    else:
        C.attn_close_bf16(b_, want)
        C.attn_close_bf16(a, want)
        # the relabelled call differs only in the order of the tree keys
        assert float(np.abs(b_ - a).max()) <= 4e-3


# ------------------------------------------- temperature-0 preservation

def _toy_target(seq):
    """Deterministic toy target: the next token is a hash of the whole
    prefix (FNV-1a over the token ids), modulo a 50-token vocabulary."""
    h = 2166136261
    for t in seq:
        h = ((h ^ int(t)) * 16777619) & 0xFFFFFFFF
    return h % 50


def test_accept_rounds_reproduce_the_target_greedy_sequence(tg):
    """Eight sequences decode in lock step: each round drafts a random tree
    per sequence (with probability 1/2 the target's continuation is planted
    along one chain), the target's greedy token after every node is computed
    on the host, tg_tree_accept picks the accepted path and the bonus token on
    the GPU, and the sequence grows by them.  After 150+ tokens each sequence
    equals the toy target's own greedy continuation of its prompt."""
    g = W.rng(78)
    B, cap = 8, 40
    seqs = [[1, 2, b] for b in range(B)]
    prompts = [list(s) for s in seqs]
    rounds = 0
    while min(len(s) for s in seqs) < 150:
        parent = np.full((B, cap), -1, np.int32)
        token = np.zeros((B, cap), np.int32)
        greedy = np.zeros((B, cap + 1), np.int32)
        n = np.zeros(B, np.int32)
        for b in range(B):
            nb = int(g.integers(1, cap + 1))
            par = W.uniform_parents(g, nb)
            tok = g.integers(0, 50, size=nb).astype(np.int32)
            if g.random() < 0.5:
                v, ctx = -1, list(seqs[b])
                for i in range(nb):
                    if par[i] == v:
                        tok[i] = _toy_target(ctx)
                        ctx.append(int(tok[i]))
                        v = i
            parent[b, :nb], token[b, :nb], n[b] = par, tok, nb
            greedy[b, 0] = _toy_target(seqs[b])
            for i in range(nb):
                greedy[b, i + 1] = _toy_target(seqs[b] + [int(tok[u]) for u in path_of(par, i)])
        A = tg.accept(*(torch.from_numpy(x).to(DEV) for x in (parent, token, n, greedy)), cap)
        torch.cuda.synchronize()
        A_, path, bonus = (t.cpu().numpy() for t in A)
        for b in range(B):
            seqs[b] += [int(token[b, u]) for u in path[b, :A_[b]]] + [int(bonus[b])]
        rounds += 1
    for b in range(B):
        ref = list(prompts[b])
        while len(ref) < len(seqs[b]):
            ref.append(_toy_target(ref))
        assert seqs[b] == ref, b
    assert rounds < 150        # trees were accepted beyond the bonus token


# ------------------------------------------------------------ many seeds

@pytest.mark.parametrize("block", range(4))
def test_expand_100_seeds(tg, block):
    for seed in range(25 * block, 25 * block + 25):
        g = W.rng([4000, seed])
        B = int(g.integers(1, 4))
        V = int(g.integers(20, 3000))
        K = int(g.integers(1, min(V, 16) + 1))
        F = int(g.integers(1, 12))
        N = int(g.integers(1, F * K + 5))
        base, _ = C.scored_tree(5000 + seed, B, 40, steps=2, width=3, K=3, cap=512)
        fr = np.stack([g.integers(-1, int(base.n_nodes[b]), size=F) for b in range(B)]
                      ).astype(np.int32)
        nf = g.integers(0, F + 1, size=B).astype(np.int32)
        logits = W.normal(g, (B, F, V), float(g.uniform(0.5, 4.0)))
        if seed % 5 == 0:                      # quantised: ties in logits and in cum
            logits = (np.round(logits * 2) / 2).astype(np.float32)
        run_expand(tg, base, logits, fr, nf, K, N)


@pytest.mark.parametrize("block", range(4))
def test_rescore_graft_100_seeds(tg, block):
    for seed in range(25 * block, 25 * block + 25):
        g = W.rng([4100, seed])
        B = int(g.integers(1, 3))
        V = int(g.integers(30, 800))
        tree, _ = C.scored_tree(6000 + seed, B, V, steps=int(g.integers(1, 4)),
                                width=int(g.integers(1, 5)), K=int(g.integers(1, 5)), cap=256)
        C.mark_visited_closed(g, tree, p_root=0.3, p_node=0.4)
        R = int(tree.n_nodes.max()) + 1
        strong = W.normal(g, (B, R, V), 2.0)
        Wsel = int(g.integers(1, 12))
        M = int(g.integers(1, min(V, 8) + 1))
        run_rescore(tg, tree, strong, Wsel, M, N=int(g.integers(1, 9)))


@pytest.mark.parametrize("block", range(4))
def test_accept_100_seeds(tg, block):
    for seed in range(25 * block, 25 * block + 25):
        g = W.rng([4200, seed])
        B, cap = int(g.integers(1, 5)), int(g.integers(1, 80))
        parent = np.full((B, cap), -1, np.int32)
        token = np.zeros((B, cap), np.int32)
        greedy = np.zeros((B, cap + 1), np.int32)
        n = g.integers(0, cap + 1, size=B).astype(np.int32)
        V = 4 if seed % 3 == 0 else 100           # a tiny vocabulary makes duplicate siblings
        for b in range(B):
            nb = int(n[b])
            par = W.uniform_parents(g, nb)
            parent[b, :nb] = par
            token[b, :nb] = g.integers(0, V, size=nb)
            full_par = np.concatenate([par, np.full(cap - nb, -1, np.int32)])
            greedy[b] = W.greedy_match_random_child(g, full_par, token[b], V + 1, 0.7)
        run_accept(tg, parent, token, n, greedy, int(g.integers(1, cap + 2)))
