"""GPU parity of the n-gram small drafter: tg_ngram_cache (prefill top-m
cache and fallback position) and tg_tree_expand_ngram (suffix match with
back-off, expansion from the matched cache row).

Cache: tokens and fallback positions bit for bit; log-probabilities within
1e-5 * max(1, |lse|) (each is fl(x - lse) with the GPU's fp32 lse).  Expansion
is run by the oracle on the GPU's own cache, so every integer output and every
stored fp32 score must agree bit for bit.
"""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import ngram as NG
from oracle import tree as OT
from tests import _cases as C

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _d(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def _cache_close(tg, logits, ctx, clen, m, rows=None):
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    tok, lp, fb = tg.ngram_cache(_d(logits), _d(ctx), _d(clen), m, d_err=err)
    torch.cuda.synchronize()
    tok, lp, fb = tok.cpu().numpy(), lp.cpu().numpy(), fb.cpu().numpy()
    B, L, V = logits.shape
    if rows is None:
        t_o, lp_o, fb_o, err_o = NG.ngram_cache(logits, ctx, clen, m)
        assert np.array_equal(tok, t_o)
        np.testing.assert_allclose(lp, lp_o, rtol=0, atol=1e-5 * max(1.0, float(np.abs(lp_o[np.isfinite(lp_o)]).max())))
        assert np.array_equal(fb, fb_o)
        assert int(err.item()) == err_o
    else:   # sampled rows at full size
        for b, i in rows:
            t_o, lp_o, _, _ = NG.ngram_cache(logits[b:b + 1, i:i + 1], ctx[b:b + 1, i:i + 1],
                                             np.array([1]), m)
            assert np.array_equal(tok[b, i], t_o[0, 0])
            np.testing.assert_allclose(lp[b, i], lp_o[0, 0], rtol=0, atol=1e-4)
        fb_o, _ = NG.fallback_position(ctx, clen, V)
        assert np.array_equal(fb, fb_o)
    return tok, lp, fb


@pytest.mark.parametrize("seed", range(4))
def test_cache_small(tg, seed):
    g = W.rng(910 + seed)
    B, L, V, m = int(g.integers(1, 4)), int(g.integers(1, 70)), [50, 1000, 4097, 9000][seed], \
        int(g.integers(1, 9))
    logits = np.round(W.normal(g, (B, L, V), 2.0), 1).astype(np.float32)   # ties
    if seed == 1:
        logits[0, 0, 3] = np.nan
    ctx = np.stack([W.token_stream(g, L, 12) for _ in range(B)])
    clen = g.integers(0, L + 1, B).astype(np.int32)
    _cache_close(tg, logits, ctx, clen, m)


def run_expand(tg, tree_h, fr, nf, ctx, clen, tok, lp, fb, K, N, n_max):
    ts = C.tree_to_dev(tg, tree_h)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    nx, nn, mp = tg.expand_ngram(ts, _d(fr), None if nf is None else _d(nf), _d(ctx), _d(clen),
                                 _d(tok), _d(lp), _d(fb), K, N, n_max, d_err=err)
    torch.cuda.synchronize()
    got = C.tree_from_dev(ts)
    want, mp_o, nx_o, nn_o, err_o = NG.expand_ngram(tree_h, fr, nf, ctx, clen, tok, lp, fb, K,
                                                    N, n_max)
    C.assert_tree_equal(got, want, "ngram expand")
    assert np.array_equal(mp.cpu().numpy(), mp_o)
    assert np.array_equal(nx.cpu().numpy(), nx_o) and np.array_equal(nn.cpu().numpy(), nn_o)
    assert int(err.item()) == err_o
    return got, nx.cpu().numpy(), nn.cpu().numpy(), mp.cpu().numpy()


@pytest.mark.parametrize("seed", range(5))
def test_expand_chain_small(tg, seed):
    """Four small steps from the root with the GPU's own cache (seed 4: a
    6000-token prompt, past what the kernel stages in LDS)."""
    g = W.rng(920 + seed)
    B, L, V, m = int(g.integers(1, 4)), int(g.integers(8, 200)), 300, 6
    if seed == 4:
        B, L = 2, 6000
    K, N, n_max = int(g.integers(1, m + 1)), int(g.integers(1, 12)), int(g.integers(1, 6))
    ctx = np.stack([W.token_stream(g, L, 20) for _ in range(B)])
    clen = g.integers(1, L + 1, B).astype(np.int32)
    logits = W.normal(g, (B, L, V), 2.0)
    tok, lp, fb = _cache_close(tg, logits, ctx, clen, m)
    t = OT.Tree.empty(B, 1024)
    fr, nf = np.full((B, 1), -1, np.int32), np.ones(B, np.int32)
    matched = 0
    for step in range(4):
        t, fr, nf, mp = run_expand(tg, t, fr, nf, ctx, clen, tok, lp, fb, K, N, n_max)
        matched += int((mp >= 0).sum())
    assert matched > 0


def test_fallback_and_errors(tg):
    """Tokens never seen in the context take the fallback row; an empty
    context and a bad frontier id leave their trees unchanged."""
    ctx = np.array([[1, 2, 3, 1, 2, 4, 0, 0], [5, 5, 6, 0, 0, 0, 0, 0]], np.int32)
    clen = np.array([6, 0], np.int32)
    g = W.rng(930)
    logits = W.normal(g, (2, 8, 16), 2.0)
    tok, lp, fb = _cache_close(tg, logits, ctx, clen, 3)
    t = OT.Tree.empty(2, 64)
    t.parent[0, :2], t.token[0, :2], t.depth[0, :2], t.n_nodes[0] = [-1, 0], [9, 9], [1, 2], 2
    fr = np.array([[1, -1, 0], [-1, -1, -1]], np.int32)
    got, nx, nn, mp = run_expand(tg, t, fr, None, ctx, clen, tok, lp, fb, 2, 4, 3)
    assert list(mp[0]) == [3, 5, 3]            # fallback (token 1 at 3), root, fallback
    assert int(got.n_nodes[1]) == 0 and int(nn[1]) == 0
    fr_bad = np.array([[7, -1, -1], [-1, -1, -1]], np.int32)
    run_expand(tg, t, fr_bad, None, ctx, np.array([6, 3], np.int32), tok, lp, fb, 2, 4, 3)


def test_llama8b_shape_prefill_and_steps(tg):
    """Prefill cache over a 2048-token synthetic prompt at V = 128256 (rows
    sampled for the oracle), then the small steps of a turn: frontier 10,
    top-8 children, n_max 4."""
    g = W.rng(940)
    L, V, m = 2048, 128256, 8
    ctx = W.token_stream(g, L, V, n_phrases=64)[None]
    clen = np.array([L], np.int32)
    logits = torch.empty((1, L, V), dtype=torch.float32, device=DEV)
    host = {}
    for r0 in range(0, L, 128):
        blk = W.normal(W.rng([941, r0]), (128, V), 3.0)
        logits[0, r0:r0 + 128] = torch.from_numpy(blk).to(DEV)
        if r0 in (0, 1024, 1920):
            host[r0] = blk
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    tok, lp, fb = tg.ngram_cache(logits, _d(ctx), _d(clen), m, d_err=err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    tok_h, lp_h, fb_h = tok.cpu().numpy(), lp.cpu().numpy(), fb.cpu().numpy()
    for r0, blk in host.items():
        for i in (0, 77, 127):
            t_o, lp_o, _, _ = NG.ngram_cache(blk[i][None, None], ctx[:, :1], np.array([1]), m)
            assert np.array_equal(tok_h[0, r0 + i], t_o[0, 0])
            np.testing.assert_allclose(lp_h[0, r0 + i], lp_o[0, 0], rtol=0, atol=1e-4)
    fb_o, _ = NG.fallback_position(ctx, clen, V)
    assert np.array_equal(fb_h, fb_o)
    t = OT.Tree.empty(1, 512)
    fr, nf = np.full((1, 1), -1, np.int32), np.ones(1, np.int32)
    for step in range(3):
        t, fr, nf, mp = run_expand(tg, t, fr, nf, ctx, clen, tok_h, lp_h, fb_h, 8, 10, 4)


@pytest.mark.parametrize("n_max", [1, 2, 4, 5, 16])
@pytest.mark.parametrize("L", [300, 4096, 4097])
def test_match_paths(tg, n_max, L):
    """The match scan's three paths against the oracle: n-grams up to 4
    tokens matched in registers, longer ones extended through LDS, and
    prompts past 4096 tokens scanned from global memory.  A 30-token
    vocabulary makes long repeated n-grams common."""
    g = W.rng([950, n_max, L])
    B, V, m, K, N = 2, 40, 4, 2, 6
    ctx = np.stack([W.token_stream(g, L, 30) for _ in range(B)])
    clen = np.array([L, L - 7], np.int32)
    logits = W.normal(g, (B, L, V), 2.0)
    tok, lp, fb = _cache_close(tg, logits, ctx, clen, m)
    t = OT.Tree.empty(B, 256)
    fr, nf = np.full((B, 1), -1, np.int32), np.ones(B, np.int32)
    lens = []
    for step in range(3):
        t, fr, nf, mp = run_expand(tg, t, fr, nf, ctx, clen, tok, lp, fb, K, N, n_max)
        lens.append(mp)
    assert all((x >= 0).any() for x in lens)


@pytest.mark.parametrize("K", [4, 8])
def test_largest_frontier_and_suffix(tg, K):
    """The largest documented call shape: F = 1024 frontier slots (the root,
    repeated), n_max = 16 and F*K = 4096 children (filling a 4096-slot tree)
    or 8192 (past the capacity: CAPACITY, the tree unchanged).  The suffixes
    and the child keys share one LDS region, so every documented combination
    launches."""
    g = W.rng(960 + K)
    B, L, V, m, F = 1, 96, 300, 8, 1024
    ctx = np.stack([W.token_stream(g, L, 20)])
    clen = np.array([L], np.int32)
    logits = W.normal(g, (B, L, V), 2.0)
    tok, lp, fb = _cache_close(tg, logits, ctx, clen, m)
    t = OT.Tree.empty(B, 4096)
    fr, nf = np.full((B, F), -1, np.int32), np.array([F], np.int32)
    got, nx, nn, mp = run_expand(tg, t, fr, nf, ctx, clen, tok, lp, fb, K, 64, 16)
    assert int(got.n_nodes[0]) == (F * K if F * K <= 4096 else 0)


def _hand_cache():
    """ctx = [7, 2, 3, 1, 2, 4]; cache row j: two candidates with exactly
    representable scores -(j+1)/4 and -(j+1)/2 (the oracle pins work this
    case by hand)."""
    ctx = np.array([[7, 2, 3, 1, 2, 4]], np.int32)
    tok = np.array([[[10, 20], [11, 21], [12, 22], [13, 23], [14, 24], [3, 7]]], np.int32)
    lp = np.array([[[-(j + 1) / 4, -(j + 1) / 2] for j in range(6)]], np.float32)
    return ctx, np.array([6], np.int32), tok, lp


def test_hand_expansion_fills_the_tree_then_overflows(tg):
    """Root step, a step that fills the 6-slot tree exactly, one that would
    overflow it (CAPACITY), and a frontier id equal to the node count."""
    ctx, clen, tok, lp = _hand_cache()
    fb = np.array([4], np.int32)
    t = OT.Tree.empty(1, 6)
    t, fr, nf, mp = run_expand(tg, t, np.full((1, 1), -1, np.int32), None, ctx, clen, tok, lp,
                               fb, 2, 2, 3)
    assert list(mp[0]) == [5]
    t, fr, nf, mp = run_expand(tg, t, fr, nf, ctx, clen, tok, lp, fb, 2, 3, 3)
    assert list(mp[0]) == [2, 0] and int(t.n_nodes[0]) == 6
    assert list(t.cum[0, 2:6]) == [-2.25, -3.0, -3.25, -3.5]
    t3, _, nn3, _ = run_expand(tg, t, np.array([[2]], np.int32), None, ctx, clen, tok, lp, fb,
                               2, 3, 3)
    assert int(t3.n_nodes[0]) == 6 and int(nn3[0]) == 0
    t4 = OT.Tree.empty(1, 16)
    t4.parent[0, :2], t4.token[0, :2], t4.depth[0, :2], t4.n_nodes[0] = [-1, 0], [3, 3], [1, 2], 2
    t5, _, nn5, _ = run_expand(tg, t4, np.array([[2]], np.int32), None, ctx, clen, tok, lp, fb,
                               2, 3, 3)
    assert int(t5.n_nodes[0]) == 2 and int(nn5[0]) == 0


@pytest.mark.parametrize("fbv", [0, -1, 6])
def test_fallback_positions_at_the_edges(tg, fbv):
    """A node whose token the context never holds takes fallback_pos: 0 is a
    position; -1 and L are not (BAD_NODE, then position L - 1)."""
    ctx, clen, tok, lp = _hand_cache()
    t = OT.Tree.empty(1, 16)
    t.parent[0, 0], t.token[0, 0], t.depth[0, 0], t.n_nodes[0] = -1, 9, 1, 1
    t.cum[0, 0] = t.logp[0, 0] = -1.0
    _, _, _, mp = run_expand(tg, t, np.array([[0]], np.int32), None, ctx, clen, tok, lp,
                             np.array([fbv], np.int32), 2, 2, 3)
    assert int(mp[0, 0]) == (0 if fbv == 0 else 5)
