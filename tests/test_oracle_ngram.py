"""Pins for the n-gram small drafter oracle (CPU only): a hand-derived
context with back-off and fallback cases, an independent string-search
implementation of the suffix match, scipy log-softmax for the prefill cache,
an independent most-frequent-token count, and the expansion's invariants."""
import numpy as np
from scipy.special import log_softmax

import workloads as W
from oracle import ngram as NG
from oracle import tree as T


def test_hand_context_match_backoff_and_fallback():
    ctx = [1, 2, 3, 1, 2, 4]                       # a b c a b d
    assert NG.match_position(ctx, ctx, 3) == 5                  # root: itself
    assert NG.match_position(ctx, ctx + [1], 3) == 3            # "a": latest a
    assert NG.match_position(ctx, ctx + [1, 2], 3) == 4         # "a b": latest
    assert NG.match_position(ctx, ctx + [1, 2, 3], 3) == 2      # "a b c"
    assert NG.match_position(ctx, ctx + [9, 2, 3], 3) == 2      # back-off to "b c"
    assert NG.match_position(ctx, ctx + [9], 3) == -1           # unseen -> fallback
    logits = np.zeros((1, 6, 10), np.float32)
    _, _, fb, err = NG.ngram_cache(logits, np.array([ctx], np.int32), np.array([6]), 2)
    # counts: 1 x2, 2 x2, 3, 4 -> tie to token 1, last occurrence at 3
    assert err == 0 and int(fb[0]) == 3


def _rfind_match(ctx, prefix, n_max):
    """The same rule by string search: tokens as ',t,' words, str.rfind."""
    hay = "," + ",".join(map(str, ctx)) + ","
    for n in range(min(n_max, len(prefix)), 0, -1):
        needle = "," + ",".join(map(str, prefix[-n:])) + ","
        i = hay.rfind(needle)
        if i >= 0:
            return hay[:i + len(needle) - 1].count(",") - 1
    return -1


def test_match_equals_string_search():
    g = W.rng(900)
    for trial in range(300):
        L = int(g.integers(1, 40))
        V = int(g.integers(2, 6))
        ctx = [int(x) for x in g.integers(0, V, L)]
        path = [int(x) for x in g.integers(0, V + 1, int(g.integers(0, 5)))]
        n_max = int(g.integers(1, 6))
        assert NG.match_position(ctx, ctx + path, n_max) == _rfind_match(ctx, ctx + path, n_max)


def test_cache_is_the_top_m_log_softmax_and_fallback_count():
    g = W.rng(901)
    B, L, V, m = 2, 7, 50, 4
    logits = W.normal(g, (B, L, V), 2.0)
    ctx = g.integers(0, 6, (B, L)).astype(np.int32)
    ctx_len = np.array([7, 5], np.int32)
    tok, lp, fb, err = NG.ngram_cache(logits, ctx, ctx_len, m)
    assert err == 0
    ref = log_softmax(logits.astype(np.float64), axis=-1)
    for b in range(B):
        for i in range(L):
            order = sorted(range(V), key=lambda v: (-float(logits[b, i, v]), v))[:m]
            assert list(tok[b, i]) == order
            np.testing.assert_allclose(lp[b, i], ref[b, i, order], rtol=0, atol=2e-6)
        c = ctx[b, :ctx_len[b]].tolist()
        best = max(c.count(x) for x in set(c))
        tok_best = min(x for x in set(c) if c.count(x) == best)
        assert int(fb[b]) == len(c) - 1 - c[::-1].index(tok_best)


def test_expand_children_come_from_the_matched_cache_row():
    g = W.rng(902)
    B, L, V, m, K = 2, 30, 12, 5, 3
    ctx = g.integers(0, 4, (B, L)).astype(np.int32)
    ctx_len = np.array([30, 17], np.int32)
    tok, lp, fb, _ = NG.ngram_cache(W.normal(g, (B, L, V), 2.0), ctx, ctx_len, m)
    t = T.Tree.empty(B, 256)
    fr = np.full((B, 1), -1, np.int32)
    nf = np.ones(B, np.int32)
    for step in range(3):
        n0 = t.n_nodes.copy()
        t2, pos, nxt, nn, err = NG.expand_ngram(t, fr, nf, ctx, ctx_len, tok, lp, fb, K, 4, 3)
        assert err == 0
        for b in range(B):
            for f in range(int(nf[b])):
                v, j = int(fr[b, f]), int(pos[b, f])
                assert 0 <= j < int(ctx_len[b])
                if v == -1:
                    assert j == int(ctx_len[b]) - 1            # root matches itself
                for k in range(K):
                    nid = int(n0[b]) + f * K + k
                    assert int(t2.token[b, nid]) == int(tok[b, j, k])
                    assert t2.logp[b, nid] == lp[b, j, k]
                    assert int(t2.parent[b, nid]) == v
            kids = [T.node_key(t2.cum[b, i], t2.depth[b, i], i)
                    for i in range(int(n0[b]), int(t2.n_nodes[b]))]
            assert [k[2] for k in sorted(kids)[:int(nn[b])]] == list(nxt[b, :int(nn[b])])
        t, fr, nf = t2, nxt, nn


def test_empty_context_is_an_error_and_leaves_the_tree():
    t = T.Tree.empty(1, 16)
    z = np.zeros((1, 1, 2), np.int32)
    t2, pos, nxt, nn, err = NG.expand_ngram(t, np.full((1, 1), -1, np.int32), None,
                                            np.zeros((1, 1), np.int32), np.array([0]),
                                            z, z.astype(np.float32), np.array([-1]), 2, 2, 3)
    assert err == T.DERR_BAD_PREFIX and int(t2.n_nodes[0]) == 0 and int(nn[0]) == 0
