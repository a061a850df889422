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


def _hand_cache():
    """ctx = [7, 2, 3, 1, 2, 4]; the cache row at position j holds two
    candidates with exactly representable scores, -(j+1)/4 and -(j+1)/2."""
    ctx = np.array([[7, 2, 3, 1, 2, 4]], np.int32)
    tok = np.array([[[10, 20], [11, 21], [12, 22], [13, 23], [14, 24], [3, 7]]], np.int32)
    lp = np.array([[[-(j + 1) / 4, -(j + 1) / 2] for j in range(6)]], np.float32)
    return ctx, np.array([6], np.int32), tok, lp


def test_hand_expansion_values_capacity_and_bad_frontier():
    """Two steps worked by hand (cum is the exact sum of the scores on the
    path, depth the path length); the second fills the 6-slot tree exactly,
    a third would overflow it (CAPACITY, unchanged), a frontier id equal to
    the node count is BAD_NODE."""
    ctx, clen, tok, lp = _hand_cache()
    fb = np.array([4], np.int32)
    t = T.Tree.empty(1, 6)
    # step 1: the root's prefix is the context itself: latest "1 2 4" ends at 5
    t1, pos, nxt, nn, err = NG.expand_ngram(t, np.full((1, 1), -1, np.int32), None, ctx, clen,
                                            tok, lp, fb, 2, 2, 3)
    assert err == 0 and list(pos[0]) == [5] and list(nxt[0]) == [0, 1] and int(nn[0]) == 2
    assert list(t1.token[0, :2]) == [3, 7] and list(t1.parent[0, :2]) == [-1, -1]
    assert list(t1.depth[0, :2]) == [1, 1] and list(t1.cum[0, :2]) == [-1.5, -3.0]
    # step 2: node 0 (token 3) matches "3" at 2; node 1 (token 7) matches "7" at 0
    t2, pos, nxt, nn, err = NG.expand_ngram(t1, nxt, nn, ctx, clen, tok, lp, fb, 2, 3, 3)
    assert err == 0 and list(pos[0]) == [2, 0] and int(t2.n_nodes[0]) == 6
    assert list(t2.token[0, 2:6]) == [12, 22, 10, 20]
    assert list(t2.parent[0, 2:6]) == [0, 0, 1, 1] and list(t2.depth[0, 2:6]) == [2, 2, 2, 2]
    assert list(t2.logp[0, 2:6]) == [-0.75, -1.5, -0.25, -0.5]
    assert list(t2.cum[0, 2:6]) == [-2.25, -3.0, -3.25, -3.5]
    assert list(nxt[0]) == [2, 3, 4] and int(nn[0]) == 3
    # step 3 would append 2 more to a full tree
    t3, _, nxt3, nn3, err = NG.expand_ngram(t2, np.array([[2]], np.int32), None, ctx, clen,
                                            tok, lp, fb, 2, 3, 3)
    assert err == T.DERR_CAPACITY and int(nn3[0]) == 0 and int(t3.n_nodes[0]) == 6
    # a partial overflow: 5 live nodes, one frontier node with K = 2 children
    # would need 7 slots of the 6; CAPACITY, nothing appended
    t5 = t2.copy()
    t5.n_nodes[0] = 5
    t6, _, _, nn6, err = NG.expand_ngram(t5, np.array([[2]], np.int32), None, ctx, clen,
                                         tok, lp, fb, 2, 3, 3)
    assert err == T.DERR_CAPACITY and int(nn6[0]) == 0 and int(t6.n_nodes[0]) == 5
    assert np.array_equal(t6.token, t5.token) and np.array_equal(t6.parent, t5.parent)
    # one child fewer fits exactly (K = 1: 5 + 1 = 6 slots)
    t7, _, _, nn7, err = NG.expand_ngram(t5, np.array([[2]], np.int32), None, ctx, clen,
                                         tok, lp, fb, 1, 3, 3)
    assert err == 0 and int(nn7[0]) == 1 and int(t7.n_nodes[0]) == 6
    # a frontier id equal to the node count is not a node
    t4 = T.Tree.empty(1, 16)
    t4.parent[0, :2], t4.token[0, :2], t4.depth[0, :2], t4.n_nodes[0] = [-1, 0], [3, 3], [1, 2], 2
    _, _, _, nn4, err = NG.expand_ngram(t4, np.array([[2]], np.int32), None, ctx, clen, tok, lp,
                                        fb, 2, 3, 3)
    assert err == T.DERR_BAD_NODE and int(nn4[0]) == 0


def test_fallback_positions_at_the_edges():
    """A node whose token the context never holds takes fallback_pos: 0 is a
    valid position; -1 and L are not (BAD_NODE, then position L - 1).  A
    context token equal to V is out of range for the fallback count."""
    ctx, clen, tok, lp = _hand_cache()
    t = T.Tree.empty(1, 16)
    t.parent[0, 0], t.token[0, 0], t.depth[0, 0], t.n_nodes[0] = -1, 9, 1, 1
    t.cum[0, 0] = t.logp[0, 0] = -1.0
    fr = np.array([[0]], np.int32)
    for f, want, want_err in [(0, 0, 0), (-1, 5, T.DERR_BAD_NODE), (6, 5, T.DERR_BAD_NODE)]:
        t2, pos, _, _, err = NG.expand_ngram(t, fr, None, ctx, clen, tok, lp,
                                             np.array([f], np.int32), 2, 2, 3)
        assert int(pos[0, 0]) == want and err == want_err
        assert list(t2.cum[0, 1:3]) == [-1.0 + lp[0, want, 0], -1.0 + lp[0, want, 1]]
    # token 5 = V (three times) is skipped: 1 and 2 tie, 1 wins, last at 0
    fbp, err = NG.fallback_position(np.array([[1, 5, 2, 5, 5]], np.int32), np.array([5]), 5)
    assert err == T.DERR_BAD_NODE and int(fbp[0]) == 0
