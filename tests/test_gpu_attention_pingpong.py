"""GPU parity of the long-prefix (eight-wave ping-pong) attention kernel.

The library sends a bf16 call to that kernel when a KV head has at least 256
query rows (N * Hq / Hkv) and the cache leaves at least 4096 prefix rows
(S_max - N); every test here asserts the route from the library's kernel
trace, in both of the kernel's modes:
  * split mode - a sequence's key tiles are dealt to several workgroups and
    merged by the combine kernel (few (batch, KV head, row tile) groups);
  * whole mode - one workgroup per (batch, KV head, row tile), no combine
    (at least 256 such groups).
Shapes are deliberately ragged: N not a multiple of 64, prefix lengths that
differ per sequence, are not multiples of 64, are below one tile (37) or
empty (0), plus one tile-aligned length; D = 64 and D = 128.

Mask checks are tolerance-free (Alg. 3 tree-attention mask):
  * support: with every key equal, each visible key has weight exactly 1
    before normalisation, so with one-hot values (tree slot j -> dimension j,
    every prefix row -> dimension D - 1) the set of non-zero outputs of a
    node is exactly its root path, plus D - 1 when the prefix is not empty;
    in whole mode the values are exactly bf16(1 / (L + t)) and
    bf16(L / (L + t)) (t = the path length), computed in fp32 as the kernel
    normalises;
  * poison: huge aligned keys and values of +-1000 on every non-ancestor tree
    slot of a node leave that node's output bit-identical;
  * V_self: a root-level node over an empty prefix returns its own value row
    exactly, even with the cache sized for a 4096-row prefix;
  * device error bits: a bad parent reads as -1 (output bit-identical to the
    corrected parent array) and a bad prefix length zeroes that sequence only.
Random inputs are compared with the fp64 oracle at the bf16 bars (max abs
error 2e-2, tensor-relative Frobenius error 1e-2).
"""
import numpy as np
import pytest
import torch

import workloads as W
from oracle.attention import path_of, tree_verify_attention, tree_verify_attention_fast
from tests import _cases as C

pytestmark = pytest.mark.gpu
DEV = "cuda"
G = 8                       # query heads per KV head
L_SPLIT = [4100, 37, 0, 4160]
L_WHOLE = [4100, 37]
MIN_PREFIX = 4096           # the cache must leave this many prefix rows


def _shape(mode, N):
    """(B, Hkv, prefix lengths) of one mode: split mode has one KV head, whole
    mode enough (batch, KV head, 256-row tile) groups to fill 256 CUs."""
    tiles = -(-N * G // 256)
    if mode == "split":
        return len(L_SPLIT), 1, list(L_SPLIT)
    B = len(L_WHOLE)
    return B, -(-256 // (B * tiles)), list(L_WHOLE)


def _s_max(N, plen):
    return max(max(plen), MIN_PREFIX) + N + 9


def _call(tg, q, k, v, parent, plen, scale, d_err=None):
    """One traced call; returns (out, names of the kernels it launched)."""
    torch.cuda.synchronize()
    tg.trace_begin(16)
    try:
        out = tg.verify_attention(q, k, v, parent, plen, scale, d_err=d_err)
        torch.cuda.synchronize()
    finally:
        recs = tg.trace_end()
    return out, [n for n, _ in recs]


def _assert_route(names, mode):
    assert "attn_pingpong" in names, names
    assert ("attn_combine" in names) == (mode == "split"), names


def _parents(g, B, N):
    """Random trees: a uniform-parent forest, a 12-level tree and a chain."""
    kinds = [W.uniform_parents(g, N), W.level_tree(g, N, 12, 8),
             np.arange(-1, N - 1, dtype=np.int32)]
    return np.stack([kinds[b % len(kinds)] for b in range(B)]).astype(np.int32)


def _dev(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a)).to(DEV)
    return t if dtype is None else t.to(dtype)


# --------------------------------------------------------------- support

@pytest.mark.parametrize("mode", ["split", "whole"])
@pytest.mark.parametrize("D", [64, 128])
def test_mask_support_exact(tg, D, mode):
    N = D - 1                                  # tree slots use dimensions 0..N-1
    B, Hkv, plen = _shape(mode, N)
    Hq = G * Hkv
    S = _s_max(N, plen)
    g = W.rng([500, D, len(plen)])
    parent = _parents(g, B, N)
    q = _dev(W.normal(g, (B, N, Hq, D)), torch.bfloat16)
    k = torch.full((B, Hkv, S, D), 0.25, dtype=torch.bfloat16, device=DEV)
    v = torch.full((B, Hkv, S, D), 1000.0, dtype=torch.bfloat16, device=DEV)  # unused rows
    for b, L in enumerate(plen):
        v[b, :, :L + N] = 0.0
        v[b, :, :L, D - 1] = 1.0
        for j in range(N):
            v[b, :, L + j, j] = 1.0
    out, names = _call(tg, q, k, v, _dev(parent), _dev(np.array(plen, np.int32)), D ** -0.5)
    _assert_route(names, mode)
    got = out.float().cpu().numpy()
    for b, L in enumerate(plen):
        for i in range(N):
            path = path_of(parent[b], i)
            t = len(path)
            support = np.zeros(D, bool)
            support[path] = True
            if L > 0:
                support[D - 1] = True
            rows = got[b, i]                                   # [Hq, D]
            assert np.array_equal(rows != 0.0, np.broadcast_to(support, rows.shape)), (b, i)
            want = np.zeros(D, np.float64)
            want[path] = 1.0 / (L + t)
            want[D - 1] = L / (L + t)
            if mode == "whole":
                inv = np.float32(1.0) / np.float32(L + t)
                exact = torch.zeros(D, dtype=torch.float32)
                exact[path] = float(inv)
                exact[D - 1] = float(np.float32(L) * inv)
                exact = exact.to(torch.bfloat16).float().numpy()
                assert np.array_equal(rows, np.broadcast_to(exact, rows.shape)), (b, i)
            else:
                np.testing.assert_allclose(rows, np.broadcast_to(want, rows.shape),
                                           rtol=1e-2, atol=0)


# ---------------------------------------------------------------- poison

@pytest.mark.parametrize("mode", ["split", "whole"])
@pytest.mark.parametrize("D", [64, 128])
def test_poisoned_non_ancestors_bitwise(tg, D, mode):
    N = 100
    B, Hkv, plen = _shape(mode, N)
    Hq = G * Hkv
    S = _s_max(N, plen)
    g = W.rng([510, D, len(plen)])
    parent = _parents(g, B, N)
    q = _dev(W.normal(g, (B, N, Hq, D)), torch.bfloat16)
    k = _dev(W.normal(g, (B, Hkv, S, D)), torch.bfloat16)
    v = _dev(W.normal(g, (B, Hkv, S, D)), torch.bfloat16)
    dpar, dlen = _dev(parent), _dev(np.array(plen, np.int32))
    base, names = _call(tg, q, k, v, dpar, dlen, D ** -0.5)
    _assert_route(names, mode)
    base = base.float().cpu().numpy()
    for b in range(B):
        L = plen[b]
        for i in (0, 41, N - 1):
            keep = set(path_of(parent[b], i))
            kp, vp = k.clone(), v.clone()
            for j in range(N):
                if j not in keep:
                    # every head of the group sees a key aligned with its query
                    kp[b, :, L + j] = q[b, i, ::G].float().mul(50.0).to(torch.bfloat16)
                    vp[b, :, L + j] = 1e3 if j % 2 else -1e3
            pois, _ = _call(tg, q, kp, vp, dpar, dlen, D ** -0.5)
            assert np.array_equal(pois[b, i].float().cpu().numpy(), base[b, i]), (b, i)


# ---------------------------------------------------------------- V_self

@pytest.mark.parametrize("mode", ["split", "whole"])
@pytest.mark.parametrize("D", [64, 128])
def test_empty_prefix_root_level_nodes_are_exactly_v_self(tg, D, mode):
    N = 64
    B, Hkv, _ = _shape(mode, N)
    Hq = G * Hkv
    plen = [0] * B
    S = N + MIN_PREFIX + 9
    g = W.rng([520, D])
    parent = np.stack([W.uniform_parents(g, N) for _ in range(B)])
    q = _dev(W.normal(g, (B, N, Hq, D)), torch.bfloat16)
    k = _dev(W.normal(g, (B, Hkv, S, D)), torch.bfloat16)
    v = _dev(W.normal(g, (B, Hkv, S, D)), torch.bfloat16)
    out, names = _call(tg, q, k, v, _dev(parent), _dev(np.array(plen, np.int32)), D ** -0.5)
    _assert_route(names, mode)
    got = out.float().cpu().numpy()
    vv = v.float().cpu().numpy()
    checked = 0
    for b in range(B):
        for i in np.nonzero(parent[b] == -1)[0]:
            for h in range(Hq):
                assert np.array_equal(got[b, i, h], vv[b, h // G, i]), (b, i, h)
            checked += 1
    assert checked >= B


# ------------------------------------------------------- random vs oracle

@pytest.mark.parametrize("mode", ["split", "whole"])
@pytest.mark.parametrize("D", [64, 128])
def test_ragged_random_vs_oracle(tg, D, mode):
    """N = 100 and per-sequence ragged prefixes; split mode is checked on
    every row, whole mode on 160 sampled rows plus the first and last."""
    N = 100
    B, Hkv, plen = _shape(mode, N)
    Hq = G * Hkv
    S = _s_max(N, plen)
    g = W.rng([530, D, len(plen)])
    parent = _parents(g, B, N)
    q = _dev(W.normal(g, (B, N, Hq, D)), torch.bfloat16)
    k = _dev(W.normal(g, (B, Hkv, S, D)), torch.bfloat16)
    v = _dev(W.normal(g, (B, Hkv, S, D)), torch.bfloat16)
    out, names = _call(tg, q, k, v, _dev(parent), _dev(np.array(plen, np.int32)), D ** -0.5)
    _assert_route(names, mode)
    got = out.float().cpu().numpy()
    qh, kh, vh = q.float().cpu().numpy(), k.float().cpu().numpy(), v.float().cpu().numpy()
    if mode == "split":
        want = tree_verify_attention_fast(qh, kh, vh, parent, np.array(plen), D ** -0.5)
        C.attn_close_bf16(got, want)
        return
    rows = [(int(g.integers(0, B)), int(g.integers(0, N)), int(g.integers(0, Hq)))
            for _ in range(160)] + [(0, 0, 0), (B - 1, N - 1, Hq - 1)]
    want = tree_verify_attention(qh, kh, vh, parent, np.array(plen), D ** -0.5, rows=rows)
    C.attn_close_bf16(np.stack([got[b, i, h] for b, i, h in rows]), want)


# --------------------------------------------------------- device errors

@pytest.mark.parametrize("mode", ["split", "whole"])
@pytest.mark.parametrize("D", [64, 128])
def test_bad_parent_and_bad_prefix(tg, D, mode):
    N = 100
    B, Hkv, plen = _shape(mode, N)
    Hq = G * Hkv
    S = _s_max(N, plen)
    g = W.rng([540, D, len(plen)])
    parent = _parents(g, B, N)
    q = _dev(W.normal(g, (B, N, Hq, D)), torch.bfloat16)
    k = _dev(W.normal(g, (B, Hkv, S, D)), torch.bfloat16)
    v = _dev(W.normal(g, (B, Hkv, S, D)), torch.bfloat16)
    dlen = _dev(np.array(plen, np.int32))
    bad = parent.copy()
    bad[0, 57] = 80          # parent >= own id: read as -1
    bad[B - 1, 3] = -7       # < -1: read as -1
    fixed = bad.copy()
    fixed[0, 57] = -1
    fixed[B - 1, 3] = -1
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    got, names = _call(tg, q, k, v, _dev(bad), dlen, D ** -0.5, d_err=err)
    _assert_route(names, mode)
    assert int(err.item()) == tg.DERR_BAD_PARENT
    ref, _ = _call(tg, q, k, v, _dev(fixed), dlen, D ** -0.5)
    assert torch.equal(got, ref)
    # sequence 1's prefix length runs past the cache: its rows are 0, the
    # other sequences' rows are unchanged
    bad_len = list(plen)
    bad_len[1] = S - N + 1
    err.zero_()
    got2, names = _call(tg, q, k, v, _dev(fixed), _dev(np.array(bad_len, np.int32)),
                        D ** -0.5, d_err=err)
    _assert_route(names, mode)
    assert int(err.item()) == tg.DERR_BAD_PREFIX
    assert bool((got2[1] == 0).all())
    keep = [b for b in range(B) if b != 1]
    assert torch.equal(got2[keep], ref[keep])
