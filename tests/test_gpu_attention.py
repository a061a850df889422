"""GPU parity of tg_tree_verify_attention against the fp64 oracle.

Bars: fp32 per-row max error <= 1e-5 x the row's max magnitude; bf16 max abs
error <= 2e-2 and tensor-relative Frobenius error <= 1e-2.  The mask is also
checked without tolerance: poisoned non-ancestor slots must leave a node's
output bit-identical, and a root-level node over an empty prefix must return
its own value row exactly.
"""
import numpy as np
import pytest
import torch

import workloads as W
from oracle.attention import path_of, tree_verify_attention, tree_verify_attention_fast
from tests import _cases as C

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _gen(seed, B, N, Hq, Hkv, D, L, scale=1.0, extra=0):
    g = W.rng(seed)
    S = L + N + extra
    q = W.normal(g, (B, N, Hq, D)) * np.float32(scale)
    k = W.normal(g, (B, Hkv, S, D)) * np.float32(scale)
    v = W.normal(g, (B, Hkv, S, D)) * np.float32(scale)
    return q, k, v


def _run(tg, q, k, v, parent, plen, sm_scale, dtype, d_err=None):
    tq = torch.from_numpy(q).to(DEV).to(dtype)
    tk = torch.from_numpy(k).to(DEV).to(dtype)
    tv = torch.from_numpy(v).to(DEV).to(dtype)
    out = tg.verify_attention(tq, tk, tv, torch.from_numpy(np.ascontiguousarray(parent, np.int32)).to(DEV),
                              torch.from_numpy(np.asarray(plen, np.int32)).to(DEV), sm_scale,
                              d_err=d_err)
    torch.cuda.synchronize()
    # the oracle sees exactly the values the GPU saw (bf16-rounded inputs)
    return (out.float().cpu().numpy(), tq.float().cpu().numpy(), tk.float().cpu().numpy(),
            tv.float().cpu().numpy())


def test_tiny_config_fp32(tg):
    """Tiny workload: B1, 4/4 heads, D64, prefix 128, 16 nodes with
    parent[i] uniform in [-1, i-1], fp32 N(0,1)."""
    cfg = W.CONFIGS["tiny"]
    g = W.rng(cfg["seed"])
    N, L, D = cfg["N"], cfg["L"], cfg["D"]
    parent = W.uniform_parents(g, N)[None]
    q = W.normal(g, (1, N, 4, D))
    k = W.normal(g, (1, 4, L + N, D))
    v = W.normal(g, (1, 4, L + N, D))
    got, q, k, v = _run(tg, q, k, v, parent, [L], D ** -0.5, torch.float32)
    want = tree_verify_attention(q, k, v, parent, [L], D ** -0.5)
    C.attn_close_f32(got, want)


def _parents(kind, g, N):
    if kind == "chain":
        return np.arange(-1, N - 1, dtype=np.int32)
    if kind == "star":
        return np.full(N, -1, np.int32)
    return W.uniform_parents(g, N)


@pytest.mark.parametrize("N", [1, 2, 17, 64, 255, 256])
@pytest.mark.parametrize("kind", ["random", "chain", "star"])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_random_small(tg, N, kind, dtype):
    seed = 1000 * N + {"random": 1, "chain": 2, "star": 3}[kind] + (7 if dtype == "bf16" else 0)
    g = W.rng(seed)
    B, Hq, Hkv = 2, 8, 2
    D = 128 if N % 2 else 64
    plen = np.array([int(g.integers(0, 300)), 0 if N < 64 else int(g.integers(1, 100))])
    L = int(plen.max())
    parent = np.stack([_parents(kind, g, N) for _ in range(B)])
    q, k, v = _gen(seed + 1, B, N, Hq, Hkv, D, L, extra=5)
    dt = torch.bfloat16 if dtype == "bf16" else torch.float32
    got, q, k, v = _run(tg, q, k, v, parent, plen, D ** -0.5, dt)
    want = tree_verify_attention_fast(q, k, v, parent, plen, D ** -0.5)
    if dtype == "bf16":
        C.attn_close_bf16(got, want)
    else:
        C.attn_close_f32(got, want)


@pytest.mark.parametrize("Hq,Hkv,N,L,D,kernel", [
    (6, 2, 77, 300, 128, "attn_mfma"),      # 3 query heads per KV head
    (10, 2, 41, 130, 64, "attn_mfma"),      # 5
    (6, 2, 90, 4200, 128, "attn_pingpong"),  # 270 rows, prefix >= 4096
    (15, 3, 60, 4100, 64, "attn_pingpong"),  # 5 per KV head, 300 rows
])
def test_group_sizes_not_powers_of_two(tg, Hq, Hkv, N, L, D, kernel):
    """Query heads per KV head that are not powers of two: a wave's 32 output
    rows then straddle nodes at any row, and each row leaves to its own
    (node, head).  Ragged per-sequence prefixes; the route is asserted."""
    g = W.rng(7000 + Hq * 100 + N)
    B = 2
    plen = np.array([L, L - 37], np.int32)
    parent = np.stack([W.uniform_parents(g, N) for _ in range(B)])
    q, k, v = _gen(7001 + N, B, N, Hq, Hkv, D, L)
    torch.cuda.synchronize()
    tg.trace_begin(16)
    try:
        got, q, k, v = _run(tg, q, k, v, parent, plen, D ** -0.5, torch.bfloat16)
    finally:
        names = [n for n, _ in tg.trace_end()]
    assert kernel in names, names
    want = tree_verify_attention_fast(q, k, v, parent, plen, D ** -0.5)
    C.attn_close_bf16(got, want)


@pytest.mark.parametrize("kind", ["random", "chain"])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_largest_tree_1024_nodes(tg, kind, dtype):
    """N = 1024, the largest verify tree: the fp32 kernel's per-wave root
    path (a 1024-deep chain) and the bf16 kernel's 32-word bitsets."""
    g = W.rng(1024 + (kind == "chain"))
    B, N, Hq, Hkv, D = 1, 1024, 2, 1, 64
    plen = np.array([50])
    parent = _parents(kind, g, N)[None]
    q, k, v = _gen(1025, B, N, Hq, Hkv, D, 50, extra=3)
    dt = torch.bfloat16 if dtype == "bf16" else torch.float32
    got, q, k, v = _run(tg, q, k, v, parent, plen, D ** -0.5, dt)
    want = tree_verify_attention_fast(q, k, v, parent, plen, D ** -0.5)
    if dtype == "bf16":
        C.attn_close_bf16(got, want)
    else:
        C.attn_close_f32(got, want)


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_empty_prefix_root_level_node_is_exactly_v_self(tg, dtype):
    g = W.rng(5)
    N, D = 40, 128
    parent = W.uniform_parents(g, N)[None]
    q, k, v = _gen(6, 1, N, 4, 2, D, 0)
    got, _, _, vv = _run(tg, q, k, v, parent, [0], D ** -0.5, dtype)
    for i in np.nonzero(parent[0] == -1)[0]:
        for h in range(4):
            assert np.array_equal(got[0, i, h], vv[0, h // 2, i]), (i, h)


def test_poisoned_non_ancestors_are_bitwise_invisible(tg):
    """Masked keys must contribute exactly nothing: huge aligned K and V=+-1e3
    on every non-ancestor tree slot of node i leave node i's output
    bit-identical (bf16 MFMA path and the fp32 path)."""
    g = W.rng(11)
    N, D, L = 70, 128, 200
    parent = W.uniform_parents(g, N)[None]
    q, k, v = _gen(12, 1, N, 4, 4, D, L)
    for dt in (torch.bfloat16, torch.float32):
        base, *_ = _run(tg, q, k, v, parent, [L], D ** -0.5, dt)
        for i in (0, 13, 37, 69):
            keep = set(path_of(parent[0], i))
            kp, vp = k.copy(), v.copy()
            for j in range(N):
                if j not in keep:
                    kp[0, :, L + j] = q[0, i, 0] * 50.0
                    vp[0, :, L + j] = 1e3 if j % 2 else -1e3
            pois, *_ = _run(tg, q, kp, vp, parent, [L], D ** -0.5, dt)
            assert np.array_equal(pois[0, i], base[0, i]), (dt, i)


def test_constant_keys_give_mean_of_visible_values(tg):
    g = W.rng(13)
    N, D, L = 30, 64, 77
    parent = W.uniform_parents(g, N)[None]
    q, _, v = _gen(14, 1, N, 2, 1, D, L)
    k = np.full((1, 1, L + N, D), 0.25, np.float32)
    got, _, _, vv = _run(tg, q, k, v, parent, [L], 0.3, torch.bfloat16)
    for i in range(N):
        vis = list(range(L)) + [L + a for a in path_of(parent[0], i)]
        want = vv[0, 0, vis].astype(np.float64).mean(axis=0)
        for h in range(2):
            np.testing.assert_allclose(got[0, i, h], want, rtol=0, atol=8e-3)


def test_llama8b_config(tg):
    """Llama-3-8B-shaped verify layer: B1, 32/8 heads, D128, prefix 2048,
    64-node verify tree (root + 63 draft nodes shaped like a pruned top-8 /
    frontier-10 expansion of depth 6), Q/K/V N(0,1)/sqrt(128) bf16.  This
    shape runs the split-prefix path."""
    cfg = W.CONFIGS["llama8b"]
    g = W.rng(cfg["seed"])
    draft = W.expansion_shaped_tree(g, 63, 6, 8, 10)
    parent = W.verify_layout_with_root(draft)[None]
    N, L, D = 64, cfg["L"], 128
    q, k, v = _gen(cfg["seed"] + 1, 1, N, 32, 8, D, L, scale=cfg["qkv_scale"])
    got, q, k, v = _run(tg, q, k, v, parent, [L], D ** -0.5, torch.bfloat16)
    want = tree_verify_attention_fast(q, k, v, parent, [L], D ** -0.5)
    C.attn_close_bf16(got, want)


def test_longctx_config(tg):
    """Long-context verify: B4, 32/8 heads, D128, prefix 8192, 128-node trees
    of exactly 10 levels with branching <= 8, N(0,1) bf16."""
    cfg = W.CONFIGS["longctx"]
    g = W.rng(cfg["seed"])
    B, N, L, D = 4, 128, cfg["L"], 128
    parent = np.stack([W.level_tree(g, N, 10, 8) for _ in range(B)])
    q, k, v = _gen(cfg["seed"] + 1, B, N, 32, 8, D, L)
    got, q, k, v = _run(tg, q, k, v, parent, [L] * B, D ** -0.5, torch.bfloat16)
    want = tree_verify_attention_fast(q, k, v, parent, [L] * B, D ** -0.5)
    C.attn_close_bf16(got, want)


def test_llama70b_config_sampled_rows(tg):
    """Llama-3-70B-shaped verify layer on one GPU: B8, 64/8 heads, D128,
    prefix 32768, 256-node trees of 12 levels, branching <= 8, N(0,1) bf16.
    The oracle recomputes 96 sampled (batch, node, head) rows."""
    cfg = W.CONFIGS["llama70b"]
    g = W.rng(cfg["seed"])
    B, N, L, D, Hq, Hkv = 8, 256, cfg["L"], 128, 64, 8
    parent = np.stack([W.level_tree(g, N, 12, 8) for _ in range(B)])
    S = L + N
    dev_q = torch.empty((B, N, Hq, D), dtype=torch.bfloat16, device=DEV)
    dev_k = torch.empty((B, Hkv, S, D), dtype=torch.bfloat16, device=DEV)
    dev_v = torch.empty((B, Hkv, S, D), dtype=torch.bfloat16, device=DEV)
    for b in range(B):   # per-sequence streams keep host memory small
        gb = W.rng([cfg["seed"], b])
        dev_q[b] = torch.from_numpy(W.normal(gb, (N, Hq, D))).to(DEV)
        dev_k[b] = torch.from_numpy(W.normal(gb, (Hkv, S, D))).to(DEV)
        dev_v[b] = torch.from_numpy(W.normal(gb, (Hkv, S, D))).to(DEV)
    out = tg.verify_attention(dev_q, dev_k, dev_v, torch.from_numpy(parent).to(DEV),
                              torch.full((B,), L, dtype=torch.int32, device=DEV), D ** -0.5)
    torch.cuda.synchronize()
    rows = [(int(g.integers(0, B)), int(g.integers(0, N)), int(g.integers(0, Hq)))
            for _ in range(96)]
    rows += [(0, 0, 0), (B - 1, N - 1, Hq - 1)]
    got = np.stack([out[b, i, h].float().cpu().numpy() for b, i, h in rows])
    want = np.empty_like(got, dtype=np.float64)
    for r, (b, i, h) in enumerate(rows):
        g0 = h // (Hq // Hkv)
        kb = dev_k[b:b + 1, g0:g0 + 1].float().cpu().numpy()
        vb = dev_v[b:b + 1, g0:g0 + 1].float().cpu().numpy()
        qb = dev_q[b:b + 1, :, h:h + 1].float().cpu().numpy()
        want[r] = tree_verify_attention(qb, kb, vb, parent[b:b + 1], [L], D ** -0.5,
                                        rows=[(0, i, 0)])[0]
    C.attn_close_bf16(got, want)


def test_device_error_bits(tg):
    g = W.rng(21)
    N, D, L = 10, 64, 20
    q, k, v = _gen(22, 2, N, 2, 2, D, L)
    parent = np.stack([W.uniform_parents(g, N) for _ in range(2)])
    bad = parent.copy()
    bad[0, 4] = 7          # parent >= own id: read as -1
    bad[1, 2] = -9         # < -1: read as -1
    fixed = bad.copy()
    fixed[0, 4] = -1
    fixed[1, 2] = -1
    for dt in (torch.bfloat16, torch.float32):
        err = torch.zeros(1, dtype=torch.int32, device=DEV)
        got, qq, kk, vv = _run(tg, q, k, v, bad, [L, L], D ** -0.5, dt, d_err=err)
        assert int(err.item()) & tg.DERR_BAD_PARENT
        ref, *_ = _run(tg, q, k, v, fixed, [L, L], D ** -0.5, dt)
        assert np.array_equal(got, ref)
        err.zero_()
        got, *_ = _run(tg, q, k, v, parent, [L, L + 1], D ** -0.5, dt, d_err=err)  # L+N > S_max
        assert int(err.item()) & tg.DERR_BAD_PREFIX
        assert np.all(got[1] == 0.0)
        ref, *_ = _run(tg, q, k, v, parent, [L, L], D ** -0.5, dt)
        assert np.array_equal(got[0], ref[0])


def test_repeatable_bitwise(tg):
    g = W.rng(31)
    N, D, L = 100, 128, 1500
    parent = W.uniform_parents(g, N)[None]
    q, k, v = _gen(32, 1, N, 16, 4, D, L)
    a, *_ = _run(tg, q, k, v, parent, [L], D ** -0.5, torch.bfloat16)
    b, *_ = _run(tg, q, k, v, parent, [L], D ** -0.5, torch.bfloat16)
    assert np.array_equal(a, b)


@pytest.mark.parametrize("D", [64, 128])
def test_many_splits_and_bad_prefix_in_split_mode(tg, D):
    """One KV head and a 4000-key prefix: the key tiles are dealt to more
    splits than one combine lane holds (more than D / 8), and with the
    second sequence's prefix length invalid (L + N > S_max) its rows are 0
    while the first sequence's are unchanged."""
    g = W.rng(40 + D)
    B, N, Hq, Hkv, L = 2, 16, 4, 1, 4000
    rows = B * N * Hq
    ws = tg.verify_attention_workspace(B, N, Hq, Hkv, D, L + N, tg.BF16)
    splits = (ws - 256) // (rows * (2 * D + 4))
    assert splits > D // 8
    parent = np.stack([W.uniform_parents(g, N) for _ in range(B)])
    q, k, v = _gen(41 + D, B, N, Hq, Hkv, D, L)
    got, qq, kk, vv = _run(tg, q, k, v, parent, [L, L], D ** -0.5, torch.bfloat16)
    want = tree_verify_attention_fast(qq, kk, vv, parent, np.array([L, L]), D ** -0.5)
    C.attn_close_bf16(got, want)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    got2, *_ = _run(tg, q, k, v, parent, [L, L + 1], D ** -0.5, torch.bfloat16, d_err=err)
    assert int(err.item()) & tg.DERR_BAD_PREFIX
    assert np.all(got2[1] == 0.0) and np.array_equal(got2[0], got[0])


def test_wide_combine_d64_sampled_rows(tg):
    """D = 64 with 32768 (node, head) rows in split mode, so the combine runs
    four-wave workgroups (eight rows per wave); 64 sampled rows plus the first
    and last against the oracle."""
    g = W.rng(47)
    B, N, L, D, Hq, Hkv = 2, 256, 2048, 64, 64, 1
    rows_total = B * N * Hq
    ws = tg.verify_attention_workspace(B, N, Hq, Hkv, D, L + N, tg.BF16)
    assert ws > 0 and rows_total // (64 // (D // 8)) >= 4 * 1024   # split mode, wide grid
    parent = np.stack([W.uniform_parents(g, N) for _ in range(B)])
    q, k, v = _gen(48, B, N, Hq, Hkv, D, L)
    dq = torch.from_numpy(q).to(DEV).to(torch.bfloat16)
    dk = torch.from_numpy(k).to(DEV).to(torch.bfloat16)
    dv = torch.from_numpy(v).to(DEV).to(torch.bfloat16)
    out = tg.verify_attention(dq, dk, dv, torch.from_numpy(parent).to(DEV),
                              torch.full((B,), L, dtype=torch.int32, device=DEV), D ** -0.5)
    torch.cuda.synchronize()
    rows = [(int(g.integers(0, B)), int(g.integers(0, N)), int(g.integers(0, Hq)))
            for _ in range(64)]
    rows += [(0, 0, 0), (B - 1, N - 1, Hq - 1)]
    got = np.stack([out[b, i, h].float().cpu().numpy() for b, i, h in rows])
    qh, kh, vh = dq.float().cpu().numpy(), dk.float().cpu().numpy(), dv.float().cpu().numpy()
    want = tree_verify_attention(qh, kh, vh, parent, np.array([L, L]), D ** -0.5, rows=rows)
    C.attn_close_bf16(got, want)
