"""The entry point that allocates nothing (tg_tree_verify_attention_noalloc)
against tg_tree_verify_attention with a workspace: same kernels, so the
outputs must be bit-identical, on consecutive calls of decreasing size that
run the split-prefix mode (the only one that uses the scratch), and on an
fp32 call (no scratch).  A shape whose workspace exceeds the scratch is
rejected on the host before anything is launched."""
import numpy as np
import pytest
import torch

import workloads as W

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _inputs(seed, B, N, Hq, Hkv, D, L, dtype):
    g = W.rng(seed)
    S = L + N + 3
    q = torch.from_numpy(W.normal(g, (B, N, Hq, D))).to(DEV).to(dtype)
    k = torch.from_numpy(W.normal(g, (B, Hkv, S, D))).to(DEV).to(dtype)
    v = torch.from_numpy(W.normal(g, (B, Hkv, S, D))).to(DEV).to(dtype)
    parent = torch.from_numpy(np.stack([W.uniform_parents(g, N) for _ in range(B)])).to(DEV)
    plen = torch.from_numpy(np.array([L - 7 * b for b in range(B)], np.int32)).to(DEV)
    return q, k, v, parent, plen


@pytest.mark.parametrize("shapes", [
    # Llama-3-8B-shaped layer (11 splits), then a smaller split-mode call
    [(1, 64, 32, 8, 128, 2048), (2, 17, 8, 2, 64, 1000)],
    # long-context-shaped (ping-pong kernel, 4 splits), then the 8B shape
    [(4, 128, 32, 8, 128, 8192), (1, 64, 32, 8, 128, 2048)],
])
def test_noalloc_matches_workspace_call_on_consecutive_calls(tg, shapes):
    outs = []
    for i, (B, N, Hq, Hkv, D, L) in enumerate(shapes):
        q, k, v, parent, plen = _inputs(900 + i, B, N, Hq, Hkv, D, L, torch.bfloat16)
        S = k.shape[2]
        need = tg.verify_attention_workspace(B, N, Hq, Hkv, D, S, tg.BF16)
        assert 0 < need <= tg.NOALLOC_SCRATCH_BYTES   # split mode, inside the scratch
        err_a = torch.zeros(1, dtype=torch.int32, device=DEV)
        err_b = torch.zeros(1, dtype=torch.int32, device=DEV)
        a = tg.verify_attention(q, k, v, parent, plen, D ** -0.5, d_err=err_a)
        b = tg.verify_attention_noalloc(q, k, v, parent, plen, D ** -0.5, d_err=err_b)
        torch.cuda.synchronize()
        assert torch.equal(a, b), (i, float((a.float() - b.float()).abs().max()))
        assert int(err_a.item()) == int(err_b.item()) == 0
        outs.append(b)
    assert outs[0].shape != outs[1].shape


def test_noalloc_fp32_and_whole_mode(tg):
    for dtype, shape in ((torch.float32, (1, 16, 4, 4, 64, 128)),
                         (torch.bfloat16, (8, 256, 64, 8, 128, 4096))):
        B, N, Hq, Hkv, D, L = shape
        q, k, v, parent, plen = _inputs(950, B, N, Hq, Hkv, D, L, dtype)
        a = tg.verify_attention(q, k, v, parent, plen, D ** -0.5)
        b = tg.verify_attention_noalloc(q, k, v, parent, plen, D ** -0.5)
        torch.cuda.synchronize()
        assert torch.equal(a, b), dtype


def test_noalloc_rejects_shapes_beyond_the_scratch(tg):
    B, N, Hq, Hkv, D, L = 1, 1020, 64, 1, 128, 60000   # 2 splits of 65280 rows: 33.9 MB
    S = L + N
    need = tg.verify_attention_workspace(B, N, Hq, Hkv, D, S, tg.BF16)
    assert need > tg.NOALLOC_SCRATCH_BYTES
    q = torch.zeros((B, N, Hq, D), dtype=torch.bfloat16, device=DEV)
    k = torch.zeros((B, Hkv, S, D), dtype=torch.bfloat16, device=DEV)
    parent = torch.full((B, N), -1, dtype=torch.int32, device=DEV)
    plen = torch.full((B,), L, dtype=torch.int32, device=DEV)
    with pytest.raises(tg.TgError) as e:
        tg.verify_attention_noalloc(q, k, k, parent, plen, D ** -0.5)
    assert e.value.status == tg.ERR_WORKSPACE
