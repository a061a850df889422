"""Host-side checks of libtreegraft.so (CPU only, no kernel is launched).

The library loads, exports every function include/treegraft.h declares, and
rejects bad arguments on the host before anything reaches the GPU.
"""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "treegraft.h")


@pytest.fixture(scope="module")
def lib():
    import paper_2608_26112_amd as tg
    if not os.path.exists(tg.LIB_PATH):
        from paper_2608_26112_amd.build import build
        build()
    return tg.load()


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(tg_[a-z_0-9]+)\s*\(", src)))


def test_header_declares_the_four_calls():
    names = _declared()
    for n in ("tg_tree_verify_attention", "tg_tree_expand_topk",
              "tg_tree_rescore_graft", "tg_tree_accept"):
        assert n in names


def test_every_declared_symbol_is_exported(lib):
    import paper_2608_26112_amd as tg
    names = _declared()
    assert sorted(tg.EXPORTED) == names
    for n in names:
        assert hasattr(lib, n), n


def test_constants_match_header():
    import paper_2608_26112_amd as tg
    src = open(HEADER).read()
    defs = dict(re.findall(r"#define\s+(TG_[A-Z_]+)\s+\(?(-?\d+)u?\)?", src))
    assert int(defs["TG_DERR_BAD_PARENT"]) == tg.DERR_BAD_PARENT
    assert int(defs["TG_DERR_CAPACITY"]) == tg.DERR_CAPACITY
    assert int(defs["TG_DERR_NONFINITE"]) == tg.DERR_NONFINITE
    assert int(defs["TG_DERR_BAD_PREFIX"]) == tg.DERR_BAD_PREFIX
    assert int(defs["TG_DERR_BAD_NODE"]) == tg.DERR_BAD_NODE
    assert int(defs["TG_NO_NODE"]) == tg.NO_NODE
    assert int(defs["TG_MAX_TOPK"]) == tg.MAX_TOPK
    assert int(defs["TG_MAX_CAP"]) == tg.MAX_CAP
    assert int(defs["TG_MAX_EXPAND_CHILDREN"]) == tg.MAX_EXPAND_CHILDREN
    assert int(defs["TG_MAX_VERIFY_NODES"]) == tg.MAX_VERIFY_NODES


def test_status_strings(lib):
    import paper_2608_26112_amd as tg
    assert tg.status_str(0) == "ok"
    assert "workspace" in tg.status_str(3)
    assert tg.status_str(99) == "unknown status"


P = ctypes.c_void_p(256)      # never dereferenced: every call below fails on the host
NULL = ctypes.c_void_p(0)


def _verify(lib, **kw):
    a = dict(q=P, k=P, v=P, parent=P, plen=P, out=P, B=1, N=16, Hq=4, Hkv=4, D=64,
             S=144, scale=0.125, dt=0, ws=NULL, wsb=0)
    a.update(kw)
    return lib.tg_tree_verify_attention(a["q"], a["k"], a["v"], a["parent"], a["plen"],
                                        a["out"], a["B"], a["N"], a["Hq"], a["Hkv"], a["D"],
                                        a["S"], a["scale"], a["dt"], a["ws"], a["wsb"],
                                        NULL, NULL)


def test_verify_attention_host_checks(lib):
    import paper_2608_26112_amd as tg
    assert _verify(lib, q=NULL) == tg.ERR_INVALID_ARG
    assert _verify(lib, Hq=6, Hkv=4) == tg.ERR_INVALID_ARG
    assert _verify(lib, S=8) == tg.ERR_INVALID_ARG            # S_max < N
    assert _verify(lib, N=0) == tg.ERR_INVALID_ARG
    assert _verify(lib, D=96) == tg.ERR_UNSUPPORTED
    assert _verify(lib, N=2048, S=4096) == tg.ERR_UNSUPPORTED
    assert _verify(lib, dt=7) == tg.ERR_INVALID_ARG
    assert _verify(lib, scale=float("nan")) == tg.ERR_INVALID_ARG
    assert _verify(lib, scale=-0.125) == tg.ERR_INVALID_ARG
    assert _verify(lib, scale=float("inf")) == tg.ERR_INVALID_ARG
    # q, the caches and out are read / written in 16-byte vectors
    for arg in ("q", "k", "v", "out"):
        assert _verify(lib, **{arg: ctypes.c_void_p(256 + 8)}) == tg.ERR_INVALID_ARG
    # a shape that needs a split workspace, called without one
    need = lib.tg_verify_attention_workspace(1, 64, 32, 8, 128, 2112, tg.BF16)
    assert need > 0
    assert _verify(lib, N=64, Hq=32, Hkv=8, D=128, S=2112, dt=tg.BF16) == tg.ERR_WORKSPACE
    assert lib.tg_verify_attention_workspace(8, 256, 64, 8, 128, 33024, tg.BF16) == 0
    assert lib.tg_verify_attention_workspace(1, 16, 4, 4, 64, 144, tg.F32) == 0


def _tree(cap=64, **null):
    import paper_2608_26112_amd as tg
    t = tg.TgTree(*(256 for _ in range(8)), cap)
    for k in null:
        setattr(t, k, 0)
    return t


def _expand(lib, tree=None, **kw):
    a = dict(logits=P, fr=P, nf=NULL, B=1, F=8, V=1000, K=4, N=8, lse=P, nxt=P, nn=P,
             ws=P, wsb=1 << 30)
    a.update(kw)
    t = _tree() if tree is None else tree
    return lib.tg_tree_expand_topk(ctypes.byref(t), a["logits"], a["fr"], a["nf"], a["B"],
                                   a["F"], a["V"], a["K"], a["N"], a["lse"], a["nxt"],
                                   a["nn"], a["ws"], a["wsb"], NULL, NULL)


def test_expand_host_checks(lib):
    import paper_2608_26112_amd as tg
    assert _expand(lib, logits=NULL) == tg.ERR_INVALID_ARG
    assert _expand(lib, tree=_tree(parent=1)) == tg.ERR_INVALID_ARG
    assert _expand(lib, K=2000) == tg.ERR_INVALID_ARG           # K > V
    assert _expand(lib, K=65, V=5000) == tg.ERR_UNSUPPORTED
    assert _expand(lib, F=200, K=64, V=5000) == tg.ERR_UNSUPPORTED
    assert _expand(lib, tree=_tree(cap=5000)) == tg.ERR_UNSUPPORTED
    assert _expand(lib, ws=NULL) == tg.ERR_WORKSPACE
    need = lib.tg_expand_topk_workspace(1, 8, 1000, 4, 8)
    assert need > 0
    assert _expand(lib, wsb=need - 1) == tg.ERR_WORKSPACE


def _rescore(lib, tree=None, **kw):
    a = dict(strong=P, B=1, R=17, V=1000, W=8, M=4, flags=0, lse=P, gf=P, ng=P, ws=P,
             wsb=1 << 30)
    a.update(kw)
    t = _tree() if tree is None else tree
    return lib.tg_tree_rescore_graft(ctypes.byref(t), a["strong"], a["B"], a["R"], a["V"],
                                     a["W"], a["M"], a["flags"], a.get("nf", NULL), a["lse"],
                                     a["gf"], a["ng"],
                                     a.get("nx", NULL), a.get("nn", NULL), a.get("N", 0),
                                     a["ws"], a["wsb"], NULL, NULL)


def test_rescore_host_checks(lib):
    import paper_2608_26112_amd as tg
    assert _rescore(lib, strong=NULL) == tg.ERR_INVALID_ARG
    assert _rescore(lib, W=0) == tg.ERR_INVALID_ARG
    assert _rescore(lib, M=2000) == tg.ERR_INVALID_ARG
    assert _rescore(lib, flags=8) == tg.ERR_UNSUPPORTED             # unknown variant bit
    assert _rescore(lib, flags=tg.POOL_NEWONLY) == tg.ERR_INVALID_ARG  # new_from missing
    big = _tree()
    big.cap = 4096                                                  # variant LDS > 160 KiB
    assert _rescore(lib, tree=big, flags=tg.GRAFT_OVERWRITE) == tg.ERR_UNSUPPORTED
    assert _rescore(lib, nx=P) == tg.ERR_INVALID_ARG              # n_next missing
    assert _rescore(lib, nx=P, nn=P, N=0) == tg.ERR_INVALID_ARG   # N must be >= 1
    assert _rescore(lib, M=100, V=5000) == tg.ERR_UNSUPPORTED
    assert _rescore(lib, ws=NULL) == tg.ERR_WORKSPACE
    need = lib.tg_rescore_graft_workspace(1, 17, 1000, 8, 4, 64)
    assert _rescore(lib, wsb=need - 1) == tg.ERR_WORKSPACE


def test_ngram_host_checks(lib):
    import paper_2608_26112_amd as tg

    def cache(**kw):
        a = dict(logits=P, ctx=P, clen=P, B=1, L=32, V=100, m=4, tok=P, lp=P, fb=P, ws=P,
                 wsb=1 << 30)
        a.update(kw)
        return lib.tg_ngram_cache(a["logits"], a["ctx"], a["clen"], a["B"], a["L"], a["V"],
                                  a["m"], a["tok"], a["lp"], a["fb"], a["ws"], a["wsb"], NULL,
                                  NULL)
    assert cache(logits=NULL) == tg.ERR_INVALID_ARG
    assert cache(m=101) == tg.ERR_INVALID_ARG
    assert cache(m=65, V=1000) == tg.ERR_UNSUPPORTED
    assert cache(ws=NULL) == tg.ERR_WORKSPACE
    assert cache(wsb=lib.tg_ngram_cache_workspace(1, 32, 100, 4) - 1) == tg.ERR_WORKSPACE

    def expand(**kw):
        a = dict(fr=P, nf=NULL, ctx=P, clen=P, tok=P, lp=P, fb=P, B=1, F=4, L=32, m=4, K=2,
                 N=4, n=3, mp=NULL, nx=P, nn=P)
        a.update(kw)
        t = _tree()
        return lib.tg_tree_expand_ngram(ctypes.byref(t), a["fr"], a["nf"], a["ctx"], a["clen"],
                                        a["tok"], a["lp"], a["fb"], a["B"], a["F"], a["L"],
                                        a["m"], a["K"], a["N"], a["n"], a["mp"], a["nx"],
                                        a["nn"], NULL, NULL)
    assert expand(ctx=NULL) == tg.ERR_INVALID_ARG
    assert expand(K=5) == tg.ERR_INVALID_ARG                      # K > m
    assert expand(n=0) == tg.ERR_INVALID_ARG
    assert expand(n=17) == tg.ERR_UNSUPPORTED
    assert expand(F=2000) == tg.ERR_UNSUPPORTED


def test_accept_logits_host_checks(lib):
    import paper_2608_26112_amd as tg

    def acc(**kw):
        a = dict(parent=P, token=P, n=P, logits=P, B=1, cap=16, R=17, V=100, md=16, g=P, A=P,
                 path=P, bonus=P)
        a.update(kw)
        return lib.tg_tree_accept_logits(a["parent"], a["token"], a["n"], a["logits"], a["B"],
                                         a["cap"], a["R"], a["V"], a["md"], a["g"], a["A"],
                                         a["path"], a["bonus"], NULL, NULL)
    assert acc(logits=NULL) == tg.ERR_INVALID_ARG
    assert acc(g=NULL) == tg.ERR_INVALID_ARG
    assert acc(V=0) == tg.ERR_INVALID_ARG
    assert acc(R=0) == tg.ERR_INVALID_ARG
    assert acc(cap=5000) == tg.ERR_UNSUPPORTED


def test_accept_host_checks(lib):
    import paper_2608_26112_amd as tg

    def acc(**kw):
        a = dict(parent=P, token=P, n=P, greedy=P, B=1, cap=16, md=16, A=P, path=P, bonus=P)
        a.update(kw)
        return lib.tg_tree_accept(a["parent"], a["token"], a["n"], a["greedy"], a["B"],
                                  a["cap"], a["md"], a["A"], a["path"], a["bonus"], NULL,
                                  NULL)
    assert acc(greedy=NULL) == tg.ERR_INVALID_ARG
    assert acc(md=-1) == tg.ERR_INVALID_ARG
    assert acc(path=NULL) == tg.ERR_INVALID_ARG
    assert acc(cap=5000) == tg.ERR_UNSUPPORTED


def test_reset_and_trace_host_checks(lib):
    import paper_2608_26112_amd as tg
    assert lib.tg_tree_reset(ctypes.byref(_tree(n_nodes=1)), 1, NULL) == tg.ERR_INVALID_ARG
    assert lib.tg_tree_reset(ctypes.byref(_tree()), 0, NULL) == tg.ERR_INVALID_ARG
    assert lib.tg_trace_begin(0) == tg.ERR_INVALID_ARG
    n = ctypes.c_int(7)
    assert lib.tg_trace_end(None, 0, ctypes.byref(n)) == tg.ERR_INVALID_ARG  # not tracing
    assert lib.tg_trace_read(None, 0, ctypes.byref(n)) == tg.ERR_INVALID_ARG


def test_python_binding_rejects_cpu_tensors():
    import torch

    import paper_2608_26112_amd as tg
    q = torch.zeros(1, 4, 2, 64)
    with pytest.raises(ValueError):
        tg.verify_attention(q, torch.zeros(1, 2, 8, 64), torch.zeros(1, 2, 8, 64),
                            torch.zeros(1, 4, dtype=torch.int32),
                            torch.zeros(1, dtype=torch.int32), 0.125)


def test_prune_and_kv_compact_host_checks(lib):
    import paper_2608_26112_amd as tg

    def prune(tree=None, **kw):
        a = dict(B=1, B_ver=8, maxp=9, out=P)
        a.update(kw)
        t = _tree() if tree is None else tree
        return lib.tg_tree_global_prune(ctypes.byref(t), a["B"], a["B_ver"], a["maxp"],
                                        *([a["out"]] * 8), NULL, NULL)
    assert prune(out=NULL) == tg.ERR_INVALID_ARG
    assert prune(B_ver=0) == tg.ERR_INVALID_ARG
    assert prune(maxp=0) == tg.ERR_INVALID_ARG
    assert prune(B_ver=5000) == tg.ERR_UNSUPPORTED
    assert prune(tree=_tree(cap=5000)) == tg.ERR_UNSUPPORTED
    assert prune(tree=_tree(cum=1)) == tg.ERR_INVALID_ARG

    def compact(**kw):
        a = dict(k=P, v=P, pl=P, path=P, n=P, B=1, H=2, S=64, D=128, maxp=4, dt=tg.BF16,
                 nl=ctypes.c_void_p(512))
        a.update(kw)
        return lib.tg_kv_compact(a["k"], a["v"], a["pl"], a["path"], a["n"], a["B"], a["H"],
                                 a["S"], a["D"], a["maxp"], a["dt"], a["nl"], NULL, NULL)
    assert compact(k=NULL) == tg.ERR_INVALID_ARG
    assert compact(nl=P) == tg.ERR_INVALID_ARG            # aliases prefix_len
    assert compact(path=NULL) == tg.ERR_INVALID_ARG
    assert compact(D=96) == tg.ERR_UNSUPPORTED
    assert compact(dt=5) == tg.ERR_INVALID_ARG
    assert compact(maxp=-1) == tg.ERR_INVALID_ARG


def test_signals_host_checks(lib):
    import paper_2608_26112_amd as tg

    def sig(tree=None, **kw):
        a = dict(fr=P, nf=NULL, B=1, F=4, W=4, L=5, ctx=NULL, prm=NULL, out=P, mg=NULL, act=NULL)
        a.update(kw)
        t = _tree() if tree is None else tree
        return lib.tg_tree_signals(ctypes.byref(t), a["fr"], a["nf"], a["B"], a["F"], a["W"],
                                   a["L"], a["ctx"], a["prm"], a["out"], a["mg"], a["act"],
                                   NULL, NULL)
    assert sig(fr=NULL) == tg.ERR_INVALID_ARG
    assert sig(out=NULL) == tg.ERR_INVALID_ARG
    assert sig(W=0) == tg.ERR_INVALID_ARG
    assert sig(L=-1) == tg.ERR_INVALID_ARG
    assert sig(prm=P) == tg.ERR_INVALID_ARG          # context / margin / action missing
    assert sig(tree=_tree(cap=5000)) == tg.ERR_UNSUPPORTED
