"""Python binding of libtreegraft.so: the MI355X tree-verify / tree-expand path.

Argument marshalling only: every call forwards torch tensors' device pointers
and the current HIP stream to the C ABI declared in include/treegraft.h; all
computation runs in the library's HIP kernels.  There is no CPU fallback: a
missing library or a non-GPU tensor is an error.

Calls (same names as the C ABI without the ``tg_`` prefix):
  verify_attention  tree attention over a prefix KV cache (Alg. 3 mask)
  expand_topk       one expansion step (Sec. 3.1; Alg. 1)
  rescore_graft     one middle-drafter step (Sec. 3.2; Alg. 2)
  accept            greedy acceptance (temperature 0)
"""
from __future__ import annotations

import ctypes
import os

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libtreegraft.so")

# status codes, dtypes, device error bits and limits of include/treegraft.h
OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_WORKSPACE, ERR_HIP = range(5)
F32, BF16 = 0, 1
DERR_BAD_PARENT = 1
DERR_CAPACITY = 2
DERR_NONFINITE = 4
DERR_BAD_PREFIX = 8
DERR_BAD_NODE = 16
NO_NODE = -2
# variant flags of rescore_graft (see include/treegraft.h)
POOL_NEWONLY = 1
GRAFT_OVERWRITE = 2
GRAFT_DEDUP = 4
MAX_TOPK = 64
MAX_CAP = 4096
MAX_EXPAND_CHILDREN = 8192
MAX_VERIFY_NODES = 1024
NOALLOC_SCRATCH_BYTES = 32 << 20

EXPORTED = (
    "tg_status_str",
    "tg_tree_reset",
    "tg_trace_begin",
    "tg_trace_read",
    "tg_trace_end",
    "tg_verify_attention_workspace",
    "tg_tree_verify_attention",
    "tg_tree_verify_attention_noalloc",
    "tg_expand_topk_workspace",
    "tg_tree_expand_topk",
    "tg_rescore_graft_workspace",
    "tg_tree_rescore_graft",
    "tg_ngram_cache_workspace",
    "tg_ngram_cache",
    "tg_tree_expand_ngram",
    "tg_tree_accept_logits",
    "tg_tree_accept",
    "tg_tree_global_prune",
    "tg_kv_compact",
    "tg_tree_signals",
)


class TgError(RuntimeError):
    """A library call returned a status other than TG_OK."""

    def __init__(self, call, status, message):
        super().__init__(f"{call}: {message} (status {status})")
        self.status = status


class TgTraceRecord(ctypes.Structure):
    _fields_ = [("kernel", ctypes.c_char_p), ("ms", ctypes.c_float)]


class TgTree(ctypes.Structure):
    _fields_ = [
        ("parent", ctypes.c_void_p),
        ("token", ctypes.c_void_p),
        ("depth", ctypes.c_void_p),
        ("logp", ctypes.c_void_p),
        ("cum", ctypes.c_void_p),
        ("visited", ctypes.c_void_p),
        ("root_visited", ctypes.c_void_p),
        ("n_nodes", ctypes.c_void_p),
        ("cap", ctypes.c_int32),
    ]


_lib = None
_vp, _i32, _sz, _u32, _f32 = (ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t,
                              ctypes.c_uint32, ctypes.c_float)


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libtreegraft.so (built by ``__graft_entry__.build()``)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built; run __graft_entry__.build() first")
    lib = ctypes.CDLL(path)
    lib.tg_status_str.restype = ctypes.c_char_p
    lib.tg_status_str.argtypes = [_i32]
    lib.tg_verify_attention_workspace.restype = _sz
    lib.tg_verify_attention_workspace.argtypes = [_i32] * 6 + [_i32]
    lib.tg_tree_verify_attention.restype = _i32
    lib.tg_tree_verify_attention.argtypes = ([_vp] * 6 + [_i32] * 6 + [_f32, _i32, _vp, _sz,
                                             _vp, _vp])
    lib.tg_tree_verify_attention_noalloc.restype = _i32
    lib.tg_tree_verify_attention_noalloc.argtypes = ([_vp] * 6 + [_i32] * 6 + [_f32, _i32, _vp,
                                                     _vp])
    lib.tg_expand_topk_workspace.restype = _sz
    lib.tg_expand_topk_workspace.argtypes = [_i32] * 5
    lib.tg_tree_expand_topk.restype = _i32
    lib.tg_tree_expand_topk.argtypes = ([ctypes.POINTER(TgTree), _vp, _vp, _vp] + [_i32] * 5 +
                                        [_vp, _vp, _vp, _vp, _sz, _vp, _vp])
    lib.tg_rescore_graft_workspace.restype = _sz
    lib.tg_rescore_graft_workspace.argtypes = [_i32] * 6
    lib.tg_tree_rescore_graft.restype = _i32
    lib.tg_tree_rescore_graft.argtypes = ([ctypes.POINTER(TgTree), _vp] + [_i32] * 5 + [_u32] +
                                          [_vp, _vp, _vp, _vp, _vp, _vp, _i32, _vp, _sz, _vp,
                                           _vp])
    lib.tg_tree_accept.restype = _i32
    lib.tg_tree_accept.argtypes = [_vp] * 4 + [_i32] * 3 + [_vp] * 5
    lib.tg_ngram_cache_workspace.restype = _sz
    lib.tg_ngram_cache_workspace.argtypes = [_i32] * 4
    lib.tg_ngram_cache.restype = _i32
    lib.tg_ngram_cache.argtypes = [_vp] * 3 + [_i32] * 4 + [_vp] * 4 + [_sz, _vp, _vp]
    lib.tg_tree_expand_ngram.restype = _i32
    lib.tg_tree_expand_ngram.argtypes = ([ctypes.POINTER(TgTree)] + [_vp] * 7 + [_i32] * 7 +
                                         [_vp] * 5)
    lib.tg_tree_accept_logits.restype = _i32
    lib.tg_tree_accept_logits.argtypes = [_vp] * 4 + [_i32] * 5 + [_vp] * 6
    lib.tg_tree_reset.restype = _i32
    lib.tg_tree_reset.argtypes = [ctypes.POINTER(TgTree), _i32, _vp]
    lib.tg_tree_global_prune.restype = _i32
    lib.tg_tree_global_prune.argtypes = [ctypes.POINTER(TgTree)] + [_i32] * 3 + [_vp] * 10
    lib.tg_tree_signals.restype = _i32
    lib.tg_tree_signals.argtypes = ([ctypes.POINTER(TgTree), _vp, _vp] + [_i32] * 4 +
                                    [_vp] * 7)
    lib.tg_kv_compact.restype = _i32
    lib.tg_kv_compact.argtypes = [_vp] * 5 + [_i32] * 6 + [_vp] * 3
    lib.tg_trace_begin.restype = _i32
    lib.tg_trace_begin.argtypes = [_i32]
    lib.tg_trace_end.restype = _i32
    lib.tg_trace_end.argtypes = [ctypes.POINTER(TgTraceRecord), _i32, ctypes.POINTER(_i32)]
    lib.tg_trace_read.restype = _i32
    lib.tg_trace_read.argtypes = [ctypes.POINTER(TgTraceRecord), _i32, ctypes.POINTER(_i32)]
    _lib = lib
    return lib


def status_str(status: int) -> str:
    return load().tg_status_str(status).decode()


def _check(call, status):
    if status != OK:
        raise TgError(call, status, status_str(status))


def _ptr(t):
    return ctypes.c_void_p(0 if t is None else t.data_ptr())


def _dev(t, name, dtype=None):
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must have dtype {dtype}, got {t.dtype}")
    return t


def _stream_obj(stream, device):
    return torch.cuda.current_stream(device) if stream is None else stream


def _stream(stream, device=None):
    return ctypes.c_void_p(_stream_obj(stream, device).cuda_stream)


def _out(t, name, shape, dtype, device):
    """A caller-supplied output, checked (GPU, contiguous, dtype, shape, on
    `device`), or a new empty tensor when `t` is None."""
    shape = tuple(int(x) for x in shape)
    if t is None:
        return torch.empty(shape, dtype=dtype, device=device)
    _dev(t, name, dtype)
    if tuple(t.shape) != shape:
        raise ValueError(f"{name} must have shape {shape}, got {tuple(t.shape)}")
    if t.device != torch.device(device):
        raise ValueError(f"{name} must be on {device}, got {t.device}")
    return t


def _in(t, name, shape, dtype, device=None):
    """A required input, checked like _out (shape entries None = any)."""
    _dev(t, name, dtype)
    if len(t.shape) != len(shape) or any(s is not None and int(a) != int(s)
                                         for a, s in zip(t.shape, shape)):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    if device is not None and t.device != torch.device(device):
        raise ValueError(f"{name} must be on {device}, got {t.device}")
    return t


def _err(d_err, device):
    """The optional device error word: one int32 (the C ABI's uint32) on `device`."""
    if d_err is None:
        return None
    _dev(d_err, "d_err", torch.int32)
    if d_err.numel() < 1 or d_err.device != torch.device(device):
        raise ValueError(f"d_err must hold at least one int32 on {device}")
    return d_err


def _tree_batch(tree, B):
    if tree.B != B:
        raise ValueError(f"the tree holds {tree.B} trees but the call has batch {B}")


# Workspaces the binding allocates when the caller passes none: one per
# (device, stream), grown to the largest size asked for and kept for later
# calls (calls on one stream are ordered, so they can share it; the library
# accepts any contents).  release_workspaces() drops them.
_WS = {}


def release_workspaces():
    """Free the workspaces the binding allocated for calls without one."""
    _WS.clear()


def _workspace(nbytes, device, workspace, stream=None):
    if nbytes == 0:
        return None, 0
    if workspace is None:
        dev = torch.device(device)
        key = (dev.index, _stream_obj(stream, dev).cuda_stream)
        workspace = _WS.get(key)
        if workspace is None or workspace.numel() < nbytes:
            workspace = torch.empty(nbytes, dtype=torch.uint8, device=dev)
            _WS[key] = workspace
    _dev(workspace, "workspace")
    return workspace, workspace.numel() * workspace.element_size()


class TreeState:
    """Device-resident draft tree (the tg_tree SoA), one row of `cap` slots per
    batch element.  Slots [0, n_nodes[b]) are live; ids are topological."""

    FIELDS = ("parent", "token", "depth", "logp", "cum", "visited",
              "root_visited", "n_nodes")

    def __init__(self, B: int, cap: int, device="cuda"):
        dev = torch.device(device)
        self.B, self.cap = B, cap
        self.parent = torch.full((B, cap), -1, dtype=torch.int32, device=dev)
        self.token = torch.zeros((B, cap), dtype=torch.int32, device=dev)
        self.depth = torch.zeros((B, cap), dtype=torch.int32, device=dev)
        self.logp = torch.zeros((B, cap), dtype=torch.float32, device=dev)
        self.cum = torch.zeros((B, cap), dtype=torch.float32, device=dev)
        self.visited = torch.zeros((B, cap), dtype=torch.uint8, device=dev)
        self.root_visited = torch.zeros((B,), dtype=torch.uint8, device=dev)
        self.n_nodes = torch.zeros((B,), dtype=torch.int32, device=dev)

    @classmethod
    def from_host(cls, arrays: dict, cap: int, device="cuda") -> "TreeState":
        """Upload host arrays (numpy or torch) with the FIELDS names."""
        B = len(arrays["n_nodes"])
        t = cls(B, cap, device)
        for f in cls.FIELDS:
            src = torch.as_tensor(arrays[f])
            getattr(t, f).copy_(src.to(getattr(t, f).dtype))
        return t

    def to_host(self) -> dict:
        return {f: getattr(self, f).cpu().numpy() for f in self.FIELDS}

    def struct(self) -> TgTree:
        return TgTree(*(getattr(self, f).data_ptr() for f in self.FIELDS), self.cap)


# ----------------------------------------------------------------- calls

def verify_attention_workspace(B, N, Hq, Hkv, D, S_max, dtype) -> int:
    return load().tg_verify_attention_workspace(B, N, Hq, Hkv, D, S_max, dtype)


def verify_attention(q, k_cache, v_cache, parent, prefix_len, sm_scale, out=None,
                     workspace=None, d_err=None, stream=None):
    """Tree-verify attention; q [B,N,Hq,D], caches [B,Hkv,S_max,D] (bf16 or fp32)."""
    lib = load()
    if q.dtype == torch.bfloat16:
        dt = BF16
    elif q.dtype == torch.float32:
        dt = F32
    else:
        raise ValueError("q must be bfloat16 or float32")
    for t, n in ((q, "q"), (k_cache, "k_cache"), (v_cache, "v_cache")):
        _dev(t, n, q.dtype)
    _dev(parent, "parent", torch.int32)
    _dev(prefix_len, "prefix_len", torch.int32)
    B, N, Hq, D = q.shape
    Hkv, S_max = k_cache.shape[1], k_cache.shape[2]
    if tuple(k_cache.shape) != (B, Hkv, S_max, D) or v_cache.shape != k_cache.shape:
        raise ValueError("k_cache/v_cache must be [B, Hkv, S_max, D]")
    dev = q.device
    for t, n in ((k_cache, "k_cache"), (v_cache, "v_cache")):
        if t.device != dev:
            raise ValueError(f"{n} must be on {dev}, got {t.device}")
    _in(parent, "parent", (B, N), torch.int32, dev)
    _in(prefix_len, "prefix_len", (B,), torch.int32, dev)
    out = _out(out, "out", q.shape, q.dtype, dev)
    d_err = _err(d_err, dev)
    nbytes = lib.tg_verify_attention_workspace(B, N, Hq, Hkv, D, S_max, dt)
    ws, wsb = _workspace(nbytes, dev, workspace, stream)
    st = lib.tg_tree_verify_attention(_ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(parent),
                                      _ptr(prefix_len), _ptr(out), B, N, Hq, Hkv, D, S_max,
                                      float(sm_scale), dt, _ptr(ws), wsb, _ptr(d_err),
                                      _stream(stream, dev))
    _check("tg_tree_verify_attention", st)
    return out


def verify_attention_noalloc(q, k_cache, v_cache, parent, prefix_len, sm_scale, out=None,
                             d_err=None, stream=None):
    """tg_tree_verify_attention_noalloc: the same call without a workspace
    (the library's per-device scratch holds the split partials; shapes that
    need more than NOALLOC_SCRATCH_BYTES are rejected).  The binding allocates
    `out` only when the caller passes none."""
    lib = load()
    if q.dtype == torch.bfloat16:
        dt = BF16
    elif q.dtype == torch.float32:
        dt = F32
    else:
        raise ValueError("q must be bfloat16 or float32")
    for t, n in ((q, "q"), (k_cache, "k_cache"), (v_cache, "v_cache")):
        _dev(t, n, q.dtype)
    B, N, Hq, D = q.shape
    Hkv, S_max = k_cache.shape[1], k_cache.shape[2]
    if tuple(k_cache.shape) != (B, Hkv, S_max, D) or v_cache.shape != k_cache.shape:
        raise ValueError("k_cache/v_cache must be [B, Hkv, S_max, D]")
    dev = q.device
    for t, n in ((k_cache, "k_cache"), (v_cache, "v_cache")):
        if t.device != dev:
            raise ValueError(f"{n} must be on {dev}, got {t.device}")
    _in(parent, "parent", (B, N), torch.int32, dev)
    _in(prefix_len, "prefix_len", (B,), torch.int32, dev)
    out = _out(out, "out", q.shape, q.dtype, dev)
    d_err = _err(d_err, dev)
    st = lib.tg_tree_verify_attention_noalloc(_ptr(q), _ptr(k_cache), _ptr(v_cache),
                                              _ptr(parent), _ptr(prefix_len), _ptr(out), B, N,
                                              Hq, Hkv, D, S_max, float(sm_scale), dt,
                                              _ptr(d_err), _stream(stream, dev))
    _check("tg_tree_verify_attention_noalloc", st)
    return out


def expand_topk_workspace(B, F, V, K, N) -> int:
    return load().tg_expand_topk_workspace(B, F, V, K, N)


def expand_topk(tree: TreeState, logits, frontier, n_frontier, K, N, row_lse=None,
                next_frontier=None, n_next=None, workspace=None, d_err=None,
                stream=None):
    """One expansion step.  logits [B,F,V] fp32, frontier [B,F] int32,
    n_frontier [B] int32 or None.  Returns (row_lse, next_frontier, n_next)."""
    lib = load()
    _dev(logits, "logits", torch.float32)
    if logits.dim() != 3:
        raise ValueError("logits must be [B, F, V]")
    B, F, V = logits.shape
    dev = logits.device
    _tree_batch(tree, B)
    _in(frontier, "frontier", (B, F), torch.int32, dev)
    if n_frontier is not None:
        _in(n_frontier, "n_frontier", (B,), torch.int32, dev)
    row_lse = _out(row_lse, "row_lse", (B, F), torch.float32, dev)
    next_frontier = _out(next_frontier, "next_frontier", (B, N), torch.int32, dev)
    n_next = _out(n_next, "n_next", (B,), torch.int32, dev)
    d_err = _err(d_err, dev)
    ws, wsb = _workspace(lib.tg_expand_topk_workspace(B, F, V, K, N), dev, workspace, stream)
    ts = tree.struct()
    st = lib.tg_tree_expand_topk(ctypes.byref(ts), _ptr(logits), _ptr(frontier),
                                 _ptr(n_frontier), B, F, V, K, N, _ptr(row_lse),
                                 _ptr(next_frontier), _ptr(n_next), _ptr(ws), wsb,
                                 _ptr(d_err), _stream(stream, dev))
    _check("tg_tree_expand_topk", st)
    return row_lse, next_frontier, n_next


def ngram_cache_workspace(B, L, V, m) -> int:
    return load().tg_ngram_cache_workspace(B, L, V, m)


def ngram_cache(logits, context, ctx_len, m, cand_tok=None, cand_logp=None,
                fallback_pos=None, workspace=None, d_err=None, stream=None):
    """n-gram drafter prefill cache.  logits [B,L,V] fp32 (row i = after
    x_<=i), context [B,L] int32, ctx_len [B] int32.  Returns (cand_tok
    [B,L,m], cand_logp [B,L,m], fallback_pos [B])."""
    lib = load()
    _dev(logits, "logits", torch.float32)
    if logits.dim() != 3:
        raise ValueError("logits must be [B, L, V]")
    B, L, V = logits.shape
    dev = logits.device
    _in(context, "context", (B, L), torch.int32, dev)
    _in(ctx_len, "ctx_len", (B,), torch.int32, dev)
    cand_tok = _out(cand_tok, "cand_tok", (B, L, m), torch.int32, dev)
    cand_logp = _out(cand_logp, "cand_logp", (B, L, m), torch.float32, dev)
    fallback_pos = _out(fallback_pos, "fallback_pos", (B,), torch.int32, dev)
    d_err = _err(d_err, dev)
    ws, wsb = _workspace(lib.tg_ngram_cache_workspace(B, L, V, m), dev, workspace, stream)
    st = lib.tg_ngram_cache(_ptr(logits), _ptr(context), _ptr(ctx_len), B, L, V, m,
                            _ptr(cand_tok), _ptr(cand_logp), _ptr(fallback_pos), _ptr(ws), wsb,
                            _ptr(d_err), _stream(stream, dev))
    _check("tg_ngram_cache", st)
    return cand_tok, cand_logp, fallback_pos


def expand_ngram(tree: TreeState, frontier, n_frontier, context, ctx_len, cand_tok, cand_logp,
                 fallback_pos, K, N, n_max, match_pos=None, next_frontier=None, n_next=None,
                 d_err=None, stream=None):
    """One small-drafter step with the n-gram drafter (see
    tg_tree_expand_ngram).  Returns (next_frontier, n_next, match_pos)."""
    lib = load()
    _dev(frontier, "frontier", torch.int32)
    if frontier.dim() != 2:
        raise ValueError("frontier must be [B, F]")
    B, F = frontier.shape
    dev = frontier.device
    _tree_batch(tree, B)
    _in(context, "context", (B, None), torch.int32, dev)
    L = context.shape[1]
    _in(ctx_len, "ctx_len", (B,), torch.int32, dev)
    _in(cand_tok, "cand_tok", (B, L, None), torch.int32, dev)
    m = cand_tok.shape[2]
    _in(cand_logp, "cand_logp", (B, L, m), torch.float32, dev)
    _in(fallback_pos, "fallback_pos", (B,), torch.int32, dev)
    if n_frontier is not None:
        _in(n_frontier, "n_frontier", (B,), torch.int32, dev)
    match_pos = _out(match_pos, "match_pos", (B, F), torch.int32, dev)
    next_frontier = _out(next_frontier, "next_frontier", (B, N), torch.int32, dev)
    n_next = _out(n_next, "n_next", (B,), torch.int32, dev)
    d_err = _err(d_err, dev)
    ts = tree.struct()
    st = lib.tg_tree_expand_ngram(ctypes.byref(ts), _ptr(frontier), _ptr(n_frontier),
                                  _ptr(context), _ptr(ctx_len), _ptr(cand_tok), _ptr(cand_logp),
                                  _ptr(fallback_pos), B, F, L, m, K, N, n_max, _ptr(match_pos),
                                  _ptr(next_frontier), _ptr(n_next), _ptr(d_err),
                                  _stream(stream, dev))
    _check("tg_tree_expand_ngram", st)
    return next_frontier, n_next, match_pos


def rescore_graft_workspace(B, R, V, W, M, cap) -> int:
    return load().tg_rescore_graft_workspace(B, R, V, W, M, cap)


def rescore_graft(tree: TreeState, strong_logits, W, M, flags=0, row_lse=None,
                  graft_frontier=None, n_graft=None, N=0, next_frontier=None, n_next=None,
                  workspace=None, d_err=None, stream=None, new_from=None):
    """One middle-drafter step.  strong_logits [B,R,V] fp32 (row 0 = root,
    1+i = node i).  flags: POOL_NEWONLY (needs new_from [B] int32),
    GRAFT_OVERWRITE, GRAFT_DEDUP.  Returns (row_lse, graft_frontier,
    n_graft), plus (next_frontier, n_next) -- the best N grafted children --
    when N > 0."""
    lib = load()
    _dev(strong_logits, "strong_logits", torch.float32)
    if strong_logits.dim() != 3:
        raise ValueError("strong_logits must be [B, R, V]")
    B, R, V = strong_logits.shape
    dev = strong_logits.device
    _tree_batch(tree, B)
    if new_from is not None:
        _in(new_from, "new_from", (B,), torch.int32, dev)
    if row_lse is None:
        row_lse = torch.full((B, R), float("nan"), dtype=torch.float32, device=dev)
    row_lse = _out(row_lse, "row_lse", (B, R), torch.float32, dev)
    graft_frontier = _out(graft_frontier, "graft_frontier", (B, W), torch.int32, dev)
    n_graft = _out(n_graft, "n_graft", (B,), torch.int32, dev)
    if N > 0:
        next_frontier = _out(next_frontier, "next_frontier", (B, N), torch.int32, dev)
        n_next = _out(n_next, "n_next", (B,), torch.int32, dev)
    d_err = _err(d_err, dev)
    ws, wsb = _workspace(lib.tg_rescore_graft_workspace(B, R, V, W, M, tree.cap), dev,
                         workspace, stream)
    ts = tree.struct()
    st = lib.tg_tree_rescore_graft(ctypes.byref(ts), _ptr(strong_logits), B, R, V, W, M,
                                   int(flags), _ptr(new_from), _ptr(row_lse),
                                   _ptr(graft_frontier),
                                   _ptr(n_graft), _ptr(next_frontier if N > 0 else None),
                                   _ptr(n_next if N > 0 else None), int(N), _ptr(ws), wsb,
                                   _ptr(d_err), _stream(stream, dev))
    _check("tg_tree_rescore_graft", st)
    if N > 0:
        return row_lse, graft_frontier, n_graft, next_frontier, n_next
    return row_lse, graft_frontier, n_graft


def accept(parent, token, n_nodes, greedy, max_depth, accept_len=None, accept_path=None,
           bonus=None, d_err=None, stream=None):
    """Greedy acceptance.  parent/token [B,cap], n_nodes [B], greedy [B,cap+1].
    Returns (accept_len [B], accept_path [B,max_depth], bonus [B])."""
    lib = load()
    for t, n in ((parent, "parent"), (token, "token"), (n_nodes, "n_nodes"),
                 (greedy, "greedy")):
        _dev(t, n, torch.int32)
    if parent.dim() != 2:
        raise ValueError("parent must be [B, cap]")
    B, cap = parent.shape
    dev = parent.device
    _in(token, "token", (B, cap), torch.int32, dev)
    _in(n_nodes, "n_nodes", (B,), torch.int32, dev)
    _in(greedy, "greedy", (B, cap + 1), torch.int32, dev)
    accept_len = _out(accept_len, "accept_len", (B,), torch.int32, dev)
    accept_path = _out(accept_path, "accept_path", (B, max_depth), torch.int32, dev)
    bonus = _out(bonus, "bonus", (B,), torch.int32, dev)
    d_err = _err(d_err, dev)
    st = lib.tg_tree_accept(_ptr(parent), _ptr(token), _ptr(n_nodes), _ptr(greedy), B, cap,
                            max_depth, _ptr(accept_len), _ptr(accept_path), _ptr(bonus),
                            _ptr(d_err), _stream(stream, dev))
    _check("tg_tree_accept", st)
    return accept_len, accept_path, bonus


def accept_logits(parent, token, n_nodes, logits, max_depth, greedy=None, accept_len=None,
                  accept_path=None, bonus=None, d_err=None, stream=None):
    """Greedy acceptance from the target's logits [B,R,V] fp32 (row 0 = after
    the prefix, 1+i = after node i).  Returns (greedy [B,cap+1], accept_len,
    accept_path, bonus)."""
    lib = load()
    for t, n in ((parent, "parent"), (token, "token"), (n_nodes, "n_nodes")):
        _dev(t, n, torch.int32)
    _dev(logits, "logits", torch.float32)
    if parent.dim() != 2:
        raise ValueError("parent must be [B, cap]")
    B, cap = parent.shape
    dev = parent.device
    _in(token, "token", (B, cap), torch.int32, dev)
    _in(n_nodes, "n_nodes", (B,), torch.int32, dev)
    _in(logits, "logits", (B, None, None), torch.float32, dev)
    R, V = logits.shape[1], logits.shape[2]
    greedy = _out(greedy, "greedy", (B, cap + 1), torch.int32, dev)
    accept_len = _out(accept_len, "accept_len", (B,), torch.int32, dev)
    accept_path = _out(accept_path, "accept_path", (B, max_depth), torch.int32, dev)
    bonus = _out(bonus, "bonus", (B,), torch.int32, dev)
    d_err = _err(d_err, dev)
    st = lib.tg_tree_accept_logits(_ptr(parent), _ptr(token), _ptr(n_nodes), _ptr(logits), B,
                                   cap, R, V, max_depth, _ptr(greedy), _ptr(accept_len),
                                   _ptr(accept_path), _ptr(bonus), _ptr(d_err),
                                   _stream(stream, dev))
    _check("tg_tree_accept_logits", st)
    return greedy, accept_len, accept_path, bonus


def global_prune(tree: TreeState, B_ver: int, max_path: int | None = None, d_err=None,
                 stream=None, out=None):
    """Alg. 3 pruning of every tree to B_ver non-root nodes plus the
    verification buffers (see tg_tree_global_prune).  Returns a dict of device
    tensors: kept, vparent, vtoken [B, B_ver]; position_ids [B, B_ver+1];
    mask [B, B_ver+1, W] uint32 bitsets; retrieval [B, B_ver+1, max_path];
    n_keep, n_leaves [B]."""
    lib = load()
    B, dev = tree.B, tree.parent.device
    M = B_ver + 1
    max_path = M if max_path is None else int(max_path)
    shapes = dict(kept=(B, B_ver), vparent=(B, B_ver), vtoken=(B, B_ver), position_ids=(B, M),
                  mask=(B, M, (M + 31) // 32), retrieval=(B, M, max_path), n_keep=(B,),
                  n_leaves=(B,))
    out = {} if out is None else out
    out = {k: _out(out.get(k), f"out['{k}']", shp, torch.int32, dev) for k, shp in shapes.items()}
    d_err = _err(d_err, dev)
    ts = tree.struct()
    st = lib.tg_tree_global_prune(ctypes.byref(ts), B, int(B_ver), max_path,
                                  *(_ptr(out[k]) for k in ("kept", "vparent", "vtoken",
                                                           "position_ids", "mask", "retrieval",
                                                           "n_keep", "n_leaves")),
                                  _ptr(d_err), _stream(stream, dev))
    _check("tg_tree_global_prune", st)
    return out


def kv_compact(k_cache, v_cache, prefix_len, path, n_path, new_prefix_len=None, d_err=None,
               stream=None):
    """Move the accepted chain's K/V rows to the end of the prefix, in place
    (see tg_kv_compact).  k_cache/v_cache [B, Hkv, S_max, D] (bf16 or fp32);
    path [B, max_path]; prefix_len, n_path [B].  Returns new_prefix_len [B]."""
    lib = load()
    _dev(k_cache, "k_cache")
    _dev(v_cache, "v_cache")
    if (k_cache.shape != v_cache.shape or k_cache.dtype != v_cache.dtype or
            k_cache.device != v_cache.device or k_cache.dim() != 4):
        raise ValueError("k_cache and v_cache must be matching [B, Hkv, S_max, D] tensors")
    if k_cache.dtype not in (torch.bfloat16, torch.float32):
        raise ValueError("k_cache must be bfloat16 or float32")
    B, Hkv, S_max, D = k_cache.shape
    dev = k_cache.device
    _in(prefix_len, "prefix_len", (B,), torch.int32, dev)
    _in(path, "path", (B, None), torch.int32, dev)
    _in(n_path, "n_path", (B,), torch.int32, dev)
    dt = {torch.bfloat16: BF16, torch.float32: F32}[k_cache.dtype]
    new_prefix_len = _out(new_prefix_len, "new_prefix_len", (B,), torch.int32, dev)
    d_err = _err(d_err, dev)
    st = lib.tg_kv_compact(_ptr(k_cache), _ptr(v_cache), _ptr(prefix_len), _ptr(path),
                           _ptr(n_path), B, Hkv, S_max, D, path.shape[1], dt,
                           _ptr(new_prefix_len), _ptr(d_err), _stream(stream, dev))
    _check("tg_kv_compact", st)
    return new_prefix_len


def tree_signals(tree: TreeState, frontier, n_frontier, W: int, lookback: int = 5,
                 context=None, params=None, d_err=None, stream=None, signals=None,
                 margin=None, action=None):
    """The ten pre-action tree signals per tree (see tg_tree_signals), and
    with `params` (3265 fp32 predictor weights) and `context` [B, 11] the
    margin [B] and action [B].  frontier [B, F] int32 (-1 = root);
    n_frontier [B] or None.  Returns (signals [B, 10], margin, action)."""
    lib = load()
    _dev(frontier, "frontier", torch.int32)
    if frontier.dim() != 2:
        raise ValueError("frontier must be [B, F]")
    B, F = frontier.shape
    dev = frontier.device
    _tree_batch(tree, B)
    if n_frontier is not None:
        _in(n_frontier, "n_frontier", (B,), torch.int32, dev)
    sig = _out(signals, "signals", (B, 10), torch.float32, dev)
    if params is not None:
        _in(params, "params", (3265,), torch.float32, dev)
        if context is None:
            raise ValueError("context [B, 11] is required with params")
        _in(context, "context", (B, 11), torch.float32, dev)
        margin = _out(margin, "margin", (B,), torch.float32, dev)
        action = _out(action, "action", (B,), torch.int32, dev)
    else:
        margin = action = None
    d_err = _err(d_err, dev)
    ts = tree.struct()
    st = lib.tg_tree_signals(ctypes.byref(ts), _ptr(frontier), _ptr(n_frontier), B, F, int(W),
                             int(lookback), _ptr(context), _ptr(params), _ptr(sig),
                             _ptr(margin), _ptr(action), _ptr(d_err), _stream(stream, dev))
    _check("tg_tree_signals", st)
    return sig, margin, action


def tree_reset(tree: TreeState, stream=None):
    """Empty every tree (n_nodes = 0, root unvisited) with a device kernel."""
    lib = load()
    ts = tree.struct()
    _check("tg_tree_reset", lib.tg_tree_reset(ctypes.byref(ts), tree.B,
                                              _stream(stream, tree.parent.device)))


def trace_begin(capacity: int = 4096):
    """Turn on per-kernel device timing (see tg_trace_begin)."""
    _check("tg_trace_begin", load().tg_trace_begin(int(capacity)))


def trace_read(max_records: int = 1 << 16):
    """Current per-kernel records without ending the trace (see tg_trace_read)."""
    lib = load()
    recs = (TgTraceRecord * max_records)()
    n = ctypes.c_int(0)
    _check("tg_trace_read", lib.tg_trace_read(recs, max_records, ctypes.byref(n)))
    return [(recs[i].kernel.decode(), float(recs[i].ms)) for i in range(n.value)]


def trace_end(max_records: int = 1 << 16):
    """Turn tracing off; returns [(kernel name, milliseconds)] in launch order."""
    lib = load()
    recs = (TgTraceRecord * max_records)()
    n = ctypes.c_int(0)
    _check("tg_trace_end", lib.tg_trace_end(recs, max_records, ctypes.byref(n)))
    return [(recs[i].kernel.decode(), float(recs[i].ms)) for i in range(n.value)]
