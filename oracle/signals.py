"""Oracle for the scheduler's tree signals and margin predictor (test
infrastructure only).

Definitions followed (App. B.2, the table of candidate tree signals; App.
B.4, the margin predictor):

  F      the current frontier (node ids, -1 = root; taken as given)
  d(v)   depth (root 0), s(v) cumulative path score, child(v) children
  D_F    = {d(v) : v in F}
  D_C    = union over d in D_F of {x : max(0, d - L) <= x <= d}
  R      = {v in V(T), root included : d(v) in D_C}
  F^     = Top_W(R, s)   preview frontier, ranked by (s desc, depth asc,
           id asc) with the root as id -1 (the tie-break used everywhere)

  depth_before              mean_{v in F} d(v)
  leaf_ratio_before         mean_{v in F} [child(v) empty]
  pre_reselect_depth_delta  mean_{F^} d - mean_{F} d
  pre_reselect_cands        |R|
  max_depth_before          max_{F} d
  collapse_debt             max(0, -pre_reselect_depth_delta)
  pre_reselect_past_ratio   mean_{v in F^} [d(v) not in D_F]
  pre_reselect_overlap      |F^ intersect F| / |F^|
  pre_reselect_score        mean of s(v) over v in F^ with s(v) finite
  finite_score_ratio_before mean_{v in F} [s(v) finite]

Reading where the paper is silent: s(v) is the stored log-domain score
(``cum``; the root's is 0), which is what makes "finite" meaningful (a path
through a zero-probability token has cum = -inf).  An empty mean is NaN (the
paper discards states with a non-finite signal).  The margin predictor is
Linear(17,64) -> ReLU -> Linear(64,32) -> ReLU -> Linear(32,1) on
x = [runtime context (4), history (7), the selected six signals in the order
depth_before, leaf_ratio_before, collapse_debt, pre_reselect_past_ratio,
pre_reselect_overlap, pre_reselect_score]; action = 1 (call) iff margin > 0.
Weights are packed row-major W1[64,17], b1[64], W2[32,64], b2[32], W3[1,32],
b3[1] (3265 numbers).
"""
from __future__ import annotations

import numpy as np

from .tree import node_key

NAMES = ("depth_before", "leaf_ratio_before", "pre_reselect_depth_delta",
         "pre_reselect_cands", "max_depth_before", "collapse_debt",
         "pre_reselect_past_ratio", "pre_reselect_overlap", "pre_reselect_score",
         "finite_score_ratio_before")
SELECTED = ("depth_before", "leaf_ratio_before", "collapse_debt",
            "pre_reselect_past_ratio", "pre_reselect_overlap", "pre_reselect_score")
N_PARAMS = 64 * 17 + 64 + 32 * 64 + 32 + 32 + 1


def _mean(xs):
    xs = list(xs)
    return float(np.mean(xs)) if xs else float("nan")


def tree_signals(parent, depth, cum, n, frontier, W, L):
    """The ten signals of one tree (n nodes; frontier = list of ids, -1 = root)."""
    par = [int(p) for p in parent[:n]]
    dep = {-1: 0}
    sc = {-1: 0.0}
    for v in range(n):
        dep[v] = int(depth[v])
        sc[v] = float(cum[v])
    children = {v: 0 for v in range(-1, n)}
    for v in range(n):
        children[par[v]] += 1
    F = [int(v) for v in frontier]
    DF = {dep[v] for v in F}
    DC = set()
    for d in DF:
        DC.update(range(max(0, d - L), d + 1))
    R = [v for v in range(-1, n) if dep[v] in DC]
    ranked = sorted(R, key=lambda v: node_key(sc[v], dep[v], v))
    Fh = ranked[:W]
    mean_f = _mean(dep[v] for v in F)
    mean_h = _mean(dep[v] for v in Fh)
    delta = mean_h - mean_f
    out = {
        "depth_before": mean_f,
        "leaf_ratio_before": _mean(1.0 if children[v] == 0 else 0.0 for v in F),
        "pre_reselect_depth_delta": delta,
        "pre_reselect_cands": float(len(R)),
        "max_depth_before": float(max(dep[v] for v in F)) if F else float("nan"),
        "collapse_debt": max(0.0, -delta) if delta == delta else float("nan"),
        "pre_reselect_past_ratio": _mean(0.0 if dep[v] in DF else 1.0 for v in Fh),
        "pre_reselect_overlap": (len(set(Fh) & set(F)) / len(Fh)) if Fh else float("nan"),
        "pre_reselect_score": _mean(sc[v] for v in Fh if np.isfinite(sc[v])),
        "finite_score_ratio_before": _mean(1.0 if np.isfinite(sc[v]) else 0.0 for v in F),
    }
    return np.array([out[k] for k in NAMES], dtype=np.float64), Fh


def unpack(params):
    p = np.asarray(params, dtype=np.float64)
    assert p.size == N_PARAMS
    o = 0
    W1 = p[o:o + 64 * 17].reshape(64, 17); o += 64 * 17
    b1 = p[o:o + 64]; o += 64
    W2 = p[o:o + 32 * 64].reshape(32, 64); o += 32 * 64
    b2 = p[o:o + 32]; o += 32
    W3 = p[o:o + 32].reshape(1, 32); o += 32
    b3 = p[o:o + 1]
    return W1, b1, W2, b2, W3, b3


def margin(context, signals, params):
    """Margin predictor on one state: context [11] (runtime 4 + history 7),
    signals [10] in NAMES order.  Returns (margin, action)."""
    x = np.concatenate([np.asarray(context, np.float64),
                        [signals[NAMES.index(k)] for k in SELECTED]])
    W1, b1, W2, b2, W3, b3 = unpack(params)
    h1 = np.maximum(W1 @ x + b1, 0.0)
    h2 = np.maximum(W2 @ h1 + b2, 0.0)
    y = float((W3 @ h2 + b3)[0])
    return y, int(y > 0)
