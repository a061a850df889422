"""Pins of the tree-signal and margin-predictor oracle (CPU)."""
from __future__ import annotations

import json
import os

import numpy as np
import pytest
import torch

import workloads as W
from oracle import signals as OS
from tests import _cases as C

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def test_signals_golden():
    gd = json.load(open(os.path.join(GOLD, "tree_signals.json")))
    par = np.array(gd["parent"])
    dep = np.array(gd["depth"])
    for c in gd["cases"]:
        cum = np.array([float(x) for x in c["cum"]], np.float32)
        sig, prev = OS.tree_signals(par, dep, cum, len(par), c["frontier"], c["W"], c["L"])
        assert prev == c["preview"]
        assert np.allclose(sig, c["signals"], rtol=0, atol=1e-6)


@pytest.mark.parametrize("seed", range(4))
def test_frontier_equal_to_its_preview(seed):
    """With L = 0 and F = the top-W nodes of one depth, R is that depth and
    the preview is F itself: overlap 1, no depth change, no debt, no past
    depths."""
    tree, _ = C.scored_tree(800 + seed, 1, 50, steps=4, width=5, K=3)
    n = int(tree.n_nodes[0])
    par, dep, cum = tree.parent[0, :n], tree.depth[0, :n], tree.cum[0, :n]
    d = int(dep.max())
    at_d = [v for v in range(n) if dep[v] == d]
    top = sorted(at_d, key=lambda v: (-float(cum[v]), v))[:3]
    sig, prev = OS.tree_signals(par, dep, cum, n, top, len(top), 0)
    s = dict(zip(OS.NAMES, sig))
    assert sorted(prev) == sorted(top)
    assert s["pre_reselect_overlap"] == 1.0
    assert s["pre_reselect_depth_delta"] == 0.0 and s["collapse_debt"] == 0.0
    assert s["pre_reselect_past_ratio"] == 0.0
    assert s["pre_reselect_cands"] == len(at_d)
    assert s["depth_before"] == s["max_depth_before"] == d


@pytest.mark.parametrize("seed", range(6))
def test_signal_ranges_on_random_trees(seed):
    g = W.rng(820 + seed)
    n = int(g.integers(1, 200))
    par = W.uniform_parents(g, n)
    dep = W.node_depths(par)
    cum = -np.abs(W.normal(g, (n,), 2.0)).astype(np.float32)
    cum[g.random(n) < 0.1] = -np.inf
    F = list(g.choice(np.arange(-1, n), size=min(n, 8), replace=False))
    Wd, L = int(g.integers(1, 12)), int(g.integers(0, 6))
    sig, prev = OS.tree_signals(par, dep, cum, n, F, Wd, L)
    s = dict(zip(OS.NAMES, sig))
    for k in ("leaf_ratio_before", "pre_reselect_past_ratio", "pre_reselect_overlap",
              "finite_score_ratio_before"):
        assert 0.0 <= s[k] <= 1.0
    assert s["collapse_debt"] == max(0.0, -s["pre_reselect_depth_delta"])
    assert len(prev) == min(Wd, int(s["pre_reselect_cands"]))
    assert s["max_depth_before"] >= s["depth_before"]


def test_margin_matches_torch_mlp():
    """The predictor is Linear(17,64)-ReLU-Linear(64,32)-ReLU-Linear(32,1)
    with 3,265 parameters; compared against torch.nn on the CPU."""
    g = W.rng(830)
    net = torch.nn.Sequential(torch.nn.Linear(17, 64), torch.nn.ReLU(), torch.nn.Linear(64, 32),
                              torch.nn.ReLU(), torch.nn.Linear(32, 1)).double()
    assert sum(p.numel() for p in net.parameters()) == OS.N_PARAMS == 3265
    with torch.no_grad():
        for prm in net.parameters():
            prm.copy_(torch.from_numpy(W.normal(g, tuple(prm.shape), 0.3)))
    packed = np.concatenate([net[0].weight.detach().numpy().ravel(), net[0].bias.detach().numpy(),
                             net[2].weight.detach().numpy().ravel(), net[2].bias.detach().numpy(),
                             net[4].weight.detach().numpy().ravel(), net[4].bias.detach().numpy()])
    for _ in range(20):
        ctx = W.normal(g, (11,), 1.0)
        sig = W.normal(g, (10,), 1.0)
        y, act = OS.margin(ctx, sig, packed)
        x = np.concatenate([ctx, [sig[OS.NAMES.index(k)] for k in OS.SELECTED]])
        ref = float(net(torch.from_numpy(x.astype(np.float64))[None])[0, 0])
        assert abs(y - ref) < 1e-12 and act == int(ref > 0)
