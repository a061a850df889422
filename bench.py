#!/usr/bin/env python3
"""Benchmark of the tree-verify / tree-expand hot path on one MI355X.

Headline (one step = one call of tg_tree_verify_attention): the
Llama-3-70B-shaped verify layer, the largest single-GPU workload - batch 8,
64 query heads / 8 KV heads, head_dim 128, bf16, a 32768-token prefix per
sequence and a 256-node draft tree per sequence (12 levels, at most 8
children per node), Q/K/V i.i.d. N(0,1).  This is target-side verification,
the largest per-call cost of a decoding turn.  `value` is the call's
algorithmic flops (4 * D per (query row, visible key); ancestors only) per
second with every input resident in HBM; `roofline` is the ping-pong
attention kernel's own launch time, taken with HIP events on the launch
stream around the timed calls (one kernel per call at this shape).

Besides the headline, the default run measures every other workload once and
reports each under `extra` with its own roofline and CPU baseline:
  tiny                the tiny fp32 workload: attention (B1, 4/4 heads, D64,
                      prefix 128, 16 nodes), one expansion (V=1000, F=8, K=4,
                      N=8) and acceptance, as one step (microseconds), timed
                      as a replayed HIP graph of steps (the eager time beside)
  attn-llama8b        the Llama-3-8B-shaped verify layer (B1, 32/8 heads,
                      prefix 2048, 64 nodes) - one call (split-prefix mode),
                      timed as a replayed HIP graph of calls (the eager loop
                      would time Python's per-call marshalling)
  attn-llama8b-x32    32 independent layers of that shape back to back
                      (310 MB), one HIP graph per step: the steady-state
                      bandwidth the single call's latency hides
  attn-longctx        long-context verify (B4, 32/8 heads, prefix 8192, 128
                      nodes of 10 levels)
  expand-twodrafter   two-drafter expansion: B8 trees of 256 nodes (a 5-step
                      weak top-10 / frontier-10 expansion pruned by Alg. 3),
                      the 64 best leaves expanded (K=10, N=60), V=128256
  rescore-twodrafter  the middle step on the same trees (257 strong rows,
                      W=60, m=10; strong = 0.8 weak + 0.6 noise)
  turn                one TreeGraft turn (schedule [1,0,1,0,1], n-gram small
                      drafter, scheduler signals, GlobalPrune to 64 nodes,
                      Llama-3-8B verify layer, accept, KV update), replayed as
                      one HIP graph
  turn-standard       the standard-construction turn (Alg. 1): six expansion
                      steps over dense logits (root, then 10-node frontiers,
                      K=8, N=10), GlobalPrune to 64 nodes, the same verify
                      layer, accept and KV update, replayed as one HIP graph
`--workload NAME` times only that workload as the headline; `--only` skips
the extras.  All inputs are seeded synthetic data with the workloads' shapes
and distributions (no model weights or datasets).  The CPU baselines time the
oracle (the tests' plain CPU reference, untuned) on a bounded sample of the
same inputs on this machine's host cores, and report how far the GPU result
is from it.

Prints ONE JSON line.  One GPU only: --gpus N > 1 exits with a message.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "tree-verify attention TB/s & TFLOP/s (% roofline); draft-tree nodes/sec"
PEAK_HBM = 8.0e12        # B/s, MI355X HBM3E
PEAK_BF16 = 2.5e15       # flop/s, dense bf16 MFMA
PEAK_FP32 = 157.3e12     # flop/s, fp32 vector
ATTN_MAIN = ("attn_pingpong", "attn_mfma", "attn_f32")   # tree-verify attention kernels
WORKLOADS = ["attn-llama70b", "tiny", "attn-llama8b", "attn-llama8b-x32", "attn-longctx",
             "expand-twodrafter", "rescore-twodrafter", "turn", "turn-standard"]


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="attn-llama70b", choices=WORKLOADS,
                    help="the headline workload (default: the Llama-3-70B-shaped layer)")
    ap.add_argument("--only", action="store_true", help="measure the headline workload only")
    ap.add_argument("--copies", type=int, default=4, help="turn: resident input copies")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="approximate CPU time of the headline's oracle baseline")
    ap.add_argument("--extra-cpu-seconds", type=float, default=3.0,
                    help="approximate CPU time of each extra workload's oracle baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration-mb", type=int, default=0,
                    help="profiling aid: run one device copy of this many MiB first, so a "
                         "counter pass can scale FETCH_SIZE/WRITE_SIZE by a known size")
    ap.add_argument("--rescore-flags", type=int, default=0,
                    help="rescore-twodrafter: middle-step variant flags (1 = pool of the "
                         "previous step's new nodes, 2 = overwriting graft, 4 = skip "
                         "duplicate siblings; the Sec. 5.3 ablations and a filter)")
    return ap.parse_args()


# ------------------------------------------------------- measured traffic

def profile_traffic(name):
    """HBM bytes per launch from a committed counter summary
    (profiles/<name>), or None when the kernel sources listed there no longer
    hash to the recorded value (the counters describe an older kernel)."""
    import hashlib
    path = os.path.join(ROOT, "profiles", name)
    try:
        fields = {}
        for line in open(path):
            if line.startswith("traffic_") and ":" in line:
                k, v = line.split(":", 1)
                fields[k.strip()] = v.strip()
        h = hashlib.sha256()
        for src in fields["traffic_sources"].split(","):
            with open(os.path.join(ROOT, src), "rb") as f:
                h.update(f.read())
        if h.hexdigest() != fields["traffic_sha256"]:
            return None
        return float(fields["traffic_bytes_per_launch"])
    except (OSError, KeyError, ValueError):
        return None


TRAFFIC_FILES = {
    ("attn-llama70b", "attn_pingpong"): "attn_pingpong_llama70b_traffic.md",
    ("attn-longctx", "attn_pingpong"): "attn_pingpong_longctx_traffic.md",
    ("expand-twodrafter", "row_partial"): "row_partial_expand_twodrafter_traffic.md",
    ("rescore-twodrafter", "row_partial"): "row_partial_rescore_twodrafter_traffic.md",
    ("turn", "row_partial"): "row_partial_turn_llama8b_traffic.md",
}


def traffic_for(workload, kernel):
    f = TRAFFIC_FILES.get((workload, kernel))
    return profile_traffic(f) if f else None


# ------------------------------------------------------------ timing

def time_calls(torch, fn, steps, warmup):
    """Average milliseconds of fn() over `steps` calls (after `warmup`),
    bracketed by HIP events on the current stream, the stream the library
    launches on, with a device synchronisation on both sides."""
    for i in range(warmup):
        fn(i)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(steps):
        fn(warmup + i)
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / steps


def time_graph(torch, fn, n_calls, reps, warmup):
    """Milliseconds per replay of one HIP graph holding fn(0) .. fn(n_calls-1),
    captured after one eager pass and replayed `warmup` times untimed, then
    `reps` times between HIP events: the device time of calls whose Python
    marshalling takes longer than the kernels, as a serving loop that
    replays graphs sees it."""
    for i in range(n_calls):
        fn(i)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for i in range(n_calls):
            fn(i)
    for _ in range(warmup):
        g.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / reps, g


def kernel_times(tg, torch, fn, steps, start=0):
    """Per-kernel device times of `steps` eager calls from the library's trace
    events (an event pair on the launch stream around each kernel; a separate
    pass from the timed one).  Returns {kernel: [launches, total ms]}."""
    torch.cuda.synchronize()
    tg.trace_begin(64 * (steps + 1))
    try:
        for i in range(steps):
            fn(start + i)
        torch.cuda.synchronize()
    finally:
        recs = tg.trace_end()
    kern = {}
    for name, ms in recs:
        d = kern.setdefault(name, [0, 0.0])
        d[0] += 1
        d[1] += ms
    return kern, recs


def kernels_json(kern, steps):
    return {k: {"launches_per_step": v[0] / steps, "avg_us": 1e3 * v[1] / v[0],
                "us_per_step": 1e3 * v[1] / steps} for k, v in kern.items()}


def blas_threads():
    try:
        from threadpoolctl import threadpool_info
        return max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        return 1


def line(value, unit, steps, warmup, ms, config, roofline, dtype, higher=True, **extra):
    out = {"metric": METRIC, "value": value, "unit": unit, "n_gpus": 1, "steps": steps,
           "warmup": warmup, "ms_per_step": ms, "higher_is_better": higher, "scaling": "weak",
           "vs_baseline": None, "dtype": dtype, "data": "synthetic", "config": config,
           "roofline": roofline}
    out.update(extra)
    return out


# ------------------------------------------------------- attention alone

ATTN_SHAPES = {
    # name: (B, Hq, Hkv, D, prefix, nodes, levels, qkv scale, dtype, description)
    "attn-llama70b": (8, 64, 8, 128, 32768, 256, 12, 1.0, "bf16",
                      "Llama-3-70B-shaped verify layer"),
    "attn-longctx": (4, 32, 8, 128, 8192, 128, 10, 1.0, "bf16", "long-context verify layer"),
    "attn-llama8b": (1, 32, 8, 128, 2048, 64, None, 1.0 / np.sqrt(128.0), "bf16",
                     "Llama-3-8B-shaped verify layer"),
    "tiny": (1, 4, 4, 64, 128, 16, "uniform", 1.0, "f32", "tiny fp32 verify layer"),
}


def attn_parents(name, g):
    Bq, _, _, _, _, Nn, levels, _, _, _ = ATTN_SHAPES[name]
    import workloads as W
    if levels is None:         # root + draft nodes shaped like a pruned expansion
        return np.stack([W.verify_layout_with_root(W.expansion_shaped_tree(g, Nn - 1, 6, 8, 10))
                         for _ in range(Bq)]).astype(np.int32)
    if levels == "uniform":
        return np.stack([W.uniform_parents(g, Nn) for _ in range(Bq)]).astype(np.int32)
    return np.stack([W.level_tree(g, Nn, levels, 8) for _ in range(Bq)]).astype(np.int32)


def path_len_sum(vpar):
    """Sum over nodes of the number of tree keys a node attends to (its
    ancestors and itself)."""
    tot = 0
    for i in range(len(vpar)):
        u = i
        while u != -1:
            tot += 1
            u = int(vpar[u])
    return tot


def attn_work(name, par):
    """Algorithmic bytes (each K/V element read once, Q read, O written, the
    parent array) and flops (4 * D per (query row, visible key), ancestors
    only) of one call."""
    Bq, Hq, Hkv, Dh, Lp, Nn, _, _, dt, _ = ATTN_SHAPES[name]
    es = 2 if dt == "bf16" else 4
    keys = sum(Nn * Lp + path_len_sum(par[b]) for b in range(Bq))
    flops = 4 * Dh * Hq * keys
    nbytes = 2 * Bq * Hkv * (Lp + Nn) * Dh * es + 2 * Bq * Nn * Hq * Dh * es + par.nbytes
    return nbytes, flops


def attn_inputs(torch, dev, name, n_copies, seed=2000):
    import workloads as W
    Bq, Hq, Hkv, Dh, Lp, Nn, _, scale, dt, _ = ATTN_SHAPES[name]
    dtype = torch.bfloat16 if dt == "bf16" else torch.float32
    S = Lp + Nn
    bufs = []
    for c in range(n_copies):
        gc = W.rng([seed, c])
        q = torch.empty((Bq, Nn, Hq, Dh), dtype=dtype, device=dev)
        k = torch.empty((Bq, Hkv, S, Dh), dtype=dtype, device=dev)
        v = torch.empty((Bq, Hkv, S, Dh), dtype=dtype, device=dev)
        for b in range(Bq):     # per-sequence draws keep host memory small
            q[b] = torch.from_numpy(W.normal(gc, (Nn, Hq, Dh)) * np.float32(scale)).to(dev)
            k[b] = torch.from_numpy(W.normal(gc, (Hkv, S, Dh)) * np.float32(scale)).to(dev)
            v[b] = torch.from_numpy(W.normal(gc, (Hkv, S, Dh)) * np.float32(scale)).to(dev)
        bufs.append((q, k, v, torch.empty_like(q)))
    return bufs


def attn_cpu_baseline(name, par, buf, budget_s):
    """The oracle on whole (batch, KV head) groups of input copy 0, in a fixed
    seeded order, until about `budget_s` seconds are spent; also the GPU's
    error against it on those groups (max abs, tensor-relative Frobenius)."""
    from oracle.attention import tree_verify_attention_fast
    import workloads as W
    Bq, Hq, Hkv, Dh, Lp, Nn, _, _, _, _ = ATTN_SHAPES[name]
    G = Hq // Hkv
    q, k, v, o = buf
    order = W.rng(77).permutation(Bq * Hkv)
    flops = nbytes = 0
    done, err_abs, num, den = 0, 0.0, 0.0, 0.0
    t_cpu = 0.0
    for gi in order:
        b, g0 = divmod(int(gi), Hkv)
        qh = q[b:b + 1, :, g0 * G:(g0 + 1) * G].float().cpu().numpy()
        kh = k[b:b + 1, g0:g0 + 1].float().cpu().numpy()
        vh = v[b:b + 1, g0:g0 + 1].float().cpu().numpy()
        t0 = time.perf_counter()
        want = tree_verify_attention_fast(qh, kh, vh, par[b:b + 1], [Lp], Dh ** -0.5)
        t_cpu += time.perf_counter() - t0
        got = o[b:b + 1, :, g0 * G:(g0 + 1) * G].float().cpu().numpy().astype(np.float64)
        err_abs = max(err_abs, float(np.abs(got - want).max()))
        num += float(((got - want) ** 2).sum())
        den += float((want ** 2).sum())
        flops += 4 * Dh * G * (Nn * Lp + path_len_sum(par[b]))
        nbytes += 2 * (Lp + Nn) * Dh * 2 + 2 * Nn * G * Dh * 2
        done += 1
        if t_cpu >= budget_s:
            break
    parity = {"groups_checked": done, "groups_total": Bq * Hkv, "max_abs_err": err_abs,
              "rel_fro_err": (num / den) ** 0.5 if den > 0 else 0.0,
              "bars": {"max_abs": 2e-2, "rel_fro": 1e-2}}
    return flops, nbytes, t_cpu, done, parity


def attention_bench(tg, torch, dev, name, steps, warmup, cpu_s):
    """tg_tree_verify_attention alone at one workload shape; inputs rotate over
    enough copies to exceed 512 MB so no timed read hits the 256 MB MALL."""
    import workloads as W
    Bq, Hq, Hkv, Dh, Lp, Nn, _, _, dt, desc = ATTN_SHAPES[name]
    es = 2 if dt == "bf16" else 4
    par = attn_parents(name, W.rng(2000))
    per_copy = 2 * Bq * Hkv * (Lp + Nn) * Dh * es
    copies = max(1, min(8, -(-(512 << 20) // per_copy)))
    bufs = attn_inputs(torch, dev, name, copies)
    parent = torch.from_numpy(par).to(dev)
    plen = torch.full((Bq,), Lp, dtype=torch.int32, device=dev)
    nws = tg.verify_attention_workspace(Bq, Nn, Hq, Hkv, Dh, Lp + Nn,
                                        tg.BF16 if dt == "bf16" else tg.F32)
    ws = torch.empty(max(nws, 1), dtype=torch.uint8, device=dev)

    def call(i):
        q, k, v, o = bufs[i % copies]
        tg.verify_attention(q, k, v, parent, plen, Dh ** -0.5, out=o, workspace=ws)

    ms = time_calls(torch, call, steps, warmup)
    timing = {"timing": "eager calls"}
    if name == "attn-llama8b":
        # a call's Python marshalling outlasts its ~15 us of kernels: the
        # eager loop measures the host, so the step is timed as one graph of
        # the copies' calls, replayed; the replay must give the eager output
        call(0)
        torch.cuda.synchronize()
        want = bufs[0][3].clone()
        ms_eager = ms
        ms_rep, graph = time_graph(torch, call, copies, max(1, steps), warmup)
        ms = ms_rep / copies
        if not torch.equal(bufs[0][3], want):
            raise RuntimeError("graph replay of the verify call differs from the eager call")
        del graph
        timing = {"timing": f"one HIP graph of the {copies} input copies' calls, replayed "
                            f"{max(1, steps)} times", "eager_ms_per_call": ms_eager}
    kern, _ = kernel_times(tg, torch, call, steps, start=0)
    call(0)                       # copy 0's output for the parity margin
    torch.cuda.synchronize()
    main_k = next(k for k in ATTN_MAIN if k in kern)
    nbytes, flops = attn_work(name, par)
    one_kernel = len(kern) == 1 and kern[main_k][0] == steps
    # the main kernel's launch time: the timed pass itself when a call is
    # that one kernel, else the trace pass's event pairs around it
    main_us = 1e3 * ms if one_kernel else 1e3 * kern[main_k][1] / kern[main_k][0]
    if dt == "f32":
        bound = "hbm" if nbytes / PEAK_HBM > flops / PEAK_FP32 else "alu"
    else:
        bound = "mfma" if flops / nbytes > PEAK_BF16 / PEAK_HBM else "hbm"
    if bound == "mfma":
        ach, peak, unit = flops / (main_us * 1e-6) / 1e12, PEAK_BF16 / 1e12, "TFLOP/s"
    elif bound == "alu":
        ach, peak, unit = flops / (main_us * 1e-6) / 1e12, PEAK_FP32 / 1e12, "TFLOP/s"
    else:
        ach, peak, unit = nbytes / (main_us * 1e-6) / 1e9, PEAK_HBM / 1e9, "GB/s"
    roof = {"bound": bound, "kernel": main_k, "achieved": ach, "peak": peak, "unit": unit,
            "frac": ach / peak, "traffic": traffic_for(name, main_k),
            "avg_launch_us": main_us,
            "launch_time_from": "timed pass (one kernel per call)" if one_kernel
            else "trace pass (event pair around each kernel)"}
    call_s = ms * 1e-3
    if bound == "hbm":
        value, vunit = nbytes / call_s / 1e12, "TB/s"
    else:
        value, vunit = flops / call_s / 1e12, "TFLOP/s"
    out = line(value, vunit, steps, warmup, ms,
               {"workload": f"{desc} (B{Bq}, {Hq}/{Hkv} heads, D{Dh}, prefix {Lp}, "
                            f"{Nn} tree nodes, {dt})", "batch": Bq, "q_heads": Hq,
                "kv_heads": Hkv, "head_dim": Dh, "prefix": Lp, "tree_nodes": Nn,
                "input_copies": copies},
               roof, dt, **{"TB/s": nbytes / call_s / 1e12, "TFLOP/s": flops / call_s / 1e12,
                            "bytes": nbytes, "flops": flops,
                            "kernels": kernels_json(kern, steps)}, **timing)
    if cpu_s > 0:
        f_cpu, b_cpu, t_cpu, done, parity = attn_cpu_baseline(name, par, bufs[0], cpu_s)
        out["cpu_baseline"] = {
            "value": (b_cpu if bound == "hbm" else f_cpu) / t_cpu / 1e12, "unit": vunit,
            "cores": blas_threads(), "kind": "oracle",
            "sample": f"{done} of {Bq * Hkv} (batch, KV head) groups of the same inputs in "
                      f"{t_cpu:.1f} s (fp64 NumPy; its matrix products on the BLAS threads "
                      f"counted in cores), rate scaled by that group's share of the work"}
        out["parity"] = parity
    return out


def attention_layers_bench(tg, torch, dev, steps, warmup, cpu_s, layers=32):
    """`layers` independent Llama-3-8B-shaped verify layers (each its own Q,
    K/V cache and output: 310 MB at 32) back to back; one step = all of them."""
    import workloads as W
    name = "attn-llama8b"
    Bq, Hq, Hkv, Dh, Lp, Nn, _, _, _, desc = ATTN_SHAPES[name]
    par = attn_parents(name, W.rng(2000))
    bufs = attn_inputs(torch, dev, name, layers, seed=2100)
    parent = torch.from_numpy(par).to(dev)
    plen = torch.full((Bq,), Lp, dtype=torch.int32, device=dev)
    nws = tg.verify_attention_workspace(Bq, Nn, Hq, Hkv, Dh, Lp + Nn, tg.BF16)
    ws = torch.empty(max(nws, 1), dtype=torch.uint8, device=dev)

    def step(i):
        for q, k, v, o in bufs:
            tg.verify_attention(q, k, v, parent, plen, Dh ** -0.5, out=o, workspace=ws)

    # the step as one HIP graph of its 32 calls, replayed (the eager loop is
    # bound by the calls' Python marshalling); a replay must give the eager
    # outputs
    ms_eager = time_calls(torch, step, steps, warmup)
    want = [b[3].clone() for b in bufs]
    ms, graph = time_graph(torch, lambda i: tg.verify_attention(
        bufs[i][0], bufs[i][1], bufs[i][2], parent, plen, Dh ** -0.5, out=bufs[i][3],
        workspace=ws), layers, steps, warmup)
    if not all(torch.equal(b[3], w) for b, w in zip(bufs, want)):
        raise RuntimeError("graph replay of the 32 verify calls differs from the eager calls")
    del graph
    kern, _ = kernel_times(tg, torch, step, max(2, steps // 4))
    nb1, fl1 = attn_work(name, par)
    nbytes, flops = layers * nb1, layers * fl1
    ach = nbytes / (ms * 1e-3)
    roof = {"bound": "hbm", "kernel": "attn_mfma + attn_combine (all launches of the step)",
            "achieved": ach / 1e9, "peak": PEAK_HBM / 1e9, "unit": "GB/s",
            "frac": ach / PEAK_HBM, "traffic": None, "avg_launch_us": None,
            "launch_time_from": "timed pass (whole step)"}
    out = line(nbytes / (ms * 1e-3) / 1e12, "TB/s", steps, warmup, ms,
               {"workload": f"{layers} independent {desc}s back to back (B{Bq}, {Hq}/{Hkv} "
                            f"heads, D{Dh}, prefix {Lp}, {Nn} tree nodes, bf16)",
                "layers": layers}, roof, "bf16",
               **{"TFLOP/s": flops / (ms * 1e-3) / 1e12, "bytes": nbytes, "flops": flops,
                  "kernels": kernels_json(kern, max(2, steps // 4)),
                  "timing": f"one HIP graph of the {layers} calls, replayed {steps} times",
                  "eager_ms_per_step": ms_eager})
    if cpu_s > 0:
        f_cpu, b_cpu, t_cpu, done, parity = attn_cpu_baseline(name, par, bufs[0], cpu_s)
        out["cpu_baseline"] = {"value": b_cpu / t_cpu / 1e12, "unit": "TB/s",
                               "cores": blas_threads(), "kind": "oracle",
                               "sample": f"{done} (batch, KV head) groups of layer 0 in "
                                         f"{t_cpu:.1f} s"}
        out["parity"] = parity
    return out


# --------------------------------------------------------- tiny workload

def tiny_bench(tg, torch, dev, steps, warmup, cpu_s):
    """The tiny fp32 workload as one step: attention, one expansion from the 8
    best nodes of a 16-node tree (V=1000, K=4, N=8) and acceptance (target
    tokens match a random child with p = 0.5).  Launch-latency bound: the
    line reports microseconds per step."""
    import workloads as W
    cfg = W.CONFIGS["tiny"]
    g = W.rng(cfg["seed"])
    Nn, Lp, Dh, Vv = cfg["N"], cfg["L"], cfg["D"], cfg["vocab"]
    parent = W.uniform_parents(g, Nn)[None]
    q = torch.from_numpy(W.normal(g, (1, Nn, 4, Dh))).to(dev)
    k = torch.from_numpy(W.normal(g, (1, 4, Lp + Nn, Dh))).to(dev)
    v = torch.from_numpy(W.normal(g, (1, 4, Lp + Nn, Dh))).to(dev)
    tok = W.distinct_sibling_tokens(g, parent[0], Vv)
    greedy = W.greedy_match_random_child(g, parent[0], tok, Vv, 0.5)
    logits = torch.from_numpy(W.normal(g, (1, 8, Vv), cfg["logit_std"])).to(dev)
    dpar = torch.from_numpy(parent).to(dev)
    plen = torch.tensor([Lp], dtype=torch.int32, device=dev)
    out = torch.empty_like(q)
    # the expansion's tree: the 16 nodes, each with a synthetic path score
    # (-depth - id / 100; it only orders the frontier and offsets the
    # children's scores) in a tree of capacity 64
    depth = W.node_depths(parent[0])
    cum = -depth.astype(np.float32) - np.float32(0.01) * np.arange(Nn, dtype=np.float32)

    def pad(a, fill, dtype):
        o = np.full((1, 64), fill, dtype)
        o[0, :Nn] = a
        return o
    base = tg.TreeState.from_host(dict(parent=pad(parent[0], -1, np.int32),
                                       token=pad(tok, 0, np.int32),
                                       depth=pad(depth, 0, np.int32),
                                       logp=pad(-1.0, 0.0, np.float32),
                                       cum=pad(cum, 0.0, np.float32),
                                       visited=np.zeros((1, 64), np.uint8),
                                       root_visited=np.zeros(1, np.uint8),
                                       n_nodes=np.array([Nn], np.int32)), 64, dev)
    order = sorted(range(Nn), key=lambda i: (-float(cum[i]), int(depth[i]), i))
    fr = torch.tensor([order[:8]], dtype=torch.int32, device=dev)
    n_trees = warmup + 2 * steps + 1
    trees = [tg.TreeState(1, 64, dev) for _ in range(n_trees)]
    for t in trees:
        for f in tg.TreeState.FIELDS:
            getattr(t, f).copy_(getattr(base, f))
    ws = torch.empty(tg.expand_topk_workspace(1, 8, Vv, 4, 8), dtype=torch.uint8, device=dev)
    lse = torch.empty((1, 8), dtype=torch.float32, device=dev)
    nx = torch.empty((1, 8), dtype=torch.int32, device=dev)
    nn = torch.empty((1,), dtype=torch.int32, device=dev)
    dtok = torch.from_numpy(tok[None]).to(dev)
    dgreedy = torch.from_numpy(greedy[None]).to(dev)
    nnodes = torch.tensor([Nn], dtype=torch.int32, device=dev)
    A = torch.empty((1,), dtype=torch.int32, device=dev)
    path = torch.empty((1, Nn), dtype=torch.int32, device=dev)
    bonus = torch.empty((1,), dtype=torch.int32, device=dev)

    def step_on(t):
        tg.verify_attention(q, k, v, dpar, plen, Dh ** -0.5, out=out)
        tg.expand_topk(t, logits, fr, None, 4, 8, row_lse=lse, next_frontier=nx,
                       n_next=nn, workspace=ws)
        tg.accept(dpar, dtok, nnodes, dgreedy, Nn, accept_len=A, accept_path=path, bonus=bonus)

    def step(i):
        step_on(trees[i])

    ms_eager = time_calls(torch, step, steps, warmup)
    # the three calls' Python marshalling (~20 us each) outlasts their
    # kernels, so the eager loop measures the host: the step is timed as one
    # graph of 8 steps on trees of their own, replayed; each captured step
    # first puts its tree back to the 16 nodes (a 4-byte device copy), so every
    # replay expands the same tree, and the replay must give the eager result
    n_g = 8
    gtrees = [tg.TreeState(1, 64, dev) for _ in range(n_g)]
    for t in gtrees:
        for f in tg.TreeState.FIELDS:
            getattr(t, f).copy_(getattr(base, f))

    def step_g(i):
        gtrees[i].n_nodes.copy_(base.n_nodes)
        step_on(gtrees[i])
    step_g(0)
    torch.cuda.synchronize()
    want = (out.clone(), nx.clone(), gtrees[0].cum.clone(), A.clone())
    ms_rep, graph = time_graph(torch, step_g, n_g, max(1, steps), warmup)
    ms = ms_rep / n_g
    got = (out, nx, gtrees[0].cum, A)
    if not all(torch.equal(a, b) for a, b in zip(got, want)):
        raise RuntimeError("graph replay of the tiny step differs from the eager step")
    del graph
    kern, _ = kernel_times(tg, torch, step, steps, start=warmup + steps)
    nbytes, flops = attn_work("tiny", parent)
    a_us = 1e3 * kern["attn_f32"][1] / kern["attn_f32"][0]
    roof = {"bound": "hbm", "kernel": "attn_f32", "achieved": nbytes / (a_us * 1e-6) / 1e9,
            "peak": PEAK_HBM / 1e9, "unit": "GB/s",
            "frac": nbytes / (a_us * 1e-6) / PEAK_HBM, "traffic": None, "avg_launch_us": a_us,
            "launch_time_from": "trace pass (event pair around each kernel)",
            "note": "launch-latency bound: 0.33 MB per call"}
    res = line(1e3 * ms, "us", steps, warmup, ms,
               {"workload": "tiny fp32 workload: attention (B1, 4/4 heads, D64, prefix 128, "
                            "16 nodes) + expansion (V=1000, F=8, K=4, N=8) + acceptance"},
               roof, "f32", higher=False, kernels=kernels_json(kern, steps),
               timing=f"one HIP graph of {n_g} steps, replayed {max(1, steps)} times",
               eager_ms_per_step=ms_eager)
    if cpu_s > 0:
        from oracle import attention as OA
        from oracle import tree as OT
        th = base.to_host()
        tree_h = OT.Tree(th["parent"], th["token"], th["depth"], th["logp"], th["cum"],
                         th["visited"], th["root_visited"], th["n_nodes"], cap=64)
        qh, kh, vh = q.cpu().numpy(), k.cpu().numpy(), v.cpu().numpy()
        lh, frh = logits.cpu().numpy(), fr.cpu().numpy()
        n, t0 = 0, time.perf_counter()
        while True:
            want = OA.tree_verify_attention(qh, kh, vh, parent, [Lp], Dh ** -0.5)
            _, _, nx_o, nn_o, _ = OT.expand(tree_h, lh, frh, None, 4, 8)
            A_o, _, _, _ = OT.accept(parent, tok[None], np.array([Nn]), greedy[None], Nn)
            n += 1
            el = time.perf_counter() - t0
            if el >= cpu_s:
                break
        step(n_trees - 1)
        torch.cuda.synchronize()
        got = out.cpu().numpy().astype(np.float64)
        rowerr = np.abs(got - want).max(axis=-1) / np.abs(want).max(axis=-1)
        res["cpu_baseline"] = {"value": 1e6 * el / n, "unit": "us", "cores": 1, "kind": "oracle",
                               "sample": f"{n} full steps in {el:.1f} s (single-threaded NumPy)"}
        res["parity"] = {"attention_max_row_rel_err": float(rowerr.max()), "bar": 1e-5,
                         "next_frontier_equal": bool(np.array_equal(nx.cpu().numpy(), nx_o)),
                         "accept_len_equal": bool(int(A.item()) == int(A_o[0]))}
    return res


# ------------------------------------------- two-drafter tree workloads

TD_B, TD_V, TD_K, TD_N, TD_W, TD_M, TD_F, TD_R = 8, 128256, 10, 60, 60, 10, 64, 257


def twodrafter_trees(tg, torch, dev):
    """The two-drafter workload's trees, built on the GPU by the library: per
    tree a 5-step weak expansion from the root (frontier 10, top-10: 410
    nodes) pruned by Alg. 3 to 256 nodes, re-indexed, with its logits rows
    re-indexed alike (row 0 = root, row 1 + i = kept node i); weak rows
    N(0,3), strong = 0.8 * weak + 0.6 * N(0,3) (correlation 0.8).  Returns
    (template TreeState, weak rows, strong rows, frontier of the 64 best
    leaves)."""
    gen = torch.Generator(device=dev)
    gen.manual_seed(3000)
    big_rows = torch.empty((TD_B, 411, TD_V), dtype=torch.float32, device=dev)
    big_rows.normal_(0.0, 3.0, generator=gen)       # row 0 root, row 1 + id
    ts = tg.TreeState(TD_B, 512, dev)
    fr = torch.full((TD_B, 1), -1, dtype=torch.int32, device=dev)
    nf = torch.ones(TD_B, dtype=torch.int32, device=dev)
    bidx = torch.arange(TD_B, device=dev)[:, None]
    for _ in range(5):
        lg = big_rows[bidx, (fr + 1).long()].contiguous()
        _, fr, nf = tg.expand_topk(ts, lg, fr.contiguous(), nf, 10, 10)
    torch.cuda.synchronize()
    assert int(ts.n_nodes.min().item()) == 410 == int(ts.n_nodes.max().item())
    pr = tg.global_prune(ts, 256)
    torch.cuda.synchronize()
    assert int(pr["n_keep"].min().item()) == 256
    kept = pr["kept"].long()
    tmpl = tg.TreeState(TD_B, 2048, dev)
    tmpl.parent[:, :256] = pr["vparent"]
    tmpl.token[:, :256] = pr["vtoken"]
    tmpl.depth[:, :256] = torch.gather(ts.depth, 1, pr["kept"].long())
    tmpl.logp[:, :256] = torch.gather(ts.logp, 1, kept)
    tmpl.cum[:, :256] = torch.gather(ts.cum, 1, kept)
    tmpl.n_nodes.fill_(256)
    rows = torch.cat([torch.zeros((TD_B, 1), dtype=torch.long, device=dev), kept + 1], dim=1)
    weak = big_rows[bidx, rows].contiguous()
    del big_rows
    noise = torch.empty_like(weak)
    noise.normal_(0.0, 3.0, generator=gen)
    strong = (0.8 * weak + 0.6 * noise).contiguous()
    del noise
    # the expansion's frontier: the 64 best leaves by (cum desc, depth asc, id asc)
    par_h, cum_h, dep_h = (tmpl.parent[:, :256].cpu().numpy(), tmpl.cum[:, :256].cpu().numpy(),
                           tmpl.depth[:, :256].cpu().numpy())
    front = np.empty((TD_B, TD_F), np.int32)
    for b in range(TD_B):
        has_kid = set(int(p) for p in par_h[b])
        leaves = [u for u in range(256) if u not in has_kid]
        leaves.sort(key=lambda u: (-float(cum_h[b, u]), int(dep_h[b, u]), u))
        front[b] = leaves[:TD_F]
    return tmpl, weak, strong, torch.from_numpy(front).to(dev)


def tree_bench(tg, torch, dev, name, steps, warmup, cpu_s, flags=0, shared=None):
    """tg_tree_expand_topk (the 64 best leaves of each tree, K=10, N=60) or
    tg_tree_rescore_graft (W=60, m=10) on the two-drafter trees; every timed
    call gets a fresh copy of the tree (the calls append to it)."""
    tmpl, weak, strong, front = shared if shared is not None else twodrafter_trees(tg, torch, dev)
    rescore = name == "rescore-twodrafter"
    bidx = torch.arange(TD_B, device=dev)[:, None]
    if rescore:
        copies = 1                                           # 1.05 GB > the MALL
        logits = [strong]
    else:
        exp_rows = weak[bidx, (front + 1).long()].contiguous()  # [B, 64, V], 263 MB
        copies = 3
        logits = [exp_rows] + [exp_rows.clone() for _ in range(copies - 1)]
    n_trees = warmup + 2 * steps + 1
    trees = [tg.TreeState(TD_B, 2048, dev) for _ in range(n_trees)]
    for ts in trees:
        for f in tg.TreeState.FIELDS:
            getattr(ts, f).copy_(getattr(tmpl, f))
    i32 = dict(dtype=torch.int32, device=dev)
    if rescore:
        ws = torch.empty(tg.rescore_graft_workspace(TD_B, TD_R, TD_V, TD_W, TD_M, 2048),
                         dtype=torch.uint8, device=dev)
        lse = torch.empty((TD_B, TD_R), dtype=torch.float32, device=dev)
        gf, ng = torch.empty((TD_B, TD_W), **i32), torch.empty((TD_B,), **i32)
        new_from = torch.full((TD_B,), 16, **i32) if flags & 1 else None

        def call(i):
            tg.rescore_graft(trees[i], logits[i % copies], TD_W, TD_M, row_lse=lse,
                             graft_frontier=gf, n_graft=ng, workspace=ws, flags=flags,
                             new_from=new_from)
        # rows read: every pool node's row and its parent's (the paper's pool:
        # the 257 rows; w/o EG: the pool ids >= 16 and their parents)
        if flags & 1:
            par_h = tmpl.parent[:, :256].cpu().numpy()
            rows_read = sum(len({u + 1 for u in range(16, 256)} |
                                {int(par_h[b, u]) + 1 for u in range(16, 256)})
                            for b in range(TD_B))
            pool = TD_B * 240
        else:
            rows_read, pool = TD_B * TD_R, TD_B * 257
        nbytes = rows_read * TD_V * 4
        nodes = pool + TD_B * TD_W * TD_M
    else:
        ws = torch.empty(tg.expand_topk_workspace(TD_B, TD_F, TD_V, TD_K, TD_N),
                         dtype=torch.uint8, device=dev)
        lse = torch.empty((TD_B, TD_F), dtype=torch.float32, device=dev)
        nx, nn = torch.empty((TD_B, TD_N), **i32), torch.empty((TD_B,), **i32)

        def call(i):
            tg.expand_topk(trees[i], logits[i % copies], front, None, TD_K, TD_N, row_lse=lse,
                           next_frontier=nx, n_next=nn, workspace=ws)
        nbytes = TD_B * TD_F * TD_V * 4
        nodes = TD_B * TD_F * TD_K
    ms = time_calls(torch, call, steps, warmup)
    kern, _ = kernel_times(tg, torch, call, steps, start=warmup + steps)
    row_us = 1e3 * kern["row_partial"][1] / kern["row_partial"][0]
    ach = nbytes / (row_us * 1e-6)
    roof = {"bound": "hbm", "kernel": "row_partial", "achieved": ach / 1e9,
            "peak": PEAK_HBM / 1e9, "unit": "GB/s", "frac": ach / PEAK_HBM,
            "traffic": traffic_for(name, "row_partial") if flags == 0 else None,
            "avg_launch_us": row_us,
            "launch_time_from": "trace pass (event pair around each kernel)"}
    out = line(nodes / (ms * 1e-3), "nodes/s", steps, warmup, ms,
               {"workload": "two-drafter " + ("rescore + graft (257 strong rows per tree, W=60, "
                                              "m=10)" if rescore else
                                              "expansion (64 leaves per tree, K=10, N=60)") +
                            ", B8 trees of 256 nodes (5-step weak expansion pruned by Alg. 3), "
                            "V=128256, fp32 logits",
                "batch": TD_B, "vocab": TD_V, "rescore_flags": flags if rescore else None,
                "input_copies": copies},
               roof, "f32", **{"call_TB/s": nbytes / (ms * 1e-3) / 1e12, "bytes": nbytes,
                               "nodes_per_call": nodes, "kernels": kernels_json(kern, steps)})
    if cpu_s > 0:
        # one more call on a fresh tree copy, input copy 0, kept for the check
        last = n_trees - 1
        call_out = trees[last]
        th = call_out.to_host()                      # the tree before the call
        call(last)
        torch.cuda.synchronize()
        got_tree = call_out.to_host()
        got = (gf.cpu().numpy(), ng.cpu().numpy()) if rescore else (nx.cpu().numpy(),
                                                                   nn.cpu().numpy())
        lse_g = lse.cpu().numpy()
        out["cpu_baseline"], out["parity"] = tree_cpu_baseline(
            rescore, th, logits[0], front.cpu().numpy(), got, got_tree, lse_g, cpu_s, nbytes)
    return out


def tree_cpu_baseline(rescore, th, logits_dev, front, got, got_tree, lse_g, budget_s, nbytes):
    """The oracle on whole trees of the same call (input copy 0) until about
    `budget_s` seconds are spent.  Parity on those trees: the oracle re-run
    with the GPU's row log-sum-exps gives every integer output and score bit
    for bit (the split check), the free oracle's selection is compared where
    its boundary gap exceeds twice the score discrepancy, and the gap, the
    discrepancy and the largest lse difference are reported."""
    from oracle import tree as OT
    done, t_cpu = 0, 0.0
    exact, free_ok, checked_free = True, True, 0
    min_gap, max_disc, max_dlse = float("inf"), 0.0, 0.0
    for b in range(TD_B):
        t1 = OT.Tree(*(th[f][b:b + 1] for f in ("parent", "token", "depth", "logp", "cum",
                                                 "visited", "root_visited", "n_nodes")),
                     cap=th["parent"].shape[1])
        lg = logits_dev[b:b + 1].cpu().numpy()
        t0 = time.perf_counter()
        if rescore:
            free, lse_f, sel_f, nsel_f, _ = OT.rescore_graft(t1, lg, TD_W, TD_M)
        else:
            free, lse_f, sel_f, nsel_f, _ = OT.expand(t1, lg, front[b:b + 1], None, TD_K, TD_N)
        t_cpu += time.perf_counter() - t0
        lse_b = np.nan_to_num(lse_g[b:b + 1], nan=0.0)
        if rescore:
            want, _, sel_o, nsel_o, _ = OT.rescore_graft(t1, lg, TD_W, TD_M, lse_override=lse_b)
        else:
            want, _, sel_o, nsel_o, _ = OT.expand(t1, lg, front[b:b + 1], None, TD_K, TD_N,
                                                 lse_override=lse_b)
        n = int(want.n_nodes[0])
        exact = exact and np.array_equal(got[0][b], sel_o[0]) and int(got[1][b]) == int(nsel_o[0])
        for f in ("parent", "token", "depth"):
            exact = exact and np.array_equal(got_tree[f][b, :n], getattr(want, f)[0, :n])
        for f in ("logp", "cum"):
            exact = exact and np.array_equal(got_tree[f][b, :n].view(np.uint32),
                                             getattr(want, f)[0, :n].view(np.uint32))
        live = ~np.isnan(lse_f[0])
        max_dlse = max(max_dlse, float(np.abs(lse_f[0][live].astype(np.float64) -
                                              lse_g[b][live].astype(np.float64)).max()))
        # selection boundary of the free oracle
        n0 = int(t1.n_nodes[0])
        if rescore:
            cand = [(-0.0, 0, -1)] + [OT.node_key(free.cum[0, u], free.depth[0, u], u)
                                      for u in range(n0) if not t1.visited[0, u]]
            disc = float(np.abs(free.cum[0, :n0].astype(np.float64) -
                                got_tree["cum"][b, :n0].astype(np.float64)).max())
        else:
            cand = [OT.node_key(free.cum[0, u], free.depth[0, u], u) for u in range(n0, n)]
            disc = float(np.abs(free.cum[0, n0:n].astype(np.float64) -
                                got_tree["cum"][b, n0:n].astype(np.float64)).max())
        cand.sort()
        k = int(nsel_f[0])
        gap = abs(cand[k][0] - cand[k - 1][0]) if 0 < k < len(cand) else float("inf")
        min_gap, max_disc = min(min_gap, gap), max(max_disc, disc)   # inf: nothing rejected
        if gap > 2 * disc:
            checked_free += 1
            free_ok = free_ok and np.array_equal(sel_f[0], got[0][b])
        done += 1
        if t_cpu >= budget_s:
            break
    cpu = {"value": nbytes * done / TD_B / t_cpu / 1e9, "unit": "GB/s", "cores": blas_threads(),
           "kind": "oracle",
           "sample": f"{done} of {TD_B} trees of the same call in {t_cpu:.1f} s (NumPy; full "
                     f"sorts), logits bytes per second"}
    parity = {"trees_checked": done, "exact_with_gpu_lse": bool(exact),
              "free_oracle_selection_equal": bool(free_ok), "free_checked_trees": checked_free,
              "min_selection_gap": min_gap if np.isfinite(min_gap) else None,
              "max_score_discrepancy": max_disc,
              "max_lse_abs_diff": max_dlse}
    return cpu, parity


# -------------------------------------------------------------- the turn
# (Llama-3-8B-shaped TreeGraft turn)
V, W_FR, M_CH = 128256, 10, 8
SCHEDULE = (1, 0, 1, 0, 1)
B, HQ, HKV, D, L, N_VER = 1, 32, 8, 128, 2048, 64     # N_VER = B_ver pruned nodes
CAP = 512
MAX_DEPTH = 8            # accept path width (the turn's trees are at most 5 deep)
R_ROWS = 313             # strong-logits rows (root + up to 312 nodes)
NG_NMAX = 4              # n-gram drafter: longest n-gram matched


def make_inputs(c, dev):
    """Input copy c (seed 1002 + 100 * c): the workload's tensors on the GPU."""
    import torch
    import workloads as W
    g = W.rng([1002, c])
    strong = torch.empty((B, R_ROWS, V), dtype=torch.float32, device=dev)
    for r0 in range(0, R_ROWS, 32):        # chunks keep host memory small
        r1 = min(R_ROWS, r0 + 32)
        strong[0, r0:r1] = torch.from_numpy(W.normal(g, (r1 - r0, V), 3.0)).to(dev)
    s = np.float32(1.0 / np.sqrt(128.0))
    S = L + N_VER
    q = torch.from_numpy(W.normal(g, (B, N_VER, HQ, D)) * s).to(dev).bfloat16()
    k = torch.from_numpy(W.normal(g, (B, HKV, S, D)) * s).to(dev).bfloat16()
    v = torch.from_numpy(W.normal(g, (B, HKV, S, D)) * s).to(dev).bfloat16()
    # the prompt and the target's prefill logits over it (row i = after x_<=i)
    ctx = W.token_stream(g, L, V, n_phrases=64)[None]
    prefill = torch.empty((B, L, V), dtype=torch.float32, device=dev)
    for r0 in range(0, L, 64):
        prefill[0, r0:r0 + 64] = torch.from_numpy(W.normal(W.rng([1002, c, 9, r0]), (64, V),
                                                           3.0)).to(dev)
    # the scheduler's inputs: predictor weights and each step's runtime
    # context + history encoding (11 values)
    params = torch.from_numpy(W.normal(g, (3265,), 0.1)).to(dev)
    sched_ctx = torch.from_numpy(W.normal(g, (len(SCHEDULE), B, 11), 1.0)).to(dev)
    return dict(strong=strong, q=q, k=k, v=v, ctx=torch.from_numpy(ctx).to(dev),
                prefill=prefill, params=params, sched_ctx=sched_ctx)


def prefill_host(c):
    """Host copy of input copy c's prefill logits (the same seeded draws)."""
    import workloads as W
    out = np.empty((B, L, V), np.float32)
    for r0 in range(0, L, 64):
        out[0, r0:r0 + 64] = W.normal(W.rng([1002, c, 9, r0]), (64, V), 3.0)
    return out


def greedy_for(tree_host):
    """Synthetic target for the pruned tree of one input copy: at each node
    (and at the prefix end) the target's greedy token is the first child's
    token with p = 0.7 per level, else another token."""
    import workloads as W
    par, tok = tree_host
    g = W.rng([1002, 7, len(par)])
    return W.greedy_match_first_child(g, par, tok, V, 0.7)


class Step:
    """All buffers of one step on one input copy, so it can be captured."""

    def __init__(self, tg, inp, dev):
        import torch
        self.tg, self.inp = tg, inp
        i32 = dict(dtype=torch.int32, device=dev)
        self.tree = tg.TreeState(B, CAP, dev)
        self.ws_r = torch.empty(tg.rescore_graft_workspace(B, R_ROWS, V, W_FR, M_CH, CAP),
                                dtype=torch.uint8, device=dev)
        # n-gram drafter: the prefill cache (built once, untimed)
        self.clen = torch.full((B,), L, **i32)
        ws_c = torch.empty(tg.ngram_cache_workspace(B, L, V, M_CH), dtype=torch.uint8,
                           device=dev)
        self.c_tok, self.c_lp, self.c_fb = tg.ngram_cache(inp["prefill"], inp["ctx"], self.clen,
                                                          M_CH, workspace=ws_c)
        torch.cuda.synchronize()
        del ws_c
        self.mpos = [torch.empty((B, W_FR), **i32) for _ in range(2)]
        self.root_fr = torch.full((B, 1), -1, **i32)
        self.sig = [torch.empty((B, 10), dtype=torch.float32, device=dev)
                    for _ in SCHEDULE]
        self.margin = [torch.empty((B,), dtype=torch.float32, device=dev) for _ in SCHEDULE]
        self.action = [torch.empty((B,), **i32) for _ in SCHEDULE]
        nv = tg.verify_attention_workspace(B, N_VER, HQ, HKV, D, L + N_VER, tg.BF16)
        self.ws_v = torch.empty(max(nv, 1), dtype=torch.uint8, device=dev)
        self.r_lse = [torch.empty((B, R_ROWS), dtype=torch.float32, device=dev) for _ in range(3)]
        self.gf = [torch.empty((B, W_FR), **i32) for _ in range(3)]
        self.ng = [torch.empty((B,), **i32) for _ in range(3)]
        self.fr = [torch.empty((B, W_FR), **i32) for _ in range(5)]
        self.nn = [torch.empty((B,), **i32) for _ in range(5)]
        M = N_VER + 1
        self.pr = dict(kept=torch.empty((B, N_VER), **i32), vparent=torch.empty((B, N_VER), **i32),
                       vtoken=torch.empty((B, N_VER), **i32),
                       position_ids=torch.empty((B, M), **i32),
                       mask=torch.empty((B, M, (M + 31) // 32), **i32),
                       retrieval=torch.empty((B, M, MAX_DEPTH + 1), **i32),
                       n_keep=torch.empty((B,), **i32), n_leaves=torch.empty((B,), **i32))
        self.plen = torch.full((B,), L, **i32)
        self.new_plen = torch.empty((B,), **i32)
        self.greedy = torch.zeros((B, N_VER + 1), **i32)
        self.out = torch.empty_like(inp["q"])
        self.A = torch.empty((B,), **i32)
        self.path = torch.empty((B, MAX_DEPTH), **i32)
        self.bonus = torch.empty((B,), **i32)

    def run(self):
        tg, x, t = self.tg, self.inp, self.tree
        tg.tree_reset(t)
        mid, small = 0, 0
        for k, a in enumerate(SCHEDULE):
            # the scheduler's pre-action state (its action is not used)
            fr_k, nf_k = (self.root_fr, None) if k == 0 else (self.fr[k - 1], self.nn[k - 1])
            tg.tree_signals(t, fr_k, nf_k, W_FR, 5, context=x["sched_ctx"][k],
                            params=x["params"], signals=self.sig[k], margin=self.margin[k],
                            action=self.action[k])
            if a == 1:       # middle-drafter step
                tg.rescore_graft(t, x["strong"], W_FR, M_CH, row_lse=self.r_lse[mid],
                                 graft_frontier=self.gf[mid], n_graft=self.ng[mid], N=W_FR,
                                 next_frontier=self.fr[k], n_next=self.nn[k],
                                 workspace=self.ws_r)
                mid += 1
            else:            # small (n-gram) step over the previous step's new nodes
                tg.expand_ngram(t, self.fr[k - 1], self.nn[k - 1], x["ctx"], self.clen,
                                self.c_tok, self.c_lp, self.c_fb, M_CH, W_FR, NG_NMAX,
                                match_pos=self.mpos[small], next_frontier=self.fr[k],
                                n_next=self.nn[k])
                small += 1
        p = tg.global_prune(t, N_VER, MAX_DEPTH + 1, out=self.pr)
        tg.verify_attention(x["q"], x["k"], x["v"], p["vparent"], self.plen, D ** -0.5,
                            out=self.out, workspace=self.ws_v)
        tg.accept(p["vparent"], p["vtoken"], p["n_keep"], self.greedy, MAX_DEPTH,
                  accept_len=self.A, accept_path=self.path, bonus=self.bonus)
        tg.kv_compact(x["k"], x["v"], self.plen, self.path, self.A,
                      new_prefix_len=self.new_plen)


def rows_read_per_step():
    """Middle-drafter logits rows one turn reads (structural: independent of
    the values).  k=1 pool {root}: row 0.  k=3 pool = 72 unvisited nodes:
    their 72 rows + the root row (parent of 8 of them).  k=5 pool = 160
    nodes: their rows + the rows of the 10 graft points of k=3 (parents of 80
    of them, already visited)."""
    return [1, 73, 170]


def ngram_bytes_per_step():
    """Bytes the two n-gram steps read: the prompt once per step (4 B a
    token) and the matched cache rows of their 8 and 10 frontier nodes (8
    candidates of 8 B: token + log-probability)."""
    return sum(L * 4 + f * M_CH * 8 for f in (8, 10))


def verify_work(vpar):
    """Algorithmic bytes and flops of the turn's verify call."""
    kv = 2 * B * HKV * (L + N_VER) * D * 2
    qo = 2 * B * N_VER * HQ * D * 2
    keys = N_VER * L + path_len_sum(vpar)
    flops = 4 * D * HQ * B * keys
    return kv + qo + vpar.nbytes, flops


def turn_cpu_baseline(inp, greedy0, budget_s):
    """The oracle (the tests' CPU reference, untuned) running the same turn on
    input copy 0 until about `budget_s` seconds have been spent."""
    from oracle import attention as OA
    from oracle import ngram as NG
    from oracle import signals as OS
    from oracle import tree as OT
    strong = inp["strong"].cpu().numpy()
    ctx = inp["ctx"].cpu().numpy()
    clen = np.array([L], np.int32)
    # the prefill cache (set-up, untimed, as on the GPU side)
    c_tok, c_lp, c_fb, _ = NG.ngram_cache(prefill_host(0), ctx, clen, M_CH)
    params = inp["params"].cpu().numpy()
    sched_ctx = inp["sched_ctx"].cpu().numpy()
    q = inp["q"].float().cpu().numpy()
    k = inp["k"].float().cpu().numpy()
    v = inp["v"].float().cpu().numpy()
    turns, t0 = 0, time.perf_counter()
    while True:
        t = OT.Tree.empty(B, CAP)
        fr = nn = None
        for step, a in enumerate(SCHEDULE):
            F_k = [-1] if step == 0 else [int(x) for x in fr[0, :int(nn[0])]]
            n = int(t.n_nodes[0])
            sig, _ = OS.tree_signals(t.parent[0], t.depth[0], t.cum[0], n, F_k, W_FR, 5)
            OS.margin(sched_ctx[step, 0], sig, params)
            if a == 1:
                t, _, _, _, _, fr, nn = OT.rescore_graft(t, strong, W_FR, M_CH, N=W_FR)
            else:
                t, _, fr, nn, _ = NG.expand_ngram(t, fr, nn, ctx, clen, c_tok, c_lp, c_fb, M_CH,
                                                  W_FR, NG_NMAX)
        n = int(t.n_nodes[0])
        pr = OT.global_prune(t.parent[0, :n], t.cum[0, :n], n, N_VER)
        par = pr["parent"][None]
        tok = t.token[0, pr["kept"]][None]
        OA.tree_verify_attention_fast(q, k, v, par, [L], D ** -0.5)
        A, path, _, _ = OT.accept(par, tok, np.array([len(pr["kept"])]), greedy0, MAX_DEPTH)
        OA.kv_compact(k, v, np.array([L]), path, A)
        turns += 1
        el = time.perf_counter() - t0
        if el >= budget_s:
            return turns, el


def turn_bench(tg, torch, dev, steps, warmup, copies, cpu_s):
    """One TreeGraft turn per step, replayed as one captured HIP graph per
    input copy (inputs rotate over `copies` resident copies, > the MALL)."""
    inputs = [make_inputs(c, dev) for c in range(copies)]
    steps_ = [Step(tg, inputs[c], dev) for c in range(copies)]
    torch.cuda.synchronize()
    # set-up (untimed): every copy's turn once; the structural guard, and the
    # synthetic target's greedy tokens for the pruned tree each copy builds
    pruned = []
    n_nodes = 8 + 64 + 80 + 80 + 80
    for st in steps_:
        st.run()
        torch.cuda.synchronize()
        assert int(st.tree.n_nodes[0].item()) == n_nodes
        assert int(st.pr["n_keep"][0].item()) == N_VER
        par = st.pr["vparent"][0].cpu().numpy()
        tok = st.pr["vtoken"][0].cpu().numpy()
        st.greedy.copy_(torch.from_numpy(greedy_for((par, tok))[None]))
        pruned.append((par, tok))
    torch.cuda.synchronize()
    graphs, timing = [], "eager launches"
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        for st in steps_:
            st.run()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    try:
        for st in steps_:
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                st.run()
            graphs.append(g)
        torch.cuda.synchronize()
        timing = "one captured HIP graph per step"
    except Exception as exc:  # report and time eager launches instead
        print(f"bench.py: graph capture failed ({exc}); timing eager launches", file=sys.stderr)
        graphs = []
    if graphs:        # replaying a graph must reproduce the eager turn
        graphs[0].replay()
        torch.cuda.synchronize()
        assert int(steps_[0].tree.n_nodes[0].item()) == n_nodes

    def run(i):
        if graphs:
            graphs[i % len(graphs)].replay()
        else:
            steps_[i % len(steps_)].run()

    ms_step = time_calls(torch, run, steps, warmup)
    eager = lambda i: steps_[i % len(steps_)].run()
    ms_eager = time_calls(torch, eager, steps, warmup)
    kern, recs = kernel_times(tg, torch, eager, steps)
    kernels = kernels_json(kern, steps)
    per_step = len(recs) // steps
    timeline = [[name, round(1e3 * ms, 2)] for name, ms in recs[-per_step:]]
    rows_r = rows_read_per_step()
    row_bytes = V * 4
    works = [verify_work(par) for par, _ in pruned]
    v_bytes = sum(w[0] for w in works) / len(works)
    v_flops = sum(w[1] for w in works) / len(works)
    step_bytes = sum(rows_r) * row_bytes + ngram_bytes_per_step() + v_bytes
    rescored = 72 + 160                       # non-root pool nodes rescored
    slowest = max(kernels, key=lambda k: kernels[k]["us_per_step"])
    dom = "row_partial"
    dom_bytes = sum(rows_r) * row_bytes
    launches = kern[dom][0]
    achieved = dom_bytes * steps / (kern[dom][1] * 1e-3)
    roof = {"bound": "hbm", "kernel": dom, "achieved": achieved / 1e9, "peak": PEAK_HBM / 1e9,
            "unit": "GB/s", "frac": achieved / PEAK_HBM,
            "traffic": traffic_for("turn", dom),
            "bytes_per_launch": dom_bytes * steps / launches,
            "avg_launch_us": 1e3 * kern[dom][1] / launches,
            "launch_time_from": "trace pass (event pair around each kernel)"}
    attn_us = sum(kernels[k]["us_per_step"] for k in ATTN_MAIN + ("attn_combine",) if k in kernels)
    out = line(step_bytes / (ms_step * 1e-3) / 1e12, "TB/s", steps, warmup, ms_step,
               {"workload": "TreeGraft turn (schedule 1,0,1,0,1) + Llama-3-8B-shaped verify "
                            "layer", "batch": B, "vocab": V, "frontier_W": W_FR,
                "children_m": M_CH, "q_heads": HQ, "kv_heads": HKV, "head_dim": D, "prefix": L,
                "verify_nodes": N_VER, "input_copies": copies,
                "small_drafter": f"n-gram (cache m = {M_CH}, n_max = {NG_NMAX})",
                "scheduler": "signals + margin predictor every step, fixed schedule",
                "timing": timing},
               roof, "fp32+bf16",
               **{"largest_kernel": {"name": slowest,
                                     "us_per_step": kernels[slowest]["us_per_step"]},
                  "draft_nodes_per_s": (n_nodes + rescored) / (ms_step * 1e-3),
                  "verify_attention": {"us": attn_us, "TB/s": v_bytes / (attn_us * 1e-6) / 1e12,
                                       "TFLOP/s": v_flops / (attn_us * 1e-6) / 1e12,
                                       "frac_hbm": v_bytes / (attn_us * 1e-6) / PEAK_HBM},
                  "step_bytes": step_bytes, "eager_ms_per_step": ms_eager,
                  "kernels": kernels, "step_timeline_us": timeline})
    if cpu_s > 0:
        turns, el = turn_cpu_baseline(inputs[0], steps_[0].greedy.cpu().numpy(), cpu_s)
        out["cpu_baseline"] = {"value": step_bytes * turns / el / 1e12, "unit": "TB/s",
                               "cores": blas_threads(), "kind": "oracle",
                               "sample": f"{turns} full turns of the same workload on input "
                                         f"copy 0 in {el:.1f} s (tree steps single-threaded "
                                         f"NumPy; attention matmuls on the BLAS threads; the "
                                         f"n-gram prefill cache built untimed first)"}
    return out


# ------------------------------------------ the standard (Alg. 1) turn
# The Llama-3-8B-shaped decoding turn with the standard construction: six
# small-drafter expansion steps over dense logits rows (the root, then the
# best-N frontier; K = 8 children per node, N = 10), GlobalPrune of the
# 392-node tree to 64 nodes, one bf16 verify-attention layer, acceptance and
# the KV update.
STD_STEPS, STD_K, STD_N = 6, 8, 10
STD_NODES = 8 + 64 + 4 * 80


def std_inputs(c, dev):
    """Input copy c (seed 1003 + c): one logits tensor per step ([1, 1, V]
    for the root step, [1, N, V] after it; N(0, 3) rows) and the verify
    layer's Q/K/V."""
    import torch
    import workloads as W
    g = W.rng([1003, c])
    logits = []
    for k in range(STD_STEPS):
        F = 1 if k == 0 else STD_N
        t = torch.empty((B, F, V), dtype=torch.float32, device=dev)
        for f in range(F):
            t[0, f] = torch.from_numpy(W.normal(W.rng([1003, c, k, f]), (V,), 3.0)).to(dev)
        logits.append(t)
    s = np.float32(1.0 / np.sqrt(128.0))
    S = L + N_VER
    q = torch.from_numpy(W.normal(g, (B, N_VER, HQ, D)) * s).to(dev).bfloat16()
    k = torch.from_numpy(W.normal(g, (B, HKV, S, D)) * s).to(dev).bfloat16()
    v = torch.from_numpy(W.normal(g, (B, HKV, S, D)) * s).to(dev).bfloat16()
    return dict(logits=logits, q=q, k=k, v=v)


class StdStep:
    """All buffers of one standard turn on one input copy (capturable)."""

    def __init__(self, tg, inp, dev):
        import torch
        self.tg, self.inp = tg, inp
        i32 = dict(dtype=torch.int32, device=dev)
        self.tree = tg.TreeState(B, CAP, dev)
        self.ws_e = torch.empty(max(1, tg.expand_topk_workspace(B, STD_N, V, STD_K, STD_N)),
                                dtype=torch.uint8, device=dev)
        self.root_fr = torch.full((B, 1), -1, **i32)
        self.lse = [torch.empty((B, 1 if k == 0 else STD_N), dtype=torch.float32, device=dev)
                    for k in range(STD_STEPS)]
        self.fr = [torch.empty((B, STD_N), **i32) for _ in range(STD_STEPS)]
        self.nn = [torch.empty((B,), **i32) for _ in range(STD_STEPS)]
        M = N_VER + 1
        self.pr = dict(kept=torch.empty((B, N_VER), **i32), vparent=torch.empty((B, N_VER), **i32),
                       vtoken=torch.empty((B, N_VER), **i32),
                       position_ids=torch.empty((B, M), **i32),
                       mask=torch.empty((B, M, (M + 31) // 32), **i32),
                       retrieval=torch.empty((B, M, MAX_DEPTH + 1), **i32),
                       n_keep=torch.empty((B,), **i32), n_leaves=torch.empty((B,), **i32))
        nv = tg.verify_attention_workspace(B, N_VER, HQ, HKV, D, L + N_VER, tg.BF16)
        self.ws_v = torch.empty(max(nv, 1), dtype=torch.uint8, device=dev)
        self.plen = torch.full((B,), L, **i32)
        self.new_plen = torch.empty((B,), **i32)
        self.greedy = torch.zeros((B, N_VER + 1), **i32)
        self.out = torch.empty_like(inp["q"])
        self.A = torch.empty((B,), **i32)
        self.path = torch.empty((B, MAX_DEPTH), **i32)
        self.bonus = torch.empty((B,), **i32)

    def run(self):
        tg, x, t = self.tg, self.inp, self.tree
        tg.tree_reset(t)
        for k in range(STD_STEPS):
            fr_k, nf_k = (self.root_fr, None) if k == 0 else (self.fr[k - 1], self.nn[k - 1])
            tg.expand_topk(t, x["logits"][k], fr_k, nf_k, STD_K, STD_N, row_lse=self.lse[k],
                           next_frontier=self.fr[k], n_next=self.nn[k], workspace=self.ws_e)
        p = tg.global_prune(t, N_VER, MAX_DEPTH + 1, out=self.pr)
        tg.verify_attention(x["q"], x["k"], x["v"], p["vparent"], self.plen, D ** -0.5,
                            out=self.out, workspace=self.ws_v)
        tg.accept(p["vparent"], p["vtoken"], p["n_keep"], self.greedy, MAX_DEPTH,
                  accept_len=self.A, accept_path=self.path, bonus=self.bonus)
        tg.kv_compact(x["k"], x["v"], self.plen, self.path, self.A,
                      new_prefix_len=self.new_plen)


def std_rows_per_step():
    """Logits rows one standard turn reads: 1 (root), 8, then 10 per step."""
    return 1 + 8 + 10 * (STD_STEPS - 2)


def std_oracle_turn(host_logits, q, k, v, greedy, lse_gpu=None):
    """The oracle's standard turn on host copies (lse_gpu: the GPU's row_lse
    per step, for the split check).  Returns the tree, prune result, the
    attention output and the acceptance."""
    from oracle import attention as OA
    from oracle import tree as OT
    t = OT.Tree.empty(B, CAP)
    fr, nn = np.full((B, 1), -1, np.int32), None
    for step in range(STD_STEPS):
        t, _, fr, nn, _ = OT.expand(t, host_logits[step], fr, nn, STD_K, STD_N,
                                    lse_override=None if lse_gpu is None else lse_gpu[step])
    n = int(t.n_nodes[0])
    pr = OT.global_prune(t.parent[0, :n], t.cum[0, :n], n, N_VER)
    par = pr["parent"][None]
    tok = t.token[0, pr["kept"]][None]
    out = OA.tree_verify_attention_fast(q, k, v, par, [L], D ** -0.5)
    A, path, bonus, _ = OT.accept(par, tok, np.array([len(pr["kept"])]), greedy, MAX_DEPTH)
    return t, pr, par, tok, out, (A, path, bonus)


def std_turn_bench(tg, torch, dev, steps, warmup, copies, cpu_s):
    """One standard turn per step, replayed as one captured HIP graph per
    input copy (inputs rotate over `copies` resident copies)."""
    inputs = [std_inputs(c, dev) for c in range(copies)]
    steps_ = [StdStep(tg, inputs[c], dev) for c in range(copies)]
    torch.cuda.synchronize()
    pruned = []
    for st in steps_:
        st.run()
        torch.cuda.synchronize()
        assert int(st.tree.n_nodes[0].item()) == STD_NODES
        assert int(st.pr["n_keep"][0].item()) == N_VER
        par = st.pr["vparent"][0].cpu().numpy()
        tok = st.pr["vtoken"][0].cpu().numpy()
        st.greedy.copy_(torch.from_numpy(greedy_for((par, tok))[None]))
        pruned.append((par, tok))
    torch.cuda.synchronize()
    # parity on input copy 0 (untimed): the oracle's turn with the GPU's
    # exported log-sum-exps must give the same tree, pruned tree and
    # acceptance bit for bit; attention within the bf16 bar
    st0 = steps_[0]
    # the K/V the attention of this run reads (earlier runs' KV updates
    # included; this run's update comes after its attention)
    qh, kh, vh = (inputs[0][n].float().cpu().numpy() for n in ("q", "k", "v"))
    st0.run()
    torch.cuda.synchronize()
    host_logits = [x.cpu().numpy() for x in inputs[0]["logits"]]
    lse_gpu = [x.cpu().numpy() for x in st0.lse]
    greedy0 = st0.greedy.cpu().numpy()
    t_o, pr_o, par_o, tok_o, out_o, acc_o = std_oracle_turn(host_logits, qh, kh, vh, greedy0,
                                                            lse_gpu)
    n = STD_NODES
    tree_eq = all(np.array_equal(getattr(t_o, f)[0, :n], getattr(st0.tree, f)[0, :n].cpu().numpy())
                  for f in ("parent", "token", "depth")) and \
        np.array_equal(t_o.cum[0, :n].view(np.uint32),
                       st0.tree.cum[0, :n].cpu().numpy().view(np.uint32))
    prune_eq = np.array_equal(par_o[0], st0.pr["vparent"][0].cpu().numpy()) and \
        np.array_equal(tok_o[0], st0.pr["vtoken"][0].cpu().numpy())
    acc_eq = int(acc_o[0][0]) == int(st0.A[0].item()) and \
        np.array_equal(acc_o[1][0], st0.path[0].cpu().numpy()) and \
        int(acc_o[2][0]) == int(st0.bonus[0].item())
    attn_err = float(np.abs(st0.out.float().cpu().numpy() - out_o).max())
    graphs, timing = [], "eager launches"
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        for st in steps_:
            st.run()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    try:
        for st in steps_:
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                st.run()
            graphs.append(g)
        torch.cuda.synchronize()
        timing = "one captured HIP graph per step"
    except Exception as exc:  # report and time eager launches instead
        print(f"bench.py: graph capture failed ({exc}); timing eager launches", file=sys.stderr)
        graphs = []
    if graphs:        # replaying a graph must reproduce the eager turn
        graphs[0].replay()
        torch.cuda.synchronize()
        assert int(steps_[0].tree.n_nodes[0].item()) == STD_NODES

    def run(i):
        if graphs:
            graphs[i % len(graphs)].replay()
        else:
            steps_[i % len(steps_)].run()

    ms_step = time_calls(torch, run, steps, warmup)
    eager = lambda i: steps_[i % len(steps_)].run()
    ms_eager = time_calls(torch, eager, steps, warmup)
    kern, recs = kernel_times(tg, torch, eager, steps)
    kernels = kernels_json(kern, steps)
    per_step = len(recs) // steps
    timeline = [[name, round(1e3 * ms, 2)] for name, ms in recs[-per_step:]]
    row_bytes = V * 4
    works = [verify_work(par) for par, _ in pruned]
    v_bytes = sum(w[0] for w in works) / len(works)
    v_flops = sum(w[1] for w in works) / len(works)
    dom_bytes = std_rows_per_step() * row_bytes
    step_bytes = dom_bytes + v_bytes
    dom = "row_partial"
    launches = kern[dom][0]
    achieved = dom_bytes * steps / (kern[dom][1] * 1e-3)
    roof = {"bound": "hbm", "kernel": dom, "achieved": achieved / 1e9, "peak": PEAK_HBM / 1e9,
            "unit": "GB/s", "frac": achieved / PEAK_HBM, "traffic": None,
            "bytes_per_launch": dom_bytes * steps / launches,
            "avg_launch_us": 1e3 * kern[dom][1] / launches,
            "launch_time_from": "trace pass (event pair around each kernel)",
            "note": "latency bound: 1-10 live rows per launch"}
    slowest = max(kernels, key=lambda k: kernels[k]["us_per_step"])
    attn_us = sum(kernels[k]["us_per_step"] for k in ATTN_MAIN + ("attn_combine",) if k in kernels)
    out = line(step_bytes / (ms_step * 1e-3) / 1e12, "TB/s", steps, warmup, ms_step,
               {"workload": "standard-construction turn (Alg. 1: 6 expansion steps over dense "
                            "logits, K = 8, N = 10) + GlobalPrune to 64 nodes + Llama-3-8B-shaped "
                            "verify layer + acceptance + KV update", "batch": B, "vocab": V,
                "children_K": STD_K, "frontier_N": STD_N, "steps": STD_STEPS,
                "q_heads": HQ, "kv_heads": HKV, "head_dim": D, "prefix": L,
                "verify_nodes": N_VER, "input_copies": copies, "timing": timing},
               roof, "fp32+bf16",
               **{"largest_kernel": {"name": slowest,
                                     "us_per_step": kernels[slowest]["us_per_step"]},
                  "draft_nodes_per_s": STD_NODES / (ms_step * 1e-3),
                  "verify_attention": {"us": attn_us, "TB/s": v_bytes / (attn_us * 1e-6) / 1e12,
                                       "TFLOP/s": v_flops / (attn_us * 1e-6) / 1e12,
                                       "frac_hbm": v_bytes / (attn_us * 1e-6) / PEAK_HBM},
                  "step_bytes": step_bytes, "eager_ms_per_step": ms_eager,
                  "kernels": kernels, "step_timeline_us": timeline,
                  "parity": {"tree_equal_with_gpu_lse": bool(tree_eq),
                             "prune_equal": bool(prune_eq), "accept_equal": bool(acc_eq),
                             "attention_max_abs_err": attn_err, "attention_bar": 2e-2}})
    if cpu_s > 0:
        turns, t0 = 0, time.perf_counter()
        while True:
            std_oracle_turn(host_logits, qh, kh, vh, greedy0)
            turns += 1
            el = time.perf_counter() - t0
            if el >= cpu_s:
                break
        out["cpu_baseline"] = {"value": step_bytes * turns / el / 1e12, "unit": "TB/s",
                               "cores": blas_threads(), "kind": "oracle",
                               "sample": f"{turns} full standard turns on input copy 0 in "
                                         f"{el:.1f} s (tree steps single-threaded NumPy, their "
                                         f"own log-sum-exps; attention matmuls on the BLAS "
                                         f"threads)"}
    return out


# ------------------------------------------------------------------ main

def run_workload(name, args, tg, torch, dev, steps, warmup, cpu_s, shared):
    if name.startswith("attn-llama8b-x32"):
        return attention_layers_bench(tg, torch, dev, steps, warmup, cpu_s)
    if name.startswith("attn-"):
        return attention_bench(tg, torch, dev, name, steps, warmup, cpu_s)
    if name == "tiny":
        return tiny_bench(tg, torch, dev, steps, warmup, cpu_s)
    if name.endswith("-twodrafter"):
        if "td" not in shared:
            shared["td"] = twodrafter_trees(tg, torch, dev)
        return tree_bench(tg, torch, dev, name, steps, warmup, cpu_s,
                          flags=args.rescore_flags if name.startswith("rescore") else 0,
                          shared=shared["td"])
    if name == "turn-standard":
        return std_turn_bench(tg, torch, dev, steps, warmup, args.copies, cpu_s)
    return turn_bench(tg, torch, dev, steps, warmup, args.copies, cpu_s)


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py: runs on one GPU only; sharding the tree-verify path over "
              "(batch, KV head) across GPUs is not implemented", file=sys.stderr)
        sys.exit(2)
    import torch

    import paper_2608_26112_amd as tg
    tg.load()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.copy_calibration_mb:
        n = args.copy_calibration_mb << 18          # float32 elements
        src = torch.ones(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    cpu_main = 0.0 if args.no_cpu_baseline else args.cpu_seconds
    cpu_extra = 0.0 if args.no_cpu_baseline else args.extra_cpu_seconds
    shared = {}
    print(f"bench.py: {args.workload} ...", file=sys.stderr, flush=True)
    out = run_workload(args.workload, args, tg, torch, dev, args.steps, args.warmup, cpu_main,
                       shared)
    if not args.only:
        extra = {}
        for name in WORKLOADS:
            if name == args.workload:
                continue
            print(f"bench.py: {name} ...", file=sys.stderr, flush=True)
            torch.cuda.empty_cache()
            extra[name] = run_workload(name, args, tg, torch, dev, max(5, args.steps),
                                       max(2, args.warmup), cpu_extra, shared)
            shared.pop("td", None) if name == "rescore-twodrafter" else None
        out["extra"] = extra
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
