#!/usr/bin/env python3
"""Benchmark of the UltraEP per-layer balancing path on one MI355X.

One step = one layer-microbatch of the hot path on the measured rank:
  count      (that rank's top-k ids -> its row of the load matrix)
  replicate  (SolveReplication over the whole EP group)
  reroute + pack  (SolveReroute, and the replicated main-expert blobs into
             per-destination staging, in one launch: the overlap of Eq. (1))
  dispatch   layout + row scatter (bf16 rows into per-replica send blocks)
on synthetic DeepSeek-V3-shaped training routing (E=256, top-8 with
8-group / top-4-group restriction, EP=64, one redundant slot per rank,
4096 tokens per rank, H=7168, F=2048).  The other 63 ranks' load rows are
resident inputs (the all-gather that delivers them is not on one GPU).  The
measured rank is the one with the most outbound replica bytes.

Timed region: K steps as HIP graph replays on one stream, bracketed by
device synchronisation; a graph holds 10 consecutive steps (when 10 divides
K), so a step does not pay a whole graph launch alone, as it would not inside
a larger training or serving graph.  one_step_graph_us reports the same
steps launched one graph per step.  (Running the packing on a
second stream instead measured slower on one GPU: the cross-queue
dependencies of the graph cost more than the overlap gains.)  The graph's outputs are checked
against an eager step.  A second pass of K eager steps records a HIP event
between consecutive launches on the launch stream (the stream holds on a
short spin kernel while the host enqueues the pass, so the events bracket
back-to-back kernels, not host gaps); the dominant kernel's average
duration gives the roofline figures, and count + plan is timed as
one pair (count_plan_eager_us).  count_plan_us is the same pair's device
latency: 20 consecutive pairs in one graph, replayed, divided by 20.  The CPU oracle is timed
single-threaded on a bounded sample of the same workload.

Prints one JSON line.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = ("plan+dispatch latency per layer-microbatch (µs); "
          "dispatch/pack HBM GB/s vs peak")
PEAK_HBM_GBPS = 8000.0
WORKLOAD_ID = 4


def hold_stream(ms=40.0):
    """Keeps the current stream busy for about `ms` milliseconds (a spin
    kernel) so that the host can enqueue a timed sequence ahead of the GPU."""
    import torch
    torch.cuda._sleep(int(ms * 1e-3 * 2.4e9))


def outbound_fan(X, n_main, rank):
    """Copies of each of `rank`'s main experts in the replica placement X
    ([R][n_slot] int32, -1 = empty): the fan-out its packing serves."""
    import numpy as np
    X = np.asarray(X)
    return np.bincount(X[(X >= 0) & (X // n_main == rank)] - rank * n_main, minlength=n_main)


def algorithmic_bytes(T, H, k, n_routed, W, fan):
    """Bytes the two HBM-bound launches of a step must move at least:
    the scatter reads every token row once, writes every routed row once and
    reads row_of_slot (int32 per slot); the packing reads each replicated
    blob (W bf16 elements) once and writes it once per copy."""
    scatter = 2 * T * H + 2 * n_routed * H + 4 * T * k
    pack = int(sum(2 * W * (1 + int(f)) for f in fan if f > 0))
    return scatter, pack


def kernel_source_digest(files):
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, "paper_2606_04101_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def load_traffic(kernel, digest):
    """HBM bytes per launch of `kernel` from the committed rocprofv3 PMC
    summary, or None if absent or taken on different kernel source."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        d = json.load(f).get(kernel)
    if not d or d.get("source_digest") != digest:
        return None
    return d.get("hbm_bytes_per_launch")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extensions", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--workloads", action="store_true",
                    help="instead of the step: count, plan, dispatch and pack of every "
                         "workload, with the oracle beside them (one JSON line each)")
    ap.add_argument("--only", type=int, action="append", default=None,
                    help="with --workloads: this workload id only (repeatable)")
    args = ap.parse_args()
    if args.workloads:
        return per_workload(args)
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}): the "
              "balancing path is replicated per rank and its collectives are not "
              "implemented here.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import gen
    import paper_2606_04101_amd as uep

    dev = torch.device("cuda:0")
    c = gen.config(WORKLOAD_ID)
    g = uep.Group(c.R, c.E, c.n_slot, c.u_min, c.beta_num, c.beta_den)
    T, k, H, W = c.T, c.k, c.H, c.W
    V = T * k

    # ---------------- inputs (generated on the host, uploaded once)
    t0 = time.time()
    tk_all = gen.topk_all(c, 0)
    tk_all_d = torch.from_numpy(tk_all).to(dev)
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    load = torch.empty((c.R, c.E), dtype=torch.int32, device=dev)
    uep.ultraep_count(tk_all_d, T, k, c.E, c.R, load, status)  # every rank's row
    plan = uep.Plan(g, dev)
    uep.ultraep_plan(load, g, plan)
    torch.cuda.synchronize()
    X = plan.slot_expert.cpu().numpy().reshape(c.R, c.n_slot)
    n_out_r = [int(((X >= 0) & (X // c.n_main == r)).sum()) for r in range(c.R)]
    rank = int(np.argmax(n_out_r))  # ties -> smallest rank
    fan = outbound_fan(X, c.n_main, rank)
    x_h = gen.activations(c, 0, rank)
    w_h = gen.weights(c, rank)
    x = torch.from_numpy(x_h.view(np.int16)).to(dev)
    w = torch.from_numpy(w_h.view(np.int16)).to(dev)
    topk_r = tk_all_d[rank].contiguous()
    load_r = load[rank]
    send = torch.empty((V, H), dtype=torch.int16, device=dev)
    ros = torch.empty(V, dtype=torch.int32, device=dev)
    boff = torch.empty(c.R * g.S + 1, dtype=torch.int64, device=dev)
    ws = torch.empty(uep.ultraep_dispatch_ws_bytes(T, k, g), dtype=torch.uint8, device=dev)
    cap = max(1, n_out_r[rank])
    staging = torch.empty((cap, W), dtype=torch.int16, device=dev)
    doff = torch.empty(c.R + 1, dtype=torch.int64, device=dev)
    torch.cuda.synchronize()
    setup_s = time.time() - t0

    calls = [
        ("count", lambda: uep.ultraep_count(topk_r, T, k, c.E, 1, load_r, status)),
        ("plan_replicate", lambda: uep.ultraep_plan_replicate(load, g, plan)),
        ("reroute_and_pack", lambda: uep.ultraep_reroute_and_pack(
            load, g, plan, w, W, rank, staging, cap, doff, status)),
        ("dispatch_layout", lambda: uep.ultraep_dispatch_layout(
            topk_r, T, k, rank, g, plan, ros, boff, ws, status)),
        ("dispatch_scatter", lambda: uep.ultraep_dispatch_scatter(
            x, T, k, H, ros, boff[-1:], send)),
    ]

    def step():
        for _, f in calls:
            f()

    outputs = (load_r, send, ros, boff, staging, doff,
               *[getattr(plan, f) for f in uep.PLAN_FIELDS])
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    ref = [t.clone() for t in outputs]

    # ---------------- timed region: K steps as graph replays.  A graph holds
    # G consecutive steps (G = 10 when it divides K): a step launched inside a
    # larger graph, as a training or serving step would launch its layers,
    # does not pay the fixed cost of a graph launch (about 8 µs here) alone.
    G = 10 if args.steps % 10 == 0 else 1

    def make_graph(n_steps):
        gr = torch.cuda.CUDAGraph()
        with torch.cuda.graph(gr):
            for _ in range(n_steps):
                step()
        return gr

    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    graph = make_graph(G)
    for t in outputs:
        t.fill_(-1)
    for _ in range(max(1, args.warmup // G)):
        graph.replay()
    torch.cuda.synchronize()
    for a, b in zip(outputs, ref):
        assert torch.equal(a, b), "graph replay differs from the eager step"
    # a HIP event between consecutive replays gives the spread of the step
    # time (per replay) next to the wall-clock mean
    n_rep = args.steps // G
    rep_ev = [torch.cuda.Event(enable_timing=True) for _ in range(n_rep + 1)]
    t_start = time.perf_counter()
    rep_ev[0].record()
    for i in range(n_rep):
        graph.replay()
        rep_ev[i + 1].record()
    torch.cuda.synchronize()
    t_graph = (time.perf_counter() - t_start) / args.steps
    rep_us = [1e3 * rep_ev[i].elapsed_time(rep_ev[i + 1]) / G for i in range(n_rep)]
    del ref, graph
    # the same steps with one step per graph launch, for reference
    graph1 = make_graph(1)
    for _ in range(max(1, args.warmup)):
        graph1.replay()
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for _ in range(args.steps):
        graph1.replay()
    torch.cuda.synchronize()
    t_graph1 = (time.perf_counter() - t_start) / args.steps
    del graph1

    # ---------------- eager pass with a HIP event between consecutive launches
    # on the launch stream: call i lasts from event i to event i + 1.  The
    # stream first holds on a short spin while the host enqueues the whole
    # pass, so no launch waits on the host and an event pair brackets the
    # kernel alone (plus the event itself)
    stream = torch.cuda.current_stream()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(len(calls) + 1)]
           for _ in range(args.steps)]
    torch.cuda.synchronize()
    hold_stream()
    for i in range(args.steps):
        evs[i][0].record(stream)
        for j, (_, f) in enumerate(calls):
            f()
            evs[i][j + 1].record(stream)
    torch.cuda.synchronize()
    t_eager = 1e-3 * evs[0][0].elapsed_time(evs[-1][-1]) / args.steps

    def span_us(j0, j1):
        return 1e3 * float(np.mean([evs[i][j0].elapsed_time(evs[i][j1])
                                    for i in range(args.steps)]))

    per_call_us = {name: span_us(j, j + 1) for j, (name, _) in enumerate(calls)}

    # ---------------- the pieces measured on their own, event-timed: the
    # packing kernel alone (its bandwidth), and count + ultraep_plan (the
    # reroute fused into the planner's last kernel) as one pair
    def eager_us(fns, reps):
        e = [torch.cuda.Event(enable_timing=True) for _ in range(reps + 1)]
        torch.cuda.synchronize()
        hold_stream()
        e[0].record(stream)
        for i in range(reps):
            for f in fns:
                f()
            e[i + 1].record(stream)
        torch.cuda.synchronize()
        return 1e3 * float(np.mean([e[i].elapsed_time(e[i + 1]) for i in range(reps)]))

    count_fn = calls[0][1]
    plan_fn = lambda: uep.ultraep_plan(load, g, plan)
    pack_fn = lambda: uep.ultraep_pack_replicas(w, W, rank, g, plan, staging, cap, doff, status)
    per_call_us["pack"] = eager_us([pack_fn], args.steps)
    per_call_us["plan"] = eager_us([plan_fn], args.steps)
    count_plan_us = eager_us([count_fn, plan_fn], args.steps)
    st = int(status.item())
    assert st == 0, f"device status {st}: {uep.ultraep_strerror(st)}"
    n_routed = int(boff[-1].item())

    # ---------------- count + plan latency without host launch gaps: 20
    # consecutive pairs captured in one graph (each pair waits for the one
    # before it on the stream), one replay, divided by 20
    n_pairs = 20
    pair_graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(pair_graph):
        for _ in range(n_pairs):
            count_fn()
            plan_fn()
    pair_graph.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    pair_us = []
    for _ in range(5):
        e0.record()
        pair_graph.replay()
        e1.record()
        torch.cuda.synchronize()
        pair_us.append(1e3 * e0.elapsed_time(e1) / n_pairs)
    count_plan_graph_us = float(np.median(pair_us))
    del pair_graph

    # ---------------- a plain copy of known size (achievable bandwidth and
    # the reference kernel for scaling the HBM byte counters)
    a = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
    b = torch.empty_like(a)
    for _ in range(3):
        b.copy_(a)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(10):
        b.copy_(a)
    e1.record()
    torch.cuda.synchronize()
    copy_gbps = 2 * a.numel() * 10 / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del a, b

    # ---------------- algorithmic bytes per launch
    scatter_bytes, pack_bytes = algorithmic_bytes(T, H, k, n_routed, W, fan)
    kern = {
        "dispatch_scatter": (scatter_bytes, per_call_us["dispatch_scatter"],
                             ["dispatch.hip", "common.hpp"]),
        "pack": (pack_bytes, per_call_us["pack"], ["pack.hip", "pack_core.hpp", "common.hpp"]),
    }
    dom = max(kern, key=lambda n: kern[n][1])
    dbytes, dus, dsrc = kern[dom]
    achieved = dbytes / (dus * 1e-6) / 1e9
    traffic = load_traffic(dom, kernel_source_digest(dsrc))

    out = {
        "metric": METRIC,
        "value": round(t_graph * 1e6, 2),
        "unit": "µs",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(t_graph * 1e3, 4),
        "step_us_spread": {"per": f"graph replay of {G} steps", "replays": n_rep,
                           "p10": round(float(np.percentile(rep_us, 10)), 2),
                           "median": round(float(np.median(rep_us)), 2),
                           "p90": round(float(np.percentile(rep_us, 90)), 2)},
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int32",
        "data": "synthetic",
        "config": {
            "workload": (f"{c.name}: DeepSeek-V3-shaped layer, E={c.E} top-{c.k} "
                         f"({c.n_group}-group/top-{c.top_group}), R={c.R} simulated "
                         f"ranks, n_slot={c.n_slot}, T={T} tokens/rank, H={H}, "
                         f"F={c.F}, bf16 rows and expert blobs (bit copies); "
                         f"measured rank {rank}"),
            "rank": rank,
            "tokens_per_rank": T,
            "routed_rows": n_routed,
            "replicas_shipped": int(n_out_r[rank]),
            "expert_blob_bytes": 2 * W,
            "timed": ("HIP graph replays of count, replicate, reroute + pack, "
                      "dispatch layout, scatter"),
            "steps_per_graph": G,
        },
        "roofline": {
            "kernel": dom,
            "bound": "hbm",
            "achieved": round(achieved, 1),
            "peak": PEAK_HBM_GBPS,
            "unit": "GB/s",
            "frac": round(achieved / PEAK_HBM_GBPS, 4),
            "traffic": traffic,
            "algorithmic_bytes_per_launch": dbytes,
            "avg_launch_us": round(dus, 2),
        },
        "kernels_us": {n: round(v, 2) for n, v in per_call_us.items()},
        "count_plan_us": round(count_plan_graph_us, 2),
        "count_plan_eager_us": round(count_plan_us, 2),
        "one_step_graph_us": round(t_graph1 * 1e6, 2),
        "eager_us_per_step": round(t_eager * 1e6, 2),
        "dispatch_scatter_GBps": round(scatter_bytes / per_call_us["dispatch_scatter"] / 1e3, 1),
        "pack_GBps": round(pack_bytes / per_call_us["pack"] / 1e3, 1) if pack_bytes else None,
        "copy_reference_GBps": round(copy_gbps, 1),
        "setup_s": round(setup_s, 2),
    }

    if not args.no_extensions:
        out["extensions"] = extensions(args, dev, stream, c, g, plan, load, rank, send,
                                       ros, boff, n_routed, w, W, fan, eager_us)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(c, tk_all, rank, x_h, w_h, cap,
                                           args.cpu_seconds)
    print(json.dumps(out), flush=True)


def extensions(args, dev, stream, c, g, plan, load, rank, send, ros, boff, n_routed,
               w, W, fan, eager_us):
    """The steps next to the balancing path, each timed with HIP events on
    the launch stream (mean over --steps launches after warm-up):
      combine      the gate-weighted gather of the experts' output rows back
                   to token order, on this step's dispatch layout;
      grad_reduce  the local gradient reduction of this rank's replicated
                   experts (fp32 gradients, blobs of the layer's size);
      relay_plan   the relay trees of the hot experts, on this layer's plan
                   and on the Qwen3-235B-shaped and DeepSeek-V3 prefill plans
                   (where experts exceed four replicas);
      pack_relay   the local packing under those trees on the
                   Qwen3-235B-shaped layer, for the rank that sends the most.
    Bandwidth figures use algorithmic bytes (each source byte read once,
    each destination byte written once) against the 8 TB/s peak."""
    import numpy as np
    import torch

    import gen
    import paper_2606_04101_amd as uep

    T, k, H = c.T, c.k, c.H
    V = T * k
    reps = max(5, min(args.steps, 50))
    res = {}

    def bw(nbytes, us):
        gbps = nbytes / (us * 1e-6) / 1e9
        return {"us": round(us, 2), "algorithmic_bytes": int(nbytes), "GBps": round(gbps, 1),
                "frac": round(gbps / PEAK_HBM_GBPS, 4)}

    def warm(f, n=3):
        for _ in range(n):
            f()
        torch.cuda.synchronize()

    # ---- combine on this step's layout (send stands in for the experts'
    # output rows: same layout and size)
    rng = np.random.default_rng(4101)
    z = rng.standard_normal((T, k))
    gate = torch.from_numpy((np.exp(z) / np.exp(z).sum(1, keepdims=True)).astype(np.float32)).to(dev)
    out_t = torch.empty((T, H), dtype=torch.int16, device=dev)
    st = torch.zeros(1, dtype=torch.int32, device=dev)
    f = lambda: uep.ultraep_combine(send, V, gate, ros, T, k, H, out_t, st)
    warm(f)
    res["combine"] = bw(2 * n_routed * H + 2 * T * H + 8 * V, eager_us([f], reps))

    # ---- gradient reduction of this rank's replicated experts
    nm = c.n_main
    n_rep = int(sum(fan))
    mg = torch.zeros((nm, W), dtype=torch.float32, device=dev)
    rg = torch.zeros((max(n_rep, 1), W), dtype=torch.float32, device=dev)
    f = lambda: uep.ultraep_grad_reduce(mg, rg, W, rank, g, plan, max(n_rep, 1), st)
    warm(f)
    res["grad_reduce"] = bw(int(sum(4 * W * (2 + 2 * fv) for fv in fan if fv > 0)),
                            eager_us([f], reps))
    res["grad_reduce"]["replicas"] = n_rep
    del mg, rg

    # ---- relay trees: latency of one call, from a graph of 20 calls
    def relay_us(gg, pl):
        src = torch.empty(max(gg.R * gg.n_slot, 1), dtype=torch.int32, device=dev)
        vol = torch.empty(gg.R, dtype=torch.int32, device=dev)
        rs = torch.empty(4, dtype=torch.int64, device=dev)
        fn = lambda: uep.ultraep_relay_plan(gg, pl, 4, src, vol, rs, st)
        warm(fn)
        gr = torch.cuda.CUDAGraph()
        with torch.cuda.graph(gr):
            for _ in range(20):
                fn()
        gr.replay()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        ts = []
        for _ in range(5):
            e0.record()
            gr.replay()
            e1.record()
            torch.cuda.synchronize()
            ts.append(1e3 * e0.elapsed_time(e1) / 20)
        return float(np.median(ts)), src, vol, rs.cpu().tolist()

    us, _, _, rst = relay_us(g, plan)
    rel = {c.name: {"us": round(us, 2), "relay_experts": rst[0], "max_send_blobs": [rst[2], rst[3]]}}
    for cid in (3, 5):
        cc = gen.config(cid)
        gg = uep.Group(cc.R, cc.E, cc.n_slot, cc.u_min, cc.beta_num, cc.beta_den)
        tk = torch.from_numpy(gen.topk_all(cc, 0)).to(dev)
        ld = torch.empty((cc.R, cc.E), dtype=torch.int32, device=dev)
        uep.ultraep_count(tk, cc.T, cc.k, cc.E, cc.R, ld, st)
        pl = uep.Plan(gg, dev)
        uep.ultraep_plan(ld, gg, pl)
        us, src, vol, rst = relay_us(gg, pl)
        rel[cc.name] = {"us": round(us, 2), "relay_experts": rst[0],
                        "max_send_blobs": [rst[2], rst[3]]}
        if cid == 3:  # the packing under these trees, for the busiest sender
            r3 = int(torch.argmax(vol).item())
            Xh = pl.slot_expert.cpu().numpy().reshape(cc.R, cc.n_slot)
            sh = src.cpu().numpy()[: cc.R * cc.n_slot].reshape(cc.R, cc.n_slot)
            n_send = int(((Xh >= 0) & (sh == r3)).sum())
            srcs = {}  # source blob -> copies
            for t in range(cc.R):
                for s_ in range(cc.n_slot):
                    if Xh[t, s_] >= 0 and sh[t, s_] == r3:
                        srcs[int(Xh[t, s_])] = srcs.get(int(Xh[t, s_]), 0) + 1
            W3 = cc.W
            w3 = torch.zeros((cc.n_main, W3), dtype=torch.int16, device=dev)
            rsrc = torch.zeros((cc.n_slot, W3), dtype=torch.int16, device=dev)
            stg = torch.empty((max(n_send, 1), W3), dtype=torch.int16, device=dev)
            doff = torch.empty(cc.R + 1, dtype=torch.int64, device=dev)
            fn = lambda: uep.ultraep_pack_relay(w3, rsrc, W3, r3, gg, pl, src, stg,
                                                max(n_send, 1), doff, st)
            warm(fn)
            res["pack_relay"] = bw(sum(2 * W3 * (1 + n) for n in srcs.values()), eager_us([fn], reps))
            res["pack_relay"].update({"workload": cc.name, "rank": r3, "copies": n_send,
                                      "source_blobs": len(srcs)})
            del w3, rsrc, stg
        del tk, ld, pl
    res["relay_plan"] = rel
    torch.cuda.synchronize()
    assert int(st.item()) == 0, f"device status {int(st.item())}"
    return res


def per_workload(args):
    """Count, plan, dispatch and pack of the five workloads, each on its
    measured rank (most outbound replicas), the oracle run beside it on the
    same inputs and every output compared byte for byte.  The Qwen3-235B-
    shaped workload runs all 16 microbatches of its drifting router and the
    DeepSeek-V3 prefill workload all 58 layers (each reported, then the
    median; the prefill layers' count + plan also back to back in one graph).
    Timing:
      count, plan, replicate, reroute   graph of 20 consecutive calls, replayed
                                        5 times: median per call
      dispatch, scatter, pack           one HIP event pair per launch (the
                                        stream holds while the host enqueues),
                                        50 launches (20 for the prefill
                                        layers), each after an untimed 512 MiB
                                        write that evicts the 256 MB MALL:
                                        median, p10, p90
      scatter, pack (clean)             the same after an untimed 512 MiB read
                                        instead: the MALL holds none of the
                                        kernel's data and no dirty lines, so
                                        the kernel pays no write-back of
                                        another kernel's output
    Every layer and microbatch uses the activations and weights of the first
    one's measured rank (the bytes moved do not depend on their values)."""
    import numpy as np
    import torch

    import gen
    import paper_2606_04101_amd as uep

    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    scratch = torch.empty(512 << 20, dtype=torch.uint8, device=dev)

    def pct(ts):
        ts = np.asarray(ts)
        return {"median": round(float(np.median(ts)), 2), "p10": round(float(np.percentile(ts, 10)), 2),
                "p90": round(float(np.percentile(ts, 90)), 2)}

    scratch_sum = torch.zeros((), dtype=torch.int64, device=dev)

    def cold_us(f, n, clean=False):
        f()
        torch.cuda.synchronize()
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(n)]
        hold_stream()
        for e0, e1 in ev:
            if clean:
                torch.sum(scratch.view(torch.int64), dim=0, out=scratch_sum)
            else:
                scratch.zero_()
            e0.record(stream)
            f()
            e1.record(stream)
        torch.cuda.synchronize()
        return pct([1e3 * e0.elapsed_time(e1) for e0, e1 in ev])

    def graph_us(fns, n=20):
        for f in fns:
            f()
        torch.cuda.synchronize()
        gr = torch.cuda.CUDAGraph()
        with torch.cuda.graph(gr):
            for _ in range(n):
                for f in fns:
                    f()
        gr.replay()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        ts = []
        for _ in range(5):
            e0.record()
            gr.replay()
            e1.record()
            torch.cuda.synchronize()
            ts.append(1e3 * e0.elapsed_time(e1) / n)
        return round(float(np.median(ts)), 2)

    gap = quality_gap_table()

    def instance(c, m, g, xw, n_cold):
        """One microbatch / layer m of workload c; xw holds the activations and
        weights (host and device) of the first instance's measured rank."""
        T, k, H, W = c.T, c.k, c.H, c.W
        V = T * k
        tk_all = gen.topk_all(c, m)
        tk_d = torch.from_numpy(tk_all).to(dev)
        st = torch.zeros(1, dtype=torch.int32, device=dev)
        load = torch.empty((c.R, c.E), dtype=torch.int32, device=dev)
        uep.ultraep_count(tk_d, T, k, c.E, c.R, load, st)
        plan = uep.Plan(g, dev)
        uep.ultraep_plan(load, g, plan)
        torch.cuda.synchronize()
        X = plan.slot_expert.cpu().numpy().reshape(c.R, c.n_slot)
        outb = [int(((X >= 0) & (X // c.n_main == r)).sum()) for r in range(c.R)]
        rank = int(np.argmax(outb))
        if not xw:
            x_h, w_h = gen.activations(c, m, rank), gen.weights(c, rank)
            xw.update(x_h=x_h, w_h=w_h, x=torch.from_numpy(x_h.view(np.int16)).to(dev),
                      w=torch.from_numpy(w_h.view(np.int16)).to(dev),
                      send=torch.empty((V, H), dtype=torch.int16, device=dev),
                      stg=torch.empty((max(1, c.R * c.n_slot), W), dtype=torch.int16, device=dev))
        x, w, send, stg = xw["x"], xw["w"], xw["send"], xw["stg"]
        tk_r = tk_d[rank].contiguous()
        load_r = load[rank]
        ros = torch.empty(V, dtype=torch.int32, device=dev)
        boff = torch.empty(c.R * g.S + 1, dtype=torch.int64, device=dev)
        ws = torch.empty(uep.ultraep_dispatch_ws_bytes(T, k, g), dtype=torch.uint8, device=dev)
        cap = max(1, outb[rank])
        doff = torch.empty(c.R + 1, dtype=torch.int64, device=dev)
        count_f = lambda: uep.ultraep_count(tk_r, T, k, c.E, 1, load_r, st)
        plan_f = lambda: uep.ultraep_plan(load, g, plan)
        disp_f = lambda: uep.ultraep_dispatch(x, tk_r, T, k, H, rank, g, plan, send, ros, boff,
                                              ws, st)
        scat_f = lambda: uep.ultraep_dispatch_scatter(x, T, k, H, ros, boff[-1:], send)
        pack_f = lambda: uep.ultraep_pack_replicas(w, W, rank, g, plan, stg, cap, doff, st)
        rec = {"workload": c.name, "m": m, "rank": rank, "replicas_shipped": outb[rank]}
        rec["count_us"] = graph_us([count_f])
        rec["plan_us"] = graph_us([plan_f])
        rec["count_plan_us"] = graph_us([count_f, plan_f])
        rec["replicate_us"] = graph_us([lambda: uep.ultraep_plan_replicate(load, g, plan)])
        rec["reroute_us"] = graph_us([lambda: uep.ultraep_plan_reroute(load, g, plan)])
        rec["max_hosts"] = int(plan.stats[5].item())
        # balancing quality: the bisection's threshold and the max rank load
        # of its plan over the mean, next to the smallest greedy-feasible
        # threshold of the stored table (written by the oracle-only script
        # tests/golden/quality_gap.py)
        Uq = plan.quota.cpu().numpy().reshape(c.E, c.R).astype(np.int64)
        mean_load = float(Uq.sum()) / c.R
        rec["tau_star"] = int(plan.stats[0].item())
        rec["imbalance_after"] = round(float(Uq.sum(0).max()) / mean_load, 4) if mean_load else 1.0
        row = gap.get(("w", c.cid, m))
        if row:
            rec["tau_min_feasible"] = row["tau_min"]
            rec["imbalance_at_tau_min"] = row["imbalance_min"]
        rec["dispatch_us"] = cold_us(disp_f, n_cold)
        rec["scatter_us"] = cold_us(scat_f, n_cold)
        rec["pack_us"] = cold_us(pack_f, n_cold) if outb[rank] else None
        rec["scatter_us_clean"] = cold_us(scat_f, n_cold, clean=True)
        rec["pack_us_clean"] = cold_us(pack_f, n_cold, clean=True) if outb[rank] else None
        torch.cuda.synchronize()
        assert int(st.item()) == 0, int(st.item())
        n_routed = int(boff[-1].item())
        sb, pb = algorithmic_bytes(T, H, k, n_routed, W, outbound_fan(X, c.n_main, rank))
        rec["scatter_bytes"] = sb
        rec["scatter_GBps"] = round(sb / rec["scatter_us"]["median"] / 1e3, 1)
        rec["pack_bytes"] = pb
        rec["pack_GBps"] = round(pb / rec["pack_us"]["median"] / 1e3, 1) if pb else None
        rec["scatter_GBps_clean"] = round(sb / rec["scatter_us_clean"]["median"] / 1e3, 1)
        rec["pack_GBps_clean"] = (round(pb / rec["pack_us_clean"]["median"] / 1e3, 1)
                                  if pb else None)
        # the CPU baseline on the same inputs, and whether it agrees byte for byte
        base = oracle_baseline(c, tk_all, rank, xw["x_h"], xw["w_h"], cap)
        o = base["outputs"]
        n_out = o["n_out"]
        exact = (np.array_equal(load.cpu().numpy(), o["counts"])
                 and all(np.array_equal(getattr(plan, f).cpu().numpy().reshape(-1),
                                        o["plan"][f].reshape(-1)) for f in uep.PLAN_FIELDS)
                 and np.array_equal(ros.cpu().numpy(), o["row_of_slot"])
                 and np.array_equal(boff.cpu().numpy(), o["block_off"])
                 and np.array_equal(send.cpu().numpy().view(np.uint16), o["send"])
                 and np.array_equal(doff.cpu().numpy(), o["dest_off"])
                 and np.array_equal(stg[:n_out].cpu().numpy().view(np.uint16), o["staging"][:n_out]))
        rec["oracle_us"] = base["us"]
        rec["bit_exact"] = bool(exact)
        del base, o
        return rec, (tk_r, load, plan, rank)

    for cid in sorted(gen.WORKLOADS):
        if args.only and cid not in args.only:
            continue
        c = gen.config(cid)
        g = uep.Group(c.R, c.E, c.n_slot, c.u_min, c.beta_num, c.beta_den)
        shape = {"R": c.R, "E": c.E, "n_slot": c.n_slot, "k": c.k, "T": c.T, "H": c.H, "F": c.F}
        ms = list(range(c.n_micro)) if cid in (3, 5) else [0]
        n_cold = 20 if cid == 5 else 50
        xw, recs, keep = {}, [], []
        for m in ms:
            rec, kp = instance(c, m, g, xw, n_cold)
            if m == 0:
                rec.update(shape)
            recs.append(rec)
            if cid == 5:
                keep.append(kp)
            print(json.dumps(rec), flush=True)
        if len(ms) > 1:
            med = lambda key, sub=None: round(float(np.median(
                [r[key][sub] if sub else r[key] for r in recs])), 2)
            summ = {"workload": c.name, "instances": len(ms), **shape,
                    "median": {"count_us": med("count_us"), "plan_us": med("plan_us"),
                               "count_plan_us": med("count_plan_us"),
                               "replicate_us": med("replicate_us"), "reroute_us": med("reroute_us"),
                               "dispatch_us": med("dispatch_us", "median"),
                               "scatter_us": med("scatter_us", "median"),
                               "pack_us": round(float(np.median([r["pack_us"]["median"] for r in recs
                                                                 if r["pack_us"]])), 2),
                               "scatter_GBps": med("scatter_GBps"),
                               "scatter_us_clean": med("scatter_us_clean", "median"),
                               "pack_us_clean": round(float(np.median(
                                   [r["pack_us_clean"]["median"] for r in recs
                                    if r["pack_us_clean"]])), 2),
                               "imbalance_after": med("imbalance_after")},
                    "max": {"count_plan_us": max(r["count_plan_us"] for r in recs),
                            "max_hosts": max(r["max_hosts"] for r in recs)},
                    "bit_exact_all": all(r["bit_exact"] for r in recs)}
            if all("imbalance_at_tau_min" in r for r in recs):
                summ["median"]["imbalance_at_tau_min"] = med("imbalance_at_tau_min")
            if cid == 5:
                # count + plan of every layer back to back: one graph, 58 pairs
                st = torch.zeros(1, dtype=torch.int32, device=dev)
                fns = []
                for tk_r, load, plan, rank in keep:
                    fns.append(lambda tk_r=tk_r, load=load, rank=rank: uep.ultraep_count(
                        tk_r, c.T, c.k, c.E, 1, load[rank], st))
                    fns.append(lambda load=load, plan=plan: uep.ultraep_plan(load, g, plan))
                tot = graph_us(fns, n=1)
                assert int(st.item()) == 0
                summ["all_layers_count_plan_us"] = {"total": tot, "per_layer": round(tot / len(ms), 2)}
            print(json.dumps({"summary": summ}), flush=True)
        del xw, recs, keep
        torch.cuda.empty_cache()


def quality_gap_table():
    """Rows of tests/golden/quality_gap.json keyed by ("w", workload,
    instance) and ("s", E, R, n_slot, alpha, tokens); empty if absent."""
    path = os.path.join(ROOT, "tests", "golden", "quality_gap.json")
    if not os.path.exists(path):
        return {}
    with open(path) as f:
        doc = json.load(f)
    out = {("w", r["workload"], r["instance"]): r for r in doc["workloads"]}
    out.update({("s", r["E"], r["R"], r["n_slot"], r["alpha"], r["tokens"]): r
                for r in doc["sweep"]})
    return out


def oracle_baseline(c, tk_all, rank, x_h, w_h, cap):
    """The CPU-baseline leg of --workloads: the oracle (single-threaded C)
    once on the same inputs as the GPU instance, each step wall-clock timed;
    its outputs come back so the caller can report whether the GPU's agree."""
    import oracle
    import paper_2606_04101_amd as uep
    oracle.lib()  # loaded before the clock starts
    og = oracle.Group(c.R, c.E, c.n_slot, c.u_min, c.beta_num, c.beta_den)

    def wall_us(f):
        t0 = time.perf_counter()
        r = f()
        return r, round(1e6 * (time.perf_counter() - t0), 1)

    (ocnt, _), t_cnt = wall_us(lambda: oracle.count(tk_all, c.E, c.R))
    op, t_plan = wall_us(lambda: oracle.plan(ocnt, og))
    (osend, oros, oboff, _), t_disp = wall_us(
        lambda: oracle.dispatch(x_h, tk_all[rank], rank, og, op, poison=False))
    (ostg, odoff, n_out, _), t_pack = wall_us(lambda: oracle.pack(w_h, rank, og, op, cap))
    return {"us": {"count_all_ranks": t_cnt, "count_one_rank": round(t_cnt / c.R, 1),
                   "plan": t_plan, "dispatch": t_disp, "pack": t_pack, "cores": 1},
            "outputs": {"counts": ocnt, "plan": {f: getattr(op, f) for f in uep.PLAN_FIELDS},
                        "row_of_slot": oros, "block_off": oboff, "send": osend,
                        "dest_off": odoff, "staging": ostg, "n_out": n_out}}


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(c, tk_all, rank, x_h, w_h, cap, budget_s):
    """The oracle (single-threaded C) on the same step, repeated until about
    budget_s seconds of CPU work have been spent (at least one step)."""
    import oracle
    og = oracle.Group(c.R, c.E, c.n_slot, c.u_min, c.beta_num, c.beta_den)
    tk_r = tk_all[rank]
    load, _ = oracle.count(tk_all, c.E, c.R)  # the resident rows, not timed
    parts = {"count": 0.0, "plan": 0.0, "dispatch": 0.0, "pack": 0.0}
    n = 0
    t_all = time.perf_counter()
    while True:
        t0 = time.perf_counter()
        row, _ = oracle.count(tk_r, c.E)
        t1 = time.perf_counter()
        load[rank] = row[0]
        p = oracle.plan(load, og)
        t2 = time.perf_counter()
        _, _, _, st = oracle.dispatch(x_h, tk_r, rank, og, p, poison=False)
        t3 = time.perf_counter()
        _, _, _, st2 = oracle.pack(w_h, rank, og, p, cap)
        t4 = time.perf_counter()
        assert st == 0 and st2 == 0
        for key, dt in zip(parts, (t1 - t0, t2 - t1, t3 - t2, t4 - t3)):
            parts[key] += dt
        n += 1
        if time.perf_counter() - t_all >= budget_s:
            break
    tot = sum(parts.values())
    return {
        "value": round(tot / n * 1e6, 1),
        "unit": "µs",
        "cores": 1,
        "kind": "oracle",
        "sample": (f"{n} full steps of the same workload and rank (count, plan, "
                   f"dispatch with row copies, pack with blob copies), "
                   f"{tot:.1f} s of single-threaded C on {os.cpu_count()} host cores"),
        "cpu_model": cpu_model(),
        "parts_us": {kk: round(v / n * 1e6, 1) for kk, v in parts.items()},
    }


if __name__ == "__main__":
    main()
