#!/usr/bin/env python3
"""Balancing quality of Algorithm 1's bisection against the smallest
greedy-feasible threshold, computed with the oracle only; writes
quality_gap.json beside this file.

Sec. 5.1 states the aim of SolveReplication as the smallest load threshold
tau whose greedy probe is feasible, and Algorithm 1 searches for it by
bisection over [tau_lo0, tau_hi0].  The probe is not monotone in tau (a
transfer below u_min ends an expert's loop, so an overloaded rank whose
last excess is smaller than u_min fails at one tau and succeeds a little
higher; the W1 worked example), so the bisection can settle above the
smallest feasible tau.  For every input this script records:
  tau_star, imbalance_star   the bisection's threshold and the max rank load
                             of its plan over the mean load (the oracle's
                             plan, which the GPU planner equals)
  tau_min, imbalance_min     the smallest tau in [tau_lo0, tau_hi0] whose
                             probe is feasible (a linear scan of probes upward
                             from tau_lo0), and the max rank load of that
                             probe's quotas over the mean
  replicas_star / _min       redundant slots the two plans consume
  inflight, inflight_no_      share of routed tokens served off their rank by
  locality                   the bisection's plan, with and without the
                             locality pass of SolveReroute
Inputs: the five seeded workloads (all 16 microbatches of the drifting
router, the first 8 prefill layers) and the solver-quality sweep's grid.

Usage: python tests/golden/quality_gap.py [--quick]
"""
from __future__ import annotations

import json
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import gen  # noqa: E402
import oracle  # noqa: E402

OUT = os.path.join(HERE, "quality_gap.json")


def smallest_feasible(load, og, lo, hi):
    """The smallest tau in [lo, hi] whose probe is feasible, with that probe's
    quotas; (None, None) if none is."""
    for tau in range(lo, hi + 1):
        feas, Ut, X, st = oracle.probe(load, og, tau)
        assert st == oracle.OK, st
        if feas:
            return tau, Ut, X
    return None, None, None


def gap_row(load, og):
    p = oracle.plan(load, og)
    assert p.status == oracle.OK
    L = int(load.sum())
    mean = L / og.R
    tau_star, lo, hi = (int(v) for v in p.stats[:3])
    U = p.quota.astype(np.int64)
    # the in-flight token ratio of this plan's reroute, and of the reroute
    # without the locality pass (every source's whole demand split by the
    # sequential largest remainder over the quotas), for Table 3's pair
    q = oracle.plan(load, og, locality=False)
    assert q.status == oracle.OK
    row = {"tau_lo0": lo, "tau_hi0": hi, "tau_star": tau_star,
           "imbalance_before": round(float(load.sum(0).reshape(og.R, -1).sum(1).max() / mean), 4),
           "imbalance_star": round(float(U.sum(0).max() / mean), 4),
           "replicas_star": int((p.slot_expert >= 0).sum()),
           "inflight": round(oracle.metrics(load, og, p)["inflight_ratio"], 4),
           "inflight_no_locality": round(oracle.metrics(load, og, q)["inflight_ratio"], 4)}
    if lo >= hi:  # already balanced: the identity plan, no probe
        row.update(tau_min=tau_star, imbalance_min=row["imbalance_star"],
                   replicas_min=row["replicas_star"])
        return row
    tmin, Ut, X = smallest_feasible(load, og, lo, hi)
    row.update(tau_min=tmin, imbalance_min=round(float(Ut.sum(0).max() / mean), 4),
               replicas_min=int((X >= 0).sum()))
    return row


def workloads():
    out = []
    for cid in (1, 2, 3, 4, 5):
        c = gen.config(cid)
        og = oracle.Group(c.R, c.E, c.n_slot, c.u_min, c.beta_num, c.beta_den)
        n = c.n_micro if c.bias == "drift" else (8 if c.bias == "burst" else 1)
        for m in range(n):
            load, st = oracle.count(gen.topk_all(c, m), c.E, c.R)
            assert st == oracle.OK
            row = gap_row(load, og)
            row.update(workload=cid, name=c.name, instance=m)
            out.append(row)
            print(f"workload {cid} #{m}: tau* {row['tau_star']} ({row['imbalance_star']}) "
                  f"tau_min {row['tau_min']} ({row['imbalance_min']})", flush=True)
    return out


def sweep(quick=False):
    import bench_solver
    out = []
    for c in bench_solver.sweep_configs(8192, quick):
        og = oracle.Group(c.R, c.E, c.n_slot, c.u_min, c.beta_num, c.beta_den)
        load, st = oracle.count(gen.topk_all(c, 0), c.E, c.R)
        assert st == oracle.OK
        row = gap_row(load, og)
        row.update(E=c.E, R=c.R, n_slot=c.n_slot, alpha=c.bias_scale, tokens=c.T)
        out.append(row)
        print(f"sweep E={c.E} R={c.R} n_slot={c.n_slot} alpha={c.bias_scale}: "
              f"{row['imbalance_star']} -> {row['imbalance_min']}", flush=True)
    return out


def main():
    quick = "--quick" in sys.argv
    t0 = time.time()
    wl = workloads()
    sw = sweep(quick)
    doc = {"what": "bisection threshold tau* against the smallest greedy-feasible tau "
                   "(linear scan of probes from tau_lo0), oracle only",
           "workloads": wl, "sweep": sw,
           "sweep_average": {k: round(float(np.mean([r[k] for r in sw])), 4)
                             for k in ("imbalance_before", "imbalance_star", "imbalance_min",
                                       "replicas_star", "replicas_min", "inflight",
                                       "inflight_no_locality")}}
    with open(OUT, "w") as f:
        json.dump(doc, f, indent=1)
    print(f"wrote {OUT} in {time.time() - t0:.0f} s")


if __name__ == "__main__":
    main()
