"""The stored table of Algorithm 1's bisection threshold against the smallest
greedy-feasible threshold (tests/golden/quality_gap.json, written by
tests/golden/quality_gap.py with the oracle only): its scan is pinned by the
hand-derived W1 example (bisection 45, linear scan 38), its rows are
reproducible, and every row is consistent (tau_lo0 <= tau_min <= tau* <=
tau_hi0, the scan's probe feasible and the one below it not, the in-flight
ratio with the locality pass at most the one without).  CPU only."""
import json
import os
import sys

import numpy as np
import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.join(HERE, "golden"))

import gen  # noqa: E402
import oracle  # noqa: E402
import quality_gap as qg  # noqa: E402

DOC = json.load(open(os.path.join(HERE, "golden", "quality_gap.json")))


def test_scan_on_the_w1_example(orc):
    # Sec. 5.1 worked example W1: R = 3, one expert per rank, one slot,
    # u_min = 10, loads (70, 20, 20): the bisection ends at 45, the smallest
    # feasible threshold is 38 (= tau_lo0)
    og = oracle.Group(3, 3, 1, 10)
    load = np.array([[70, 0, 0], [0, 20, 0], [0, 0, 20]], np.int32)
    row = qg.gap_row(load, og)
    assert (row["tau_lo0"], row["tau_star"], row["tau_min"]) == (38, 45, 38)
    assert row["imbalance_star"] == round(45 / (110 / 3), 4)
    # the probe at 38 moves 18 to rank 1 and 14 to rank 2: loads (38, 38, 34)
    assert row["imbalance_min"] == round(38 / (110 / 3), 4)
    assert row["replicas_star"] == 1 and row["replicas_min"] == 2


@pytest.mark.parametrize("cid", [2, 4])
def test_rows_reproduce(orc, cid):
    c = gen.config(cid)
    og = oracle.Group(c.R, c.E, c.n_slot, c.u_min, c.beta_num, c.beta_den)
    load, _ = oracle.count(gen.topk_all(c, 0), c.E, c.R)
    row = qg.gap_row(load, og)
    stored = [r for r in DOC["workloads"] if r["workload"] == cid and r["instance"] == 0][0]
    for key, v in row.items():
        assert stored[key] == v, key


def test_rows_are_consistent(orc):
    rows = DOC["workloads"] + DOC["sweep"]
    assert len(DOC["workloads"]) == 1 + 1 + 16 + 1 + 8 and len(DOC["sweep"]) == 54
    for r in rows:
        assert r["tau_lo0"] <= r["tau_min"] <= r["tau_star"] <= max(r["tau_hi0"], r["tau_lo0"])
        assert r["imbalance_min"] <= r["imbalance_before"] + 1e-9
        # the locality pass serves min(lambda_{t,e}, u_{e,t}) of every source
        # on its own rank, the most any split can keep there (Sec. 5.2)
        assert 0.0 <= r["inflight"] <= r["inflight_no_locality"] <= 1.0


@pytest.mark.parametrize("idx", [1, 3, 11, 18])
def test_scan_is_minimal(orc, idx):
    """probe(tau_min) is feasible and probe(tau_min - 1) is not (or tau_min is
    the search's lower end), recomputed for a few workload instances."""
    r = DOC["workloads"][idx]
    c = gen.config(r["workload"])
    og = oracle.Group(c.R, c.E, c.n_slot, c.u_min, c.beta_num, c.beta_den)
    load, _ = oracle.count(gen.topk_all(c, r["instance"]), c.E, c.R)
    assert oracle.probe(load, og, r["tau_min"])[0]
    if r["tau_min"] > r["tau_lo0"]:
        assert not oracle.probe(load, og, r["tau_min"] - 1)[0]
