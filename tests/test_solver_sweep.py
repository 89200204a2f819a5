"""The solver-quality sweep's metric code (bench_solver.metrics) against the
oracle's own diagnostics on the same plans, and by hand on a tiny plan; and
(GPU) the planner against the oracle on settings of the sweep grid."""
import numpy as np
import pytest
import torch

import bench_solver
import gen
import oracle


def _sweep_config(E, k, R, NS, alpha, T=512):
    return gen.Config(900, "sweep_test", R=R, E=E, n_slot=NS, k=k, T=T, H=8, F=8,
                      u_min=1024 if T >= 1024 else 32, bias="zipf", zipf_s=1.0, bias_scale=alpha)


@pytest.mark.parametrize("cid", [1, 2, 3, 4])
def test_metrics_match_the_oracle_diagnostics(cid):
    c = gen.config(cid)
    g = oracle.Group(c.R, c.E, c.n_slot, c.u_min, c.beta_num, c.beta_den)
    load, _ = oracle.count(gen.topk_all(c, 0), c.E, c.R)
    p = oracle.plan(load, g)
    m = bench_solver.metrics(load, p.quota, p.host_ptr, p.host_rank, p.reroute)
    o = oracle.metrics(load, g, p)
    assert m["imbalance_before"] == pytest.approx(o["imbalance_before"])
    assert m["imbalance_after"] == pytest.approx(o["imbalance_after"])
    assert m["replicas"] == o["n_replicas"] and m["max_hosts"] == o["max_hosts"]
    assert m["inflight"] == pytest.approx(o["inflight_ratio"])
    # without the locality pass the oracle's split is sequential largest
    # remainder; the sweep reports the proportional share, which it tracks
    q = oracle.plan(load, g, locality=False)
    o2 = oracle.metrics(load, g, q)
    assert abs(m["inflight_no_locality_proportional"] - o2["inflight_ratio"]) < 0.02


def test_metrics_by_hand():
    """R = 2, one main expert each; expert 0 (30 tokens from rank 0, 10 from
    rank 1) keeps quota 25 at home and 15 on a replica on rank 1; expert 1
    has 5 tokens from rank 1.  With locality, rank 1 serves its own 10
    tokens of expert 0 on its replica, and rank 0 keeps 25 and sends 5 to
    rank 1: 5 of 45 tokens are in flight."""
    load = np.array([[30, 0], [10, 5]], np.int32)
    U = np.array([[25, 15], [0, 5]], np.int32)       # u_{0,0}=25, u_{0,1}=15
    hp = np.array([0, 2, 3], np.int32)
    hr = np.array([0, 1, 1, -1], np.int32)
    # q[r][j]: rank 0 -> (e0@0: 25, e0@1: 5); rank 1 -> (e0@0: 0, e0@1: 10, e1@1: 5)
    Q = np.array([[25, 5, 0, 0], [0, 10, 5, 0]], np.int64)
    m = bench_solver.metrics(load, U, hp, hr, Q)
    assert m["imbalance_before"] == pytest.approx(40 / 22.5)
    assert m["imbalance_after"] == pytest.approx(25 / 22.5)
    assert m["replicas"] == 1 and m["sum_hosts"] == 3 and m["max_hosts"] == 2
    assert m["inflight"] == pytest.approx(5 / 45)       # rank 0's 5 tokens on rank 1
    # proportional split: local share = 30*25/40 + 10*15/40 + 5*5/5
    assert m["inflight_no_locality_proportional"] == pytest.approx(1 - (18.75 + 3.75 + 5) / 45)


@pytest.mark.gpu
@pytest.mark.parametrize("E,k,R,NS,alpha", [(128, 8, 16, 1, 0.2), (128, 8, 64, 4, 0.5),
                                            (256, 8, 32, 2, 0.35), (256, 8, 64, 4, 0.5),
                                            (256, 8, 64, 1, 0.2)])
def test_sweep_settings_plan_parity(E, k, R, NS, alpha):
    import gpu_path as gp
    c = _sweep_config(E, k, R, NS, alpha, T=2048)
    g, og = gp.groups(R, E, NS, c.u_min, c.beta_num, c.beta_den)
    tk = gen.topk_all(c, 0)
    counts, st = gp.gpu_count(tk, E)
    ocounts, _ = oracle.count(tk, E, R)
    assert st == 0 and np.array_equal(counts, ocounts)
    gp.assert_plan_equal(gp.gpu_plan(ocounts, g), oracle.plan(ocounts, og))
