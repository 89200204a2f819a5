"""Invariants I1-I13 of the oracle on the five synthetic workloads, on a
seeded corpus of small adversarial cases and on a mid-size corpus (no GPU)."""
import numpy as np
import pytest

import fuzz
from invariants import check_dispatch, check_pack, check_plan


def _plan_case(orc, load, g):
    p = orc.plan(load, g)
    assert p.status == 0, p.status
    check_plan(load, g, p)
    # I7: the bisection stopped at tau_lo0 or right above an infeasible probe
    tau, lo0, hi0 = (int(v) for v in p.stats[:3])
    if lo0 < hi0 and tau > lo0:
        assert not orc.probe(load, g, tau - 1)[0]
    # the emitted quotas are exactly the last feasible probe's
    if p.stats[4] > 0:
        f, Ut, X, st = orc.probe(load, g, tau)
        assert f and st == 0
        assert np.array_equal(Ut, p.quota) and np.array_equal(X, p.slot_expert)
    return p


WORKLOADS = [(1, 0), (2, 0), (3, 0), (3, 5), (3, 15), (4, 0), (5, 0), (5, 57)]


@pytest.mark.parametrize("cid,m", WORKLOADS)
def test_workload_invariants(orc, gen_mod, cid, m):
    c = gen_mod.config(cid)
    g = orc.Group(c.R, c.E, c.n_slot, c.u_min, c.beta_num, c.beta_den)
    tk = gen_mod.topk_all(c, m)
    load, st = orc.count(tk, c.E, c.R)
    assert st == 0
    # I1: counts match a naive per-expert tally and the number of slots
    assert load.sum() == tk.size
    r0 = tk[0].reshape(-1)
    assert all(load[0, e] == int((r0 == e).sum()) for e in range(0, c.E, 7))
    p = _plan_case(orc, load, g)
    # I13: the plan depends on the load matrix only
    p2 = orc.plan(load.copy(), g)
    assert all(np.array_equal(getattr(p, f), getattr(p2, f)) for f in
               ("slot_expert", "quota", "host_ptr", "host_rank", "host_pslot",
                "reroute", "stats"))
    X = p.slot_expert
    outb = [int(((X >= 0) & (X // c.n_main == r)).sum()) for r in range(c.R)]
    rstar = int(np.argmax(outb))
    for r in sorted({0, rstar, c.R - 1}):
        x = gen_mod.bits16(gen_mod.key(1, cid, m, r), (c.T, 8))
        send, ros, boff, st = orc.dispatch(x, tk[r], r, g, p)
        assert st == 0
        check_dispatch(x, tk[r], r, g, p, send, ros, boff)
        w = gen_mod.bits16(gen_mod.key(2, cid, r), (c.n_main, 40))
        cap = g.R * g.n_slot
        staging, doff, n_out, st = orc.pack(w, r, g, p, cap)
        assert st == 0
        check_pack(w, r, g, p, staging, doff, n_out)


@pytest.mark.parametrize("seed", range(0, 160))
def test_fuzz_case(orc, seed):
    c = fuzz.make_case(seed)
    g = orc.Group(c["R"], c["E"], c["n_slot"], c["u_min"], c["beta_num"],
                  c["beta_den"])
    load, st = orc.count(c["topk"], g.E, g.R)
    assert st == 0
    valid = c["topk"] >= 0
    assert load.sum() == valid.sum()
    p = _plan_case(orc, load, g)
    rng = c["rng"]
    for r in sorted({0, g.R - 1}):
        x = rng.integers(0, 2 ** 16, (c["T"], c["H"])).astype(np.uint16)
        send, ros, boff, st = orc.dispatch(x, c["topk"][r], r, g, p)
        assert st == 0
        check_dispatch(x, c["topk"][r], r, g, p, send, ros, boff)
        w = rng.integers(0, 2 ** 16, (g.n_main, c["W"])).astype(np.uint16)
        staging, doff, n_out, st = orc.pack(w, r, g, p, g.R * g.n_slot)
        assert st == 0
        check_pack(w, r, g, p, staging, doff, n_out)


@pytest.mark.parametrize("seed", range(0, 48))
def test_mid_case(orc, seed):
    """The mid-size corpus: up to 64 ranks, 1024 experts, top-64."""
    c = fuzz.make_mid_case(seed)
    g = orc.Group(c["R"], c["E"], c["n_slot"], c["u_min"], c["beta_num"],
                  c["beta_den"])
    load, st = orc.count(c["topk"], g.E, g.R)
    assert st == 0
    assert load.sum() == (c["topk"] >= 0).sum()
    p = _plan_case(orc, load, g)
    rng = c["rng"]
    X = p.slot_expert.reshape(g.R, max(g.n_slot, 0))
    outb = [int(((X >= 0) & (X // g.n_main == r)).sum()) for r in range(g.R)]
    for r in sorted({0, int(np.argmax(outb)), g.R - 1}):
        x = rng.integers(0, 2 ** 16, (c["T"], 8)).astype(np.uint16)
        send, ros, boff, st = orc.dispatch(x, c["topk"][r], r, g, p)
        assert st == 0
        check_dispatch(x, c["topk"][r], r, g, p, send, ros, boff)
        w = rng.integers(0, 2 ** 16, (g.n_main, 16)).astype(np.uint16)
        staging, doff, n_out, st = orc.pack(w, r, g, p, g.R * g.n_slot)
        assert st == 0
        check_pack(w, r, g, p, staging, doff, n_out)


def test_error_classification(orc):
    g = orc.Group(4, 8, 1, 1)
    tk = np.array([[0, 9], [1, -2]], np.int32)
    _, st = orc.count(tk, 8)
    assert st == orc.EDATA
    load = np.ones((4, 8), np.int32)
    load[1, 2] = -1
    assert orc.plan(load, g).status == orc.EDATA
    # a load row that disagrees with the routed tokens
    load = np.ones((4, 8), np.int32)
    p = orc.plan(load, g)
    x = np.zeros((2, 8), np.uint16)
    tk = np.array([[0, 1], [2, 3]], np.int32)
    _, _, _, st = orc.dispatch(x, tk, 0, g, p)
    assert st == orc.EDATA
    # staging too small
    load = np.zeros((4, 8), np.int32)
    load[0, 0] = 100
    p = orc.plan(load, g)
    assert p.stats[4] > 0
    w = np.zeros((2, 8), np.uint16)
    _, doff, n_out, st = orc.pack(w, 0, g, p, cap=int(p.stats[4]) - 1)
    assert st == orc.ENOSPC and n_out == p.stats[4]
    # bad groups
    for bad in [orc.Group(3, 8, 1, 1), orc.Group(4, 8, -1, 1),
                orc.Group(4, 8, 1, 0), orc.Group(4, 8, 1, 1, 99, 100)]:
        assert orc.plan(np.zeros((bad.R, bad.E), np.int32), bad).status == orc.EINVAL


def test_inflight_ratio_without_locality(orc):
    """Without the local-consumption pass, uniform traffic on a balanced
    group ships a fraction (R-1)/R of the tokens off-rank: 98.4 % at R=64,
    the figure the paper quotes for its planner without locality."""
    R = 64
    g = orc.Group(R, 4 * R, 2, 1024)
    rng = np.random.default_rng(5)
    tk = rng.integers(0, g.E, (R, 4096, 8)).astype(np.int32)
    load, _ = orc.count(tk, g.E, R)
    p = orc.plan(load, g, locality=False)
    m = orc.metrics(load, g, p)
    assert abs(m["inflight_ratio"] - (1 - 1 / R)) < 2e-3
    p = orc.plan(load, g, locality=True)
    assert orc.metrics(load, g, p)["inflight_ratio"] <= m["inflight_ratio"]
