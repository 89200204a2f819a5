"""Parity of the relay-tree entry points (Sec. 6.2) with the oracle, element
by element: ultraep_relay_plan on plans of the five workloads, the fuzz
corpus and dense random slot maps with many hot experts, and
ultraep_pack_relay on every rank of trees that do relay.  Needs an MI355X."""
import numpy as np
import pytest
import torch

import fuzz
import gen
import oracle
from test_oracle_relay import csr_from_slots

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    import gpu_path as gp
    import paper_2606_04101_amd as uep


def gpu_relay(g, plan, threshold):
    R, NS = g.R, g.n_slot
    src = torch.full((max(R * NS, 1),), -9, dtype=torch.int32, device=gp.DEV)
    vol = torch.full((R,), -9, dtype=torch.int32, device=gp.DEV)
    stats = torch.full((4,), -9, dtype=torch.int64, device=gp.DEV)
    st = gp.zero_status()
    uep.ultraep_relay_plan(g, plan, threshold, src, vol, stats, st)
    torch.cuda.synchronize()
    return (src.cpu().numpy()[:R * NS].reshape(R, NS), vol.cpu().numpy(),
            stats.cpu().numpy(), int(st.item()))


def plan_on_device(g, p, stats6=0):
    """A uep.Plan holding the slot map and host lists of p (a plan object
    with numpy fields), stats zero apart from stats[6]."""
    plan = uep.Plan(g, gp.DEV)
    plan.slot_expert.copy_(torch.from_numpy(np.ascontiguousarray(p.slot_expert, np.int32).reshape(-1)))
    plan.host_ptr.copy_(torch.from_numpy(np.ascontiguousarray(p.host_ptr, np.int32)))
    plan.host_rank.copy_(torch.from_numpy(np.ascontiguousarray(p.host_rank, np.int32)))
    plan.host_pslot.copy_(torch.from_numpy(np.ascontiguousarray(p.host_pslot, np.int32)))
    plan.stats.zero_()
    plan.stats[6] = stats6
    return plan


def check(g, og, plan, op, threshold):
    o = oracle.relay(og, op, threshold)
    assert o.status == oracle.OK
    src, vol, stats, st = gpu_relay(g, plan, threshold)
    assert st == 0
    assert np.array_equal(src, o.slot_src), "slot_src"
    assert np.array_equal(vol, o.send_vol), "send_vol"
    assert np.array_equal(stats, o.stats), "relay_stats"
    return o


@pytest.mark.parametrize("cid,m", [(1, 0), (2, 0), (3, 0), (3, 9), (4, 0), (4, 1), (5, 0), (5, 31)])
@pytest.mark.parametrize("threshold", [0, 1, 2, 4])
def test_relay_workloads(cid, m, threshold):
    c = gen.config(cid)
    g, og = gp.groups(c.R, c.E, c.n_slot, c.u_min, c.beta_num, c.beta_den)
    load, _ = oracle.count(gen.topk_all(c, m), c.E, c.R)
    op = oracle.plan(load, og)
    plan = gp.gpu_plan(load, g)
    gp.assert_plan_equal(plan, op)
    check(g, og, plan, op, threshold)


@pytest.mark.parametrize("seed", range(0, 160, 3))
def test_relay_fuzz(seed):
    case = fuzz.make_case(seed)
    g, og = gp.groups(case["R"], case["E"], case["n_slot"], case["u_min"],
                      case["beta_num"], case["beta_den"])
    tk = case["topk"]
    load = oracle.count(tk, g.E, g.R)[0] if tk.shape[1] > 0 else np.zeros((g.R, g.E), np.int32)
    op = oracle.plan(load, og)
    plan = gp.gpu_plan(load, g)
    for thr in (0, 1, 4):
        check(g, og, plan, op, thr)


def dense_slot_map(seed, R, E, NS, n_hot):
    """Random slot map in which n_hot experts fill most slots: fan-outs up to
    R - 1, several hot experts per home rank, some empty slots."""
    rng = np.random.default_rng(seed)
    nm = E // R
    hot = rng.choice(E, n_hot, replace=False)
    X = np.full((R, NS), -1, np.int32)
    for t in range(R):
        cand = [e for e in rng.permutation(hot) if e // nm != t]
        cand += [e for e in rng.permutation(E) if e // nm != t and e not in cand]
        k = 0
        for s in range(NS):
            if rng.random() < 0.1:
                continue
            X[t, s] = cand[k]
            k += 1
    return X


@pytest.mark.parametrize("seed,R,E,NS,n_hot", [(0, 64, 64, 4, 5), (1, 64, 256, 4, 12),
                                               (2, 32, 128, 8, 6), (3, 64, 64, 1, 2),
                                               (4, 16, 1024, 16, 30), (5, 64, 128, 4, 40)])
@pytest.mark.parametrize("threshold", [0, 4, 9])
def test_relay_dense_slot_maps(seed, R, E, NS, n_hot, threshold):
    g, og = gp.groups(R, E, NS, 1)
    p = csr_from_slots(R, E, NS, dense_slot_map(seed, R, E, NS, n_hot))
    plan = plan_on_device(g, p)
    o = check(g, og, plan, p, threshold)
    if threshold == 4 and n_hot <= 12:
        assert o.stats[0] > 0  # the case does build relay trees


def test_relay_hand_cases():
    """The hand-derived oracle pins, through the library."""
    R, E, NS = 8, 8, 2
    X = np.full((R, NS), -1, np.int32)
    X[1:8, 0] = 0
    X[2:5, 1] = 1
    X[5, 1] = 2
    g, og = gp.groups(R, E, NS, 1)
    p = csr_from_slots(R, E, NS, X)
    src, vol, stats, st = gpu_relay(g, plan_on_device(g, p), 4)
    assert st == 0
    assert src[:, 0].tolist() == [-1, 3, 4, 0, 0, 0, 5, 3]
    assert vol.tolist() == [3, 3, 1, 2, 1, 1, 0, 0]
    assert stats.tolist() == [1, 3, 7, 3]
    X = np.full((10, 1), -1, np.int32)
    X[1:, 0] = 0
    g, og = gp.groups(10, 10, 1, 1)
    p = csr_from_slots(10, 10, 1, X)
    src, vol, stats, st = gpu_relay(g, plan_on_device(g, p), 4)
    assert st == 0 and src[:, 0].tolist() == [-1, 0, 0, 0, 1, 2, 3, 1, 2, 3]


def test_relay_flags_inconsistent_plans():
    X = np.full((10, 1), -1, np.int32)
    X[1:, 0] = 0
    g, og = gp.groups(10, 10, 1, 1)
    p = csr_from_slots(10, 10, 1, X)
    # the planner's own status
    assert gpu_relay(g, plan_on_device(g, p, stats6=uep.ULTRAEP_EDATA), 4)[3] == uep.ULTRAEP_EDATA
    # host list not in ascending rank order
    p.host_rank = p.host_rank.copy()
    p.host_rank[3], p.host_rank[4] = p.host_rank[4], p.host_rank[3]
    assert gpu_relay(g, plan_on_device(g, p), 4)[3] == uep.ULTRAEP_EDATA
    # a replica entry whose slot holds another expert
    p = csr_from_slots(10, 10, 1, X)
    p.slot_expert = p.slot_expert.copy()
    p.slot_expert[5, 0] = 3
    assert gpu_relay(g, plan_on_device(g, p), 4)[3] == uep.ULTRAEP_EDATA


def gpu_pack_relay(w, relay_src, rank, g, plan, slot_src, cap):
    n_main, W = w.shape
    st = gp.zero_status()
    staging = torch.full((max(cap, 1), W), 0x3C3C, dtype=torch.int16, device=gp.DEV)
    doff = torch.full((g.R + 1,), -9, dtype=torch.int64, device=gp.DEV)
    src = torch.from_numpy(np.ascontiguousarray(slot_src, np.int32).reshape(-1)).to(gp.DEV)
    uep.ultraep_pack_relay(gp.dev_u16(w), gp.dev_u16(relay_src), W, rank, g, plan, src,
                           staging, cap, doff, st)
    torch.cuda.synchronize()
    return gp.host_u16(staging), doff.cpu().numpy(), int(st.item())


def check_pack_relay(g, og, plan, X, rel, W, seed, ranks=None):
    rng = np.random.default_rng(seed)
    cap = g.R * g.n_slot
    n_relaying = 0
    for rank in (ranks if ranks is not None else range(g.R)):
        w = rng.integers(0, 1 << 16, (g.n_main, W), dtype=np.uint16)
        rs = rng.integers(0, 1 << 16, (max(g.n_slot, 1), W), dtype=np.uint16)
        ostg, odoff, n_out, ost = oracle.pack_relay(w, rs, rank, og, X, rel.slot_src, cap)
        assert ost == oracle.OK
        stg, doff, st = gpu_pack_relay(w, rs, rank, g, plan, rel.slot_src, cap)
        assert st == 0
        assert np.array_equal(doff, odoff), f"dest_off rank {rank}"
        assert np.array_equal(stg[:n_out], ostg[:n_out]), f"staging rank {rank}"
        assert (stg[n_out:cap] == 0x3C3C).all()
        Xr = np.asarray(X).reshape(g.R, g.n_slot)
        n_relaying += int(((Xr >= 0) & (rel.slot_src == rank) & (Xr // g.n_main != rank)).sum() > 0)
    return n_relaying


@pytest.mark.parametrize("seed,R,E,NS,n_hot,W", [(0, 64, 64, 4, 5, 4104), (1, 64, 256, 4, 12, 1 << 16),
                                                 (2, 32, 128, 8, 6, 8), (4, 16, 1024, 16, 30, 512)])
def test_pack_relay_dense_slot_maps(seed, R, E, NS, n_hot, W):
    g, og = gp.groups(R, E, NS, 1)
    p = csr_from_slots(R, E, NS, dense_slot_map(seed, R, E, NS, n_hot))
    plan = plan_on_device(g, p)
    rel = oracle.relay(og, p, 4)
    assert rel.stats[0] > 0
    assert check_pack_relay(g, og, plan, p.slot_expert, rel, W, seed) > 0


@pytest.mark.parametrize("cid,threshold", [(3, 4), (3, 1), (4, 1), (5, 4)])
def test_pack_relay_workloads(cid, threshold):
    """Trees of the workloads' plans (each of these relays at least one
    expert), every rank, blobs of 8 * 512 elements."""
    c = gen.config(cid)
    g, og = gp.groups(c.R, c.E, c.n_slot, c.u_min, c.beta_num, c.beta_den)
    load, _ = oracle.count(gen.topk_all(c, 0), c.E, c.R)
    op = oracle.plan(load, og)
    plan = gp.gpu_plan(load, g)
    rel = oracle.relay(og, op, threshold)
    assert rel.stats[0] > 0
    assert check_pack_relay(g, og, plan, op.slot_expert, rel, 8 * 512, cid) > 0


def test_pack_relay_flags_orphan_relay():
    """A slot whose sender is a rank that holds no copy of its expert."""
    X = np.full((10, 1), -1, np.int32)
    X[1:9, 0] = 0  # expert 0 on ranks 1..8; rank 9 holds nothing
    g, og = gp.groups(10, 10, 1, 1)
    plan = plan_on_device(g, csr_from_slots(10, 10, 1, X))
    src = np.full((10, 1), -1, np.int32)
    src[1:9, 0] = 0
    src[8, 0] = 9
    w = np.zeros((1, 64), np.uint16)
    rs = np.zeros((1, 64), np.uint16)
    assert gpu_pack_relay(w, rs, 9, g, plan, src, 9)[2] == uep.ULTRAEP_EDATA
