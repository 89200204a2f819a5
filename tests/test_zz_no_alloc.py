"""ultraep_plan_noalloc (the planner with the library's fixed per-device
workspace) against ultraep_plan with a caller workspace, through the C ABI:
every plan buffer byte-equal on consecutive calls, each later call on a
smaller group than the one before, so that a call finds the array holding
a larger plan's state; the oracle's plan is compared too.  Needs an MI355X."""
import numpy as np
import pytest
import torch

import gen
import oracle

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    import gpu_path as gp
    import paper_2606_04101_amd as uep


def _poisoned_plan(g):
    plan = uep.Plan(g, gp.DEV)
    for f in uep.PLAN_FIELDS:
        getattr(plan, f).fill_(-12345)
    return plan


def _largest_group_load(seed):
    """R = 64, E = 1024, four slots per rank (the largest supported group),
    Zipf-skewed routing so that the planner replicates."""
    rng = np.random.default_rng(seed)
    R, E, T, k = 64, 1024, 256, 8
    w = 1.0 / np.arange(1, E + 1) ** 1.1
    p = w[rng.permutation(E)]
    p /= p.sum()
    ids = rng.choice(E, size=(R, T * k), p=p).astype(np.int32)
    load = np.stack([np.bincount(ids[r], minlength=E) for r in range(R)]).astype(np.int32)
    return (R, E, 4, 16), load


def _workload_load(cid):
    c = gen.config(cid)
    load, _ = oracle.count(gen.topk_all(c, 0), c.E, c.R)
    return (c.R, c.E, c.n_slot, c.u_min), load


def test_noalloc_plan_equals_plan_on_calls_of_shrinking_size():
    print("no-alloc planner: largest group, DeepSeek-V3 training layer, tiny workload", flush=True)
    cases = [_largest_group_load(7), _workload_load(4), _workload_load(1)]
    sizes = []
    for (R, E, NS, u_min), load in cases:
        g, og = gp.groups(R, E, NS, u_min)
        sizes.append(uep.ultraep_plan_ws_bytes(g))
        ld = gp.dev_i32(load)
        ref = _poisoned_plan(g)
        ref.ws.copy_(torch.randint(0, 256, ref.ws.shape, dtype=torch.uint8, device=gp.DEV))
        uep.ultraep_plan(ld, g, ref)
        got = _poisoned_plan(g)
        uep.ultraep_plan_noalloc(ld, g, got)
        torch.cuda.synchronize()
        for f in uep.PLAN_FIELDS:
            gp.assert_same(f"R={R} E={E} {f}", getattr(got, f).cpu().numpy(),
                           getattr(ref, f).cpu().numpy())
        op = oracle.plan(load, og)
        assert op.status == 0
        gp.assert_plan_equal(got, op)
        assert int(got.stats[6].item()) == 0
        assert int(got.stats[4].item()) > 0  # each case replicates
    assert sizes[0] > sizes[1] > sizes[2]


def test_noalloc_plan_back_to_back_on_one_stream():
    """Two groups planned alternately without a host synchronisation in
    between: each call finds the previous call's contents in the array."""
    (a_shape, a_load), (b_shape, b_load) = _workload_load(2), _workload_load(3)
    ga, oga = gp.groups(*a_shape)
    gb, ogb = gp.groups(*b_shape)
    la, lb = gp.dev_i32(a_load), gp.dev_i32(b_load)
    pa, pb = _poisoned_plan(ga), _poisoned_plan(gb)
    for _ in range(2):
        uep.ultraep_plan_noalloc(la, ga, pa)
        uep.ultraep_plan_noalloc(lb, gb, pb)
    torch.cuda.synchronize()
    gp.assert_plan_equal(pa, oracle.plan(a_load, oga))
    gp.assert_plan_equal(pb, oracle.plan(b_load, ogb))


def test_noalloc_plan_rejects_unsupported_groups():
    g = uep.Group(3, 8, 1, 1)  # E % R != 0: no launch
    plan = uep.Plan(uep.Group(4, 8, 1, 1), gp.DEV)
    with pytest.raises(uep.UltraEPError):
        uep.ultraep_plan_noalloc(gp.dev_i32(np.zeros((3, 8), np.int32)), g, plan)
