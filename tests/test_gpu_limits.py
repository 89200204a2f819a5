"""The whole path at the limits the C ABI accepts: the largest group (R = 64,
E = 1024, R * n_slot = 256), one main expert per rank, the largest top-k
(k = 64, which takes the multi-pass combine), and the one-rank, one-expert
group.  Count, plan, dispatch, pack and combine are compared with the oracle
byte for byte.  Needs an MI355X."""
import numpy as np
import pytest
import torch

import oracle

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    import gpu_path as gp
    import paper_2606_04101_amd as uep


def _skewed_ids(rng, R, T, k, E):
    """Top-k rows without repeats, drawn with a Zipf-like skew so that the
    planner replicates several experts."""
    w = 1.0 / np.arange(1, E + 1) ** 1.1
    w = w[rng.permutation(E)]
    p = w / w.sum()
    tk = np.empty((R, T, k), np.int32)
    for r in range(R):
        for t in range(T):
            tk[r, t] = rng.choice(E, k, replace=False, p=p)
    return tk


def _combine_check(g, plan, x, tk_r, rank, rng):
    T, H = x.shape
    k = tk_r.shape[1]
    send, ros, boff, st = gp.gpu_dispatch(x, tk_r, rank, g, plan)
    assert st == 0
    gate = rng.random((T, k)).astype(np.float32)
    out = torch.empty((T, H), dtype=torch.int16, device=gp.DEV)
    stt = gp.zero_status()
    uep.ultraep_combine(gp.dev_u16(send), send.shape[0], torch.from_numpy(gate).to(gp.DEV),
                        gp.dev_i32(ros), T, k, H, out, stt)
    torch.cuda.synchronize()
    assert int(stt.item()) == 0
    oout, ost = oracle.combine(send, gate, ros)
    assert ost == 0
    assert np.array_equal(gp.host_u16(out), oout)


@pytest.mark.parametrize("R,E,NS,T,k,u_min", [
    (64, 1024, 4, 256, 8, 16),   # largest group, R * n_slot = 256
    (64, 64, 4, 300, 8, 8),      # one main expert per rank
    (16, 128, 2, 96, 64, 4),     # largest top-k
    (1, 1, 0, 5, 1, 1),          # one rank, one expert, no slots
    (2, 2, 3, 40, 2, 1),         # more slots than other experts
])
def test_limits(R, E, NS, T, k, u_min):
    rng = np.random.default_rng(R * 1000 + E + NS + k)
    g, og = gp.groups(R, E, NS, u_min)
    tk = _skewed_ids(rng, R, T, k, E)
    counts, st = gp.gpu_count(tk, E)
    ocounts, ost = oracle.count(tk, E, R)
    assert st == ost == 0
    assert np.array_equal(counts, ocounts)
    op = oracle.plan(ocounts, og)
    assert op.status == 0
    plan = gp.gpu_plan(ocounts, g)
    gp.assert_plan_equal(plan, op)
    gp.assert_plan_equal(gp.gpu_plan(ocounts, g, split=True), op)
    X = op.slot_expert.reshape(R, max(NS, 0))
    outb = [int(((X >= 0) & (X // (E // R) == r)).sum()) for r in range(R)]
    for r in sorted({0, int(np.argmax(outb)), R - 1}):
        x = rng.integers(0, 1 << 16, (T, 72)).astype(np.uint16)
        w = rng.integers(0, 1 << 16, (E // R, 40)).astype(np.uint16)
        gp.check_rank(x, tk[r], w, r, g, og, plan, op)
        _combine_check(g, plan, x, tk[r], r, rng)
