"""Packing, relay packing and gradient reduction on ranks with more than 256
source blobs, so that a workgroup numbers its expert groups over several
256-wide passes: two ranks of 512 or 300 main experts (R = 2, E = 1024 or
600), and, with relay trees, four ranks of 256 main experts plus redundant
slots (R = 4, E = 1024), with the replicated experts spread over every pass.  Byte-equal (bit-equal for the
fp32 reduction) to the oracle.  Needs an MI355X."""
import numpy as np
import pytest
import torch

import oracle
from test_oracle_relay import csr_from_slots

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    import gpu_path as gp
    from test_gpu_combine_reduce import check_reduce
    from test_gpu_relay import check_pack_relay, plan_on_device


def spread_slot_map(seed, R, E, NS):
    """Every slot holds a distinct non-local expert; half of the slots take
    local indices of 256 and above where the ranks have them, so that later
    group passes are used."""
    rng = np.random.default_rng(seed)
    nm = E // R
    X = np.full((R, NS), -1, np.int32)
    for t in range(R):
        cand = [e for e in rng.permutation(E) if e // nm != t]
        hi = [e for e in cand if e % nm >= 256]
        lo = [e for e in cand if e % nm < 256]
        n_hi = min(NS // 2, len(hi))
        pick = hi[:n_hi] + lo[: NS - n_hi]
        for s in range(NS):
            if rng.random() < 0.05:
                continue
            X[t, s] = pick[s]
    return X


def _groups_by_pass(X, rank, nm):
    """Local ids of this rank's replicated experts, split at 256."""
    loc = sorted({int(e) % nm for e in np.asarray(X).reshape(-1) if e >= 0 and e // nm == rank})
    return [l for l in loc if l < 256], [l for l in loc if l >= 256]


@pytest.mark.parametrize("seed,R,E,NS,W", [(0, 2, 1024, 128, 520), (1, 2, 1024, 64, 8),
                                           (2, 2, 600, 100, 4104)])
def test_pack_many_local_experts(seed, R, E, NS, W):
    g, og = gp.groups(R, E, NS, 1)
    p = csr_from_slots(R, E, NS, spread_slot_map(seed, R, E, NS))
    plan = plan_on_device(g, p)
    rng = np.random.default_rng(seed)
    cap = R * NS
    for rank in range(R):
        lo, hi = _groups_by_pass(p.slot_expert, rank, g.n_main)
        assert lo and hi  # groups in the first and in a later pass
        w = rng.integers(0, 1 << 16, (g.n_main, W), dtype=np.uint16)
        ostg, odoff, n_out, ost = oracle.pack(w, rank, og, p, cap)
        assert ost == oracle.OK
        stg, doff, st = gp.gpu_pack(w, rank, g, plan, cap)
        assert st == 0
        assert np.array_equal(doff, odoff), f"dest_off rank {rank}"
        assert np.array_equal(stg[:n_out], ostg[:n_out]), f"staging rank {rank}"
        assert (stg[n_out:] == 0x3C3C).all()


@pytest.mark.parametrize("seed,R,E,NS,W", [(3, 2, 1024, 128, 12), (4, 2, 600, 100, 4100)])
def test_grad_reduce_many_local_experts(seed, R, E, NS, W):
    g, og = gp.groups(R, E, NS, 1)
    p = csr_from_slots(R, E, NS, spread_slot_map(seed, R, E, NS))
    plan = plan_on_device(g, p)
    rng = np.random.default_rng(seed)
    for rank in range(R):
        assert all(_groups_by_pass(p.slot_expert, rank, g.n_main))
        assert check_reduce(g, og, plan, p.slot_expert, rank, W, rng) > 0


def relay_slot_map(seed, R, E, NS):
    """Expert 0 of rank 0 on every other rank (a relay tree at threshold 1),
    the other slots as in spread_slot_map."""
    X = spread_slot_map(seed, R, E, NS)
    nm = E // R
    for t in range(1, R):
        if 0 not in X[t]:
            X[t, 0] = 0
    # keep each row free of duplicates
    for t in range(R):
        seen = set()
        for s in range(NS):
            e = int(X[t, s])
            if e >= 0 and (e in seen or e // nm == t):
                X[t, s] = -1
            seen.add(e)
    return X


@pytest.mark.parametrize("seed,R,E,NS,W", [(8, 4, 1024, 2, 520), (6, 4, 1024, 8, 64)])
def test_pack_relay_many_sources(seed, R, E, NS, W):
    """n_main + n_slot = 258 or 264 sources: a relay's forwarded blob
    (source n_main + s) sits in the second group pass."""
    g, og = gp.groups(R, E, NS, 1)
    p = csr_from_slots(R, E, NS, relay_slot_map(seed, R, E, NS))
    plan = plan_on_device(g, p)
    rel = oracle.relay(og, p, 1)
    assert rel.stats[0] > 0
    X = np.asarray(p.slot_expert).reshape(R, NS)
    # some relay also sends one of its own mains (a first-pass group)
    both = [r for r in range(R)
            if ((X >= 0) & (rel.slot_src == r) & (X // g.n_main != r)).any()
            and ((X >= 0) & (rel.slot_src == r) & (X // g.n_main == r)).any()]
    assert both
    assert check_pack_relay(g, og, plan, p.slot_expert, rel, W, seed) > 0
