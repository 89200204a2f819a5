"""A wide randomized sweep of the whole path on small rows: 1000 seeded
groups (1 to 64 ranks, up to 1024 experts, 0 to 4 redundant slots per rank)
and routings (distinct top-k per token from uniform, Zipf-skewed or hot-rank
expert popularity, a quarter of the slots masked, or ids with repeats), from
0 to 2500 tokens per rank and top-1 to top-8.  The counts, every plan buffer,
and for two ranks the dispatch (send, row_of_slot, block_off, through both
the one-call and the split entry points) and the packing (staging, dest_off)
are compared with the oracle byte for byte; a second sweep covers the
relay trees, the relay packing, the combine gather and the gradient
reduction.  Needs an MI355X."""
import numpy as np
import pytest
import torch

import oracle

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    import gpu_path as gp


def sweep_routing(seed):
    rng = np.random.default_rng(70_000 + seed)
    R = int(rng.choice([1, 2, 3, 4, 7, 8, 16, 24, 32, 64]))
    nm = int(rng.choice([1, 2, 3, 4, 8, 16]))
    nm = min(nm, 1024 // R)
    E = R * nm
    NS = min(int(rng.integers(0, 5)), 256 // R)
    k = int(min(rng.choice([1, 2, 4, 6, 8]), E))
    T = int(rng.choice([0, 1, 37, 500, 1024, 2500]))
    u_min = int(rng.choice([1, 4, 16, 64]))
    kind = int(rng.integers(0, 5))
    if kind == 0:
        p = np.full(E, 1.0 / E)
    elif kind == 1:  # Zipf-skewed expert popularity
        p = 1.0 / np.arange(1, E + 1) ** rng.uniform(0.5, 1.5)
        rng.shuffle(p)
        p /= p.sum()
    else:  # the experts of a few ranks are hot
        p = np.ones(E)
        for h in rng.choice(R, max(1, R // 4), replace=False):
            p[h * nm:(h + 1) * nm] *= rng.uniform(5, 40)
        p /= p.sum()
    tk = rng.choice(E, (R, T, k), p=p).astype(np.int32)
    if kind != 4:  # distinct experts per token: redraw repeats (kind 4 keeps them)
        for j in range(1, k):
            for _ in range(64):
                dup = (tk[:, :, j:j + 1] == tk[:, :, :j]).any(axis=2)
                if not dup.any():
                    break
                tk[:, :, j][dup] = rng.choice(E, int(dup.sum()), p=p)
    if kind == 3:
        tk[rng.random(tk.shape) < 0.25] = -1
    H = 8 * int(rng.integers(1, 25))
    W = 8 * int(rng.integers(1, 65))
    return rng, tk, R, E, NS, k, T, u_min, H, W


@pytest.mark.parametrize("block", range(4))
def test_dispatch_sweep(block):
    checked = 0
    for seed in range(block * 250, (block + 1) * 250):
        rng, tk, R, E, NS, k, T, u_min, H, W = sweep_routing(seed)
        where = f"seed {seed} (R={R} E={E} n_slot={NS} k={k} T={T} u_min={u_min} H={H} W={W})"
        g, og = gp.groups(R, E, NS, u_min)
        try:
            load, ost = oracle.count(tk, E, R)
            assert ost == 0
            if T > 0:
                counts, st = gp.gpu_count(tk, E)
                assert st == 0
                gp.assert_same("counts", counts, load)
            op = oracle.plan(load, og)
            if op.status != oracle.OK:
                continue
            plan = gp.gpu_plan(load, g)
            gp.assert_plan_equal(plan, op)
            X = op.slot_expert.reshape(R, max(NS, 0))
            outb = [int(((X >= 0) & (X // (E // R) == r)).sum()) for r in range(R)]
            for i, r in enumerate(sorted({int(np.argmax(outb)), int(rng.integers(0, R))})):
                x = rng.integers(0, 1 << 16, (T, H)).astype(np.uint16)
                w = rng.integers(0, 1 << 16, (E // R, W)).astype(np.uint16)
                gp.check_rank(x, tk[r], w, r, g, og, plan, op, split=bool((seed + i) % 2))
        except AssertionError as ex:
            raise AssertionError(f"{where}: {ex}") from None
        checked += 1
    assert checked > 200


@pytest.mark.parametrize("block", range(2))
def test_extension_sweep(block):
    """The adjacent steps on the same routings: relay trees at thresholds 0
    and 2 and the relay packing of two ranks, the combine gather of one
    rank's dispatched rows with softmax gates, and the gradient reduction of
    two ranks, against the oracle."""
    from test_gpu_combine_reduce import bf16_normals, check_combine, check_reduce, softmax_gates
    from test_gpu_relay import check as check_relay
    from test_gpu_relay import check_pack_relay
    checked = 0
    for seed in range(1000 + block * 150, 1000 + (block + 1) * 150):
        rng, tk, R, E, NS, k, T, u_min, H, W = sweep_routing(seed)
        where = f"seed {seed} (R={R} E={E} n_slot={NS} k={k} T={T} u_min={u_min} H={H} W={W})"
        g, og = gp.groups(R, E, NS, u_min)
        try:
            load, _ = oracle.count(tk, E, R)
            op = oracle.plan(load, og)
            if op.status != oracle.OK:
                continue
            plan = gp.gpu_plan(load, g)
            gp.assert_plan_equal(plan, op)
            X = op.slot_expert.reshape(R, max(NS, 0))
            outb = [int(((X >= 0) & (X // (E // R) == r)).sum()) for r in range(R)]
            ranks = sorted({int(np.argmax(outb)), int(rng.integers(0, R))})
            for threshold in (0, 2):
                rel = check_relay(g, og, plan, op, threshold)
                check_pack_relay(g, og, plan, op.slot_expert, rel, W, seed, ranks=ranks)
            r = ranks[-1]
            if T > 0:
                send, ros, _, st = gp.gpu_dispatch(bf16_normals(rng, (T, H)), tk[r], r, g, plan)
                assert st == 0
                check_combine(send, softmax_gates(rng, T, k), ros)
            for r in ranks:
                check_reduce(g, og, plan, op.slot_expert, r, 4 * int(rng.integers(1, 200)), rng)
        except AssertionError as ex:
            raise AssertionError(f"{where}: {ex}") from None
        checked += 1
    assert checked > 120
