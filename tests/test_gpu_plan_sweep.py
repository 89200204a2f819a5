"""A wide randomized sweep of the planner: 2000 seeded groups and load
matrices (2 to 64 ranks, up to 1024 experts, 0 to 4 redundant slots per
rank, u_min from 1 to 256, four beta values; uniform, Zipf-skewed, hot-rank,
one-hot-expert and sparse loads at three scales), every plan buffer of
ultraep_plan and of the split entry points against the oracle.  Needs an
MI355X (about 3 s)."""
import numpy as np
import pytest
import torch

import oracle

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    import gpu_path as gp


def sweep_case(seed):
    rng = np.random.default_rng(90_000 + seed)
    R = int(rng.choice([2, 3, 5, 8, 13, 16, 31, 32, 48, 64]))
    nm = int(rng.choice([1, 2, 3, 4, 8, 16]))
    nm = min(nm, 1024 // R)
    E = R * nm
    NS = min(int(rng.integers(0, 5)), 256 // R)
    u_min = int(rng.choice([1, 4, 16, 64, 256]))
    beta = [(101, 100), (100, 100), (11, 10), (3, 2)][int(rng.integers(0, 4))]
    kind = int(rng.integers(0, 5))
    scale = int(rng.choice([100, 1000, 30000]))
    if kind == 0:
        load = rng.integers(0, scale, (R, E))
    elif kind == 1:  # Zipf-skewed experts
        w = 1.0 / np.arange(1, E + 1) ** rng.uniform(0.5, 1.6)
        rng.shuffle(w)
        load = rng.poisson(scale * E * w / w.sum(), (R, E))
    elif kind == 2:  # a quarter of the ranks hot on every expert
        load = rng.integers(0, scale // 10 + 1, (R, E))
        for h in rng.choice(R, max(1, R // 4), replace=False):
            load[:, h * nm:(h + 1) * nm] += rng.integers(scale // 2, scale, (R, nm))
    elif kind == 3:  # one hot expert
        load = rng.integers(0, scale // 20 + 1, (R, E))
        load[:, int(rng.integers(0, E))] += rng.integers(scale, 4 * scale, R)
    else:  # sparse
        load = rng.integers(0, scale, (R, E)) * (rng.random((R, E)) < 0.2)
    return load.astype(np.int32), R, E, NS, u_min, beta


@pytest.mark.parametrize("block", range(4))
def test_plan_sweep(block):
    checked = 0
    for seed in range(block * 500, (block + 1) * 500):
        load, R, E, NS, u_min, beta = sweep_case(seed)
        g, og = gp.groups(R, E, NS, u_min, *beta)
        op = oracle.plan(load, og)
        if op.status != oracle.OK:
            continue
        try:
            gp.assert_plan_equal(gp.gpu_plan(load, g), op)
            gp.assert_plan_equal(gp.gpu_plan(load, g, split=True), op)
        except AssertionError as ex:
            raise AssertionError(f"seed {seed} (R={R} E={E} n_slot={NS} u_min={u_min} "
                                 f"beta={beta}): {ex}") from None
        checked += 1
    assert checked > 450
