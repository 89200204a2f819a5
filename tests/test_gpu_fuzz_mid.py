"""Parity on the mid-size corpus of tests/fuzz.py (make_mid_case): groups of
up to 64 ranks (not only powers of two) and 1024 experts, top-k up to 64,
blocks above 32768 ids, rows above 8192 elements, ragged blob widths and
u_min from 1 up to the mean expert load.  Count, both planner entry points,
dispatch, pack and combine on three ranks, the relay trees and the gradient
reduction are compared with the oracle byte for byte.  Needs an MI355X."""
import numpy as np
import pytest
import torch

import fuzz
import oracle
from test_gpu_combine_reduce import bf16_normals, check_combine, check_reduce, softmax_gates
from test_gpu_relay import check as check_relay

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    import gpu_path as gp


@pytest.mark.parametrize("seed", range(48))
def test_mid_parity(seed):
    c = fuzz.make_mid_case(seed)
    print(f"mid case {seed}: {c['pattern']} R={c['R']} E={c['E']} NS={c['n_slot']} "
          f"k={c['k']} T={c['T']} H={c['H']} W={c['W']} u_min={c['u_min']}", flush=True)
    g, og = gp.groups(c["R"], c["E"], c["n_slot"], c["u_min"], c["beta_num"], c["beta_den"])
    tk = c["topk"]
    T, k = c["T"], c["k"]
    if T > 0:
        counts, st = gp.gpu_count(tk, g.E)
        ocounts, ost = oracle.count(tk, g.E, g.R)
        assert st == ost == 0
        assert np.array_equal(counts, ocounts)
    else:
        ocounts = np.zeros((g.R, g.E), np.int32)
    op = oracle.plan(ocounts, og)
    assert op.status == 0
    plan = gp.gpu_plan(ocounts, g)
    gp.assert_plan_equal(plan, op)
    gp.assert_plan_equal(gp.gpu_plan(ocounts, g, split=True), op)
    rng = c["rng"]
    X = op.slot_expert.reshape(g.R, max(g.n_slot, 0))
    outb = [int(((X >= 0) & (X // g.n_main == r)).sum()) for r in range(g.R)]
    for r in sorted({0, int(np.argmax(outb)), g.R - 1}):
        x = bf16_normals(rng, (T, c["H"]))
        w = rng.integers(0, 1 << 16, (g.n_main, c["W"])).astype(np.uint16)
        gp.check_rank(x, tk[r], w, r, g, og, plan, op, split=bool(seed % 2))
        if T > 0:
            send, ros, _, st = gp.gpu_dispatch(x, tk[r], r, g, plan)
            assert st == 0
            check_combine(send, softmax_gates(rng, T, k), ros)
        check_reduce(g, og, plan, op.slot_expert, r, 8 * int(rng.integers(1, 600)), rng)
    for threshold in (0, 2):
        check_relay(g, og, plan, op, threshold)
