"""The HIP planner, dispatch and packing on the hand-worked examples of
tests/golden/, compared with the values derived there by hand (not with the
oracle's output): tau*, the bisection's bounds and probe count, X, U, the
host lists and Q, and for W4 the dispatch layout and the packing order.
Needs an MI355X."""
import json
import os

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    import gpu_path as gp
    import paper_2606_04101_amd as uep

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


@pytest.mark.parametrize("name", ["W0_single_hot_expert.json", "W1_nonmonotone_bisection.json",
                                  "W2_proportional_split.json", "W4_two_slots_dispatch_pack.json",
                                  "W5_visit_order.json", "W7_source_order.json"])
@pytest.mark.parametrize("split", [False, True])
def test_plan_matches_hand_derivation(name, split):
    d = _load(name)
    grp = d["group"]
    g, _ = gp.groups(grp["R"], grp["E"], grp["n_slot"], grp["u_min"], grp["beta_num"],
                     grp["beta_den"])
    load = np.array(d["load"], np.int32)
    plan = gp.gpu_plan(load, g, split=split)
    stats = plan.stats.cpu().numpy()
    assert stats[6] == 0
    assert stats[0] == d["tau_star"]
    assert stats[3] == len(d["trace"])
    if "tau_lo0" in d:
        assert (stats[1], stats[2]) == (d["tau_lo0"], d["tau_hi0"])
    R, E = grp["R"], grp["E"]
    assert plan.slot_expert.cpu().numpy().reshape(R, grp["n_slot"]).tolist() == d["slot_expert"]
    U = plan.quota.cpu().numpy().reshape(E, R)
    if "quota" in d:
        assert U.tolist() == d["quota"]
    if "quota_nonzero" in d:
        exp = np.zeros_like(U)
        for key, v in d["quota_nonzero"].items():
            e, t = map(int, key.split(","))
            exp[e, t] = v
        assert np.array_equal(U, exp)
    csr = d.get("reroute_csr", d)
    for f in ("host_ptr", "host_rank", "host_pslot"):
        if f in csr:
            assert getattr(plan, f).cpu().numpy().tolist() == csr[f], f
    if "reroute" in d:
        ncol = E + R * grp["n_slot"]
        assert plan.reroute.cpu().numpy().reshape(R, ncol).tolist() == d["reroute"]


def test_w4_dispatch_and_pack_match_hand_derivation():
    d = _load("W4_two_slots_dispatch_pack.json")
    grp = d["group"]
    g, _ = gp.groups(grp["R"], grp["E"], grp["n_slot"], grp["u_min"], grp["beta_num"],
                     grp["beta_den"])
    plan = gp.gpu_plan(np.array(d["load"], np.int32), g)
    topk = np.array(d["topk"], np.int32)
    T, k = topk.shape
    x = (np.arange(T)[:, None] * 100 + np.arange(8)[None, :]).astype(np.uint16)
    send, ros, boff, st = gp.gpu_dispatch(x, topk, d["dispatch_rank"], g, plan)
    assert st == 0
    assert boff.tolist() == d["block_off"]
    assert ros.tolist() == d["row_of_slot"]
    nv = int(boff[-1])
    assert [int(r[0]) // 100 for r in send[:nv]] == d["send_token_of_row"][:nv]
    n_main = grp["E"] // grp["R"]
    w = (np.arange(n_main)[:, None] * 1000 + np.arange(8)[None, :]).astype(np.uint16)
    stg, doff, st = gp.gpu_pack(w, d["pack_rank"], g, plan, 4)
    assert st == 0
    assert doff.tolist() == d["dest_off"]
    n_out = len(d["pack_experts"])
    # pack_experts: the main-expert index (row of w_main) each entry copies
    assert [int(r[0]) // 1000 for r in stg[:n_out]] == d["pack_experts"]
