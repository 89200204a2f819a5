"""No entry point writes outside its buffers: every output, workspace and
status word sits between two guard bands of a known byte pattern, and after
each call (plans, dispatch, packing, relay trees, combine, reduction) both
bands must be intact and the outputs equal to the oracle's.  The five
workloads at full size (the tight staging capacity included) and mid-size
fuzz cases.  Needs an MI355X."""
import numpy as np
import pytest
import torch

import fuzz
import gen
import oracle

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    import gpu_path as gp
    import paper_2606_04101_amd as uep

GUARD = 4096  # bytes on each side
PAT = 0xA5


class Guarded:
    """Device buffers carved from larger byte tensors with guard bands."""

    def __init__(self):
        self.bufs = []

    def __call__(self, shape, dtype, fill=None):
        shape = (shape,) if isinstance(shape, int) else tuple(shape)
        n = int(np.prod(shape)) if shape else 1
        nbytes = n * torch.empty(0, dtype=dtype).element_size()
        full = torch.full((2 * GUARD + nbytes,), PAT, dtype=torch.uint8, device=gp.DEV)
        view = full[GUARD:GUARD + nbytes].view(dtype).view(shape)
        if fill is not None:
            view.fill_(fill)
        self.bufs.append((full, nbytes))
        return view

    def check(self, what):
        torch.cuda.synchronize()
        for i, (full, nbytes) in enumerate(self.bufs):
            lo = full[:GUARD]
            hi = full[GUARD + nbytes:]
            assert bool((lo == PAT).all()), f"{what}: buffer {i} written below its start"
            assert bool((hi == PAT).all()), f"{what}: buffer {i} written past its end"


def guarded_plan(G, g):
    plan = uep.Plan(g, gp.DEV)
    sizes = uep.ultraep_plan_sizes(g)
    for f, n in zip(uep.PLAN_FIELDS, sizes):
        dt = torch.int64 if f == "stats" else torch.int32
        setattr(plan, f, G(n, dt, fill=-7))
    plan.c = uep.PlanBuf(*[getattr(plan, f).data_ptr() if getattr(plan, f).numel() else None
                           for f in uep.PLAN_FIELDS])
    plan.ws = G(uep.ultraep_plan_ws_bytes(g), torch.uint8, fill=0x3C)
    return plan


def run_guarded(c_R, c_E, NS, u_min, beta, tk_all, x_h, rank, W, seed):
    """Every entry point on one workload with guarded buffers, the guard
    bands checked after each call and the outputs compared with the oracle."""
    g, og = gp.groups(c_R, c_E, NS, u_min, *beta)
    R, T, k = tk_all.shape
    E = c_E
    V, H = T * k, x_h.shape[1]
    G = Guarded()
    st = G(1, torch.int32, fill=0)
    counts = G((R, E), torch.int32, fill=-1)
    uep.ultraep_count(gp.dev_i32(tk_all), T, k, E, R, counts, st)
    G.check("count")
    ocnt, _ = oracle.count(tk_all, E, R)
    gp.assert_same("counts", counts.cpu().numpy(), ocnt)
    op = oracle.plan(ocnt, og)
    assert op.status == oracle.OK
    plan = guarded_plan(G, g)
    uep.ultraep_plan(counts, g, plan)
    G.check("plan")
    gp.assert_plan_equal(plan, op)
    plan2 = guarded_plan(G, g)
    uep.ultraep_plan_replicate(counts, g, plan2)
    uep.ultraep_plan_reroute(counts, g, plan2)
    G.check("plan_replicate + plan_reroute")
    gp.assert_plan_equal(plan2, op)
    plan3 = guarded_plan(G, g)
    uep.ultraep_plan_noalloc(counts, g, plan3)
    G.check("plan_noalloc")
    gp.assert_plan_equal(plan3, op)

    # dispatch
    send = G((V, H), torch.int16, fill=0x5A5A)
    ros = G(V, torch.int32, fill=-9)
    boff = G(R * g.S + 1, torch.int64, fill=-9)
    ws = G(uep.ultraep_dispatch_ws_bytes(T, k, g), torch.uint8, fill=0x77)
    xd = gp.dev_u16(x_h)
    uep.ultraep_dispatch(xd, gp.dev_i32(tk_all[rank]), T, k, H, rank, g, plan, send, ros, boff,
                         ws, st)
    G.check("dispatch")
    osend, oros, oboff, ost = oracle.dispatch(x_h, tk_all[rank], rank, og, op)
    assert ost == 0 and int(st.item()) == 0
    gp.assert_same("row_of_slot", ros.cpu().numpy(), oros)
    gp.assert_same("block_off", boff.cpu().numpy(), oboff)
    gp.assert_same("send", gp.host_u16(send), osend)

    # packing with the exact capacity (staging ends where the last entry ends)
    rng = np.random.default_rng(seed)
    w_h = rng.integers(0, 1 << 16, (g.n_main, W), dtype=np.uint16)
    ostg, odoff, n_out, ost = oracle.pack(w_h, rank, og, op, R * NS)
    assert ost == 0
    cap = max(n_out, 1)
    stg = G((cap, W), torch.int16, fill=0x3C3C)
    doff = G(R + 1, torch.int64, fill=-9)
    wd = gp.dev_u16(w_h)
    uep.ultraep_pack_replicas(wd, W, rank, g, plan, stg, cap, doff, st)
    G.check("pack")
    gp.assert_same("staging", gp.host_u16(stg)[:n_out], ostg[:n_out])
    gp.assert_same("dest_off", doff.cpu().numpy(), odoff)
    stg2 = G((cap, W), torch.int16, fill=0x3C3C)
    doff2 = G(R + 1, torch.int64, fill=-9)
    uep.ultraep_reroute_and_pack(counts, g, plan2, wd, W, rank, stg2, cap, doff2, st)
    G.check("reroute_and_pack")
    gp.assert_same("staging (reroute_and_pack)", gp.host_u16(stg2)[:n_out], ostg[:n_out])
    gp.assert_plan_equal(plan2, op)
    if n_out > 1:  # one entry too few: ENOSPC and nothing written past the buffer
        st_small = G(1, torch.int32, fill=0)
        stg3 = G((n_out - 1, W), torch.int16, fill=0x3C3C)
        uep.ultraep_pack_replicas(wd, W, rank, g, plan, stg3, n_out - 1,
                                  G(R + 1, torch.int64), st_small)
        G.check("pack, capacity one short")
        assert int(st_small.item()) == uep.ULTRAEP_ENOSPC
    assert int(st.item()) == 0

    # relay trees and the packing under them
    src = G(max(R * NS, 1), torch.int32, fill=-9)
    vol = G(R, torch.int32, fill=-9)
    rst = G(4, torch.int64, fill=-9)
    uep.ultraep_relay_plan(g, plan, 1, src, vol, rst, st)
    G.check("relay_plan")
    rel = oracle.relay(og, op, 1)
    gp.assert_same("slot_src", src.cpu().numpy()[:R * NS], rel.slot_src.reshape(-1))
    rs_h = rng.integers(0, 1 << 16, (max(NS, 1), W), dtype=np.uint16)
    ostg_r, odoff_r, n_r, ost = oracle.pack_relay(w_h, rs_h, rank, og, op.slot_expert,
                                                  rel.slot_src, R * NS)
    assert ost == 0
    stg4 = G((max(n_r, 1), W), torch.int16, fill=0x3C3C)
    uep.ultraep_pack_relay(wd, gp.dev_u16(rs_h), W, rank, g, plan, src, stg4, max(n_r, 1),
                           G(R + 1, torch.int64), st)
    G.check("pack_relay")
    gp.assert_same("staging (relay)", gp.host_u16(stg4)[:n_r], ostg_r[:n_r])

    # combine over the send rows, gradient reduction over the staging layout
    gate_h = rng.random((T, k)).astype(np.float32)
    out = G((T, H), torch.int16, fill=0x1111)
    uep.ultraep_combine(send, V, torch.from_numpy(gate_h).to(gp.DEV), ros, T, k, H, out, st)
    G.check("combine")
    oout, _ = oracle.combine(osend, gate_h, oros)
    gp.assert_same("combine out", gp.host_u16(out), oout)
    Wf = W // 2
    main_h = rng.standard_normal((g.n_main, Wf)).astype(np.float32)
    rg_h = rng.standard_normal((max(n_out, 1), Wf)).astype(np.float32)
    mg = G((g.n_main, Wf), torch.float32)
    mg.copy_(torch.from_numpy(main_h))
    rg = G((max(n_out, 1), Wf), torch.float32)
    rg.copy_(torch.from_numpy(rg_h))
    uep.ultraep_grad_reduce(mg, rg, Wf, rank, g, plan, max(n_out, 1), st)
    G.check("grad_reduce")
    omg, org, on, ost = oracle.grad_reduce(main_h, rg_h[:n_out], rank, og, op.slot_expert,
                                           max(n_out, 1))
    assert ost == 0 and on == n_out
    assert np.array_equal(mg.cpu().numpy().view(np.uint32), omg.view(np.uint32))
    assert int(st.item()) == 0


def _rstar(op, n_main):
    X = op.slot_expert
    return int(np.argmax([((X >= 0) & (X // n_main == r)).sum() for r in range(X.shape[0])]))


@pytest.mark.parametrize("cid,m", [(1, 0), (2, 0), (3, 4), (4, 0), (5, 0)])
def test_guard_bands_workloads(cid, m):
    print(f"guard bands: workload {cid} instance {m}", flush=True)
    c = gen.config(cid)
    tk = gen.topk_all(c, m)
    load, _ = oracle.count(tk, c.E, c.R)
    op = oracle.plan(load, oracle.Group(c.R, c.E, c.n_slot, c.u_min, c.beta_num, c.beta_den))
    rank = _rstar(op, c.n_main)
    x_h = gen.activations(c, m, rank)
    run_guarded(c.R, c.E, c.n_slot, c.u_min, (c.beta_num, c.beta_den), tk, x_h, rank,
                8 * 1000 + 8, cid)


# fuzz cases whose plans replicate (hot, duplicate, Zipf, masked, two-hot and
# balanced routing; 2 to 8 ranks, 1 to 3 slots)
@pytest.mark.parametrize("seed", [7, 13, 17, 22, 73, 100, 107, 119, 149, 151])
def test_guard_bands_fuzz(seed):
    case = fuzz.make_case(seed)
    tk = case["topk"]
    print(f"guard bands: fuzz case {seed}", flush=True)
    R, E, NS = case["R"], case["E"], case["n_slot"]
    load, _ = oracle.count(tk, E, R)
    op = oracle.plan(load, oracle.Group(R, E, NS, case["u_min"], case["beta_num"],
                                        case["beta_den"]))
    rank = _rstar(op, E // R)
    rng = np.random.default_rng(seed)
    x_h = rng.integers(0, 1 << 16, (tk.shape[1], 24), dtype=np.uint16)
    run_guarded(R, E, NS, case["u_min"], (case["beta_num"], case["beta_den"]), tk, x_h, rank,
                40, seed)
