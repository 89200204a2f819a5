"""Helpers that run the HIP library on device tensors and compare its outputs
with the oracle's, buffer by buffer (test infrastructure)."""
from __future__ import annotations

import numpy as np
import torch

import oracle
import paper_2606_04101_amd as uep

DEV = torch.device("cuda:0")


def groups(R, E, n_slot, u_min, beta_num=101, beta_den=100):
    return (uep.Group(R, E, n_slot, u_min, beta_num, beta_den),
            oracle.Group(R, E, n_slot, u_min, beta_num, beta_den))


def dev_i32(a):
    return torch.from_numpy(np.ascontiguousarray(a, np.int32)).to(DEV)


def dev_u16(a):
    return torch.from_numpy(np.ascontiguousarray(a, np.uint16).view(np.int16)).to(DEV)


def host_u16(t):
    return t.cpu().numpy().view(np.uint16)


def zero_status():
    return torch.zeros(1, dtype=torch.int32, device=DEV)


def gpu_count(topk_all, E):
    n_groups, T, k = topk_all.shape
    st = zero_status()
    counts = torch.full((n_groups, E), -7, dtype=torch.int32, device=DEV)
    uep.ultraep_count(dev_i32(topk_all), T, k, E, n_groups, counts, st)
    torch.cuda.synchronize()
    return counts.cpu().numpy(), int(st.item())


def gpu_plan(load, g, split=False):
    """split: SolveReplication and SolveReroute through their own entry points
    instead of ultraep_plan."""
    plan = uep.Plan(g, DEV)
    for f in uep.PLAN_FIELDS:  # poison: every element must be written
        getattr(plan, f).fill_(-12345)
    # the workspace's contents on entry must not matter
    plan.ws.copy_(torch.randint(0, 256, plan.ws.shape, dtype=torch.uint8, device=DEV))
    ld = dev_i32(load)
    if split:
        uep.ultraep_plan_replicate(ld, g, plan)
        uep.ultraep_plan_reroute(ld, g, plan)
    else:
        uep.ultraep_plan(ld, g, plan)
    torch.cuda.synchronize()
    return plan


def assert_same(name, gpu, orc, limit=6):
    """Raises unless the two arrays are equal, naming the number of differing
    elements and the first ones by index, with the GPU and oracle values."""
    gpu, orc = np.asarray(gpu), np.asarray(orc)
    if gpu.shape != orc.shape:
        raise AssertionError(f"{name}: shape {gpu.shape} against the oracle's {orc.shape}")
    if np.array_equal(gpu, orc):
        return
    bad = np.argwhere(gpu != orc)
    first = [(tuple(int(v) for v in ix), gpu[tuple(ix)].item(), orc[tuple(ix)].item())
             for ix in bad[:limit]]
    rows = np.unique(bad[:, 0]) if gpu.ndim > 1 else None
    more = f" in {rows.size} rows (first rows {rows[:8].tolist()})" if rows is not None else ""
    raise AssertionError(f"{name}: {len(bad)} of {gpu.size} elements differ{more}; "
                         f"first (index, gpu, oracle): {first}")


def assert_plan_equal(plan, op):
    for f in uep.PLAN_FIELDS:
        a = getattr(plan, f).cpu().numpy().reshape(-1)
        b = getattr(op, f).reshape(-1)
        if not np.array_equal(a, b):
            bad = np.nonzero(a != b)[0][:8]
            raise AssertionError(f"plan field {f} differs at {bad.tolist()}: "
                                 f"gpu {a[bad].tolist()} oracle {b[bad].tolist()}")


def gpu_dispatch(x, topk, rank, g, plan, split=False):
    T, H = x.shape
    k = topk.shape[1]
    V = T * k
    st = zero_status()
    send = torch.full((V, H), 0x5A5A, dtype=torch.int16, device=DEV)
    ros = torch.full((V,), -9, dtype=torch.int32, device=DEV)
    boff = torch.full((g.R * g.S + 1,), -9, dtype=torch.int64, device=DEV)
    ws = torch.empty(uep.ultraep_dispatch_ws_bytes(T, k, g), dtype=torch.uint8, device=DEV)
    xd, tkd = dev_u16(x), dev_i32(topk)
    if split:
        uep.ultraep_dispatch_layout(tkd, T, k, rank, g, plan, ros, boff, ws, st)
        uep.ultraep_dispatch_scatter(xd, T, k, H, ros, boff[-1:], send)
    else:
        uep.ultraep_dispatch(xd, tkd, T, k, H, rank, g, plan, send, ros, boff, ws, st)
    torch.cuda.synchronize()
    return host_u16(send), ros.cpu().numpy(), boff.cpu().numpy(), int(st.item())


def gpu_pack(w, rank, g, plan, cap):
    n_main, W = w.shape
    st = zero_status()
    staging = torch.full((max(cap, 0), W), 0x3C3C, dtype=torch.int16, device=DEV)
    doff = torch.full((g.R + 1,), -9, dtype=torch.int64, device=DEV)
    uep.ultraep_pack_replicas(dev_u16(w), W, rank, g, plan, staging, cap, doff, st)
    torch.cuda.synchronize()
    return host_u16(staging), doff.cpu().numpy(), int(st.item())


def check_rank(x, topk, w, rank, g, og, plan, op, cap=None, split=False):
    """Dispatch and pack of one rank on the GPU against the oracle."""
    osend, oros, oboff, ost = oracle.dispatch(x, topk, rank, og, op)
    assert ost == 0
    send, ros, boff, st = gpu_dispatch(x, topk, rank, g, plan, split=split)
    assert st == 0, st
    assert_same(f"block_off rank {rank}", boff, oboff)
    assert_same(f"row_of_slot rank {rank}", ros, oros)
    assert_same(f"send rank {rank}", send, osend)
    if w is not None:
        cap = g.R * g.n_slot if cap is None else cap
        ostg, odoff, n_out, ost = oracle.pack(w, rank, og, op, cap)
        assert ost == 0
        stg, doff, st = gpu_pack(w, rank, g, plan, cap)
        assert st == 0, st
        assert_same(f"dest_off rank {rank}", doff, odoff)
        assert_same(f"staging rank {rank}", stg[:n_out], ostg[:n_out])
        assert (stg[n_out:] == 0x3C3C).all(), "staging written past n_out"
