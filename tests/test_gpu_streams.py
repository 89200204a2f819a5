"""Reentrancy across streams: the library keeps no state between calls, so
two complete pipelines (count, plan, dispatch, pack, relay trees, combine)
with their own buffers, launched interleaved call by call on two streams,
must each give the oracle's bytes.  Both streams keep the default priority.
Needs an MI355X."""
import numpy as np
import pytest
import torch

import gen
import oracle

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    import gpu_path as gp
    import paper_2606_04101_amd as uep


OUT_POISON = 0x7FA5  # a NaN payload: the combine writes every NaN as 0x7FC0


class Pipe:
    """One workload's buffers and its calls, in order."""

    def __init__(self, cid, m, W):
        c = gen.config(cid)
        self.c, self.m, self.W = c, m, W
        self.g, self.og = gp.groups(c.R, c.E, c.n_slot, c.u_min, c.beta_num, c.beta_den)
        self.tk_all = gen.topk_all(c, m)
        load, _ = oracle.count(self.tk_all, c.E, c.R)
        self.op = oracle.plan(load, self.og)
        X = self.op.slot_expert
        outb = [int(((X >= 0) & (X // c.n_main == r)).sum()) for r in range(c.R)]
        self.rank = int(np.argmax(outb))
        self.x_h = gen.activations(c, m, self.rank)
        self.w_h = gen.weights(c, self.rank, W=W)
        rng = np.random.default_rng(cid * 100 + m)
        self.gate_h = rng.random((c.T, c.k)).astype(np.float32)
        T, k, H, g = c.T, c.k, c.H, self.g
        V = T * k
        dev = gp.DEV
        self.tk_d = gp.dev_i32(self.tk_all)
        self.tk_r = self.tk_d[self.rank].contiguous()
        self.x, self.w = gp.dev_u16(self.x_h), gp.dev_u16(self.w_h)
        self.gate = torch.from_numpy(self.gate_h).to(dev)
        self.st = gp.zero_status()
        self.load = torch.empty((c.R, c.E), dtype=torch.int32, device=dev)
        self.plan = uep.Plan(g, dev)
        self.send = torch.empty((V, H), dtype=torch.int16, device=dev)
        self.ros = torch.empty(V, dtype=torch.int32, device=dev)
        self.boff = torch.empty(c.R * g.S + 1, dtype=torch.int64, device=dev)
        self.ws = torch.empty(uep.ultraep_dispatch_ws_bytes(T, k, g), dtype=torch.uint8, device=dev)
        self.cap = c.R * c.n_slot
        self.stg = torch.zeros((self.cap, W), dtype=torch.int16, device=dev)
        self.doff = torch.empty(c.R + 1, dtype=torch.int64, device=dev)
        self.src = torch.empty(max(c.R * c.n_slot, 1), dtype=torch.int32, device=dev)
        self.vol = torch.empty(c.R, dtype=torch.int32, device=dev)
        self.rst = torch.empty(4, dtype=torch.int64, device=dev)
        self.out = torch.full((T, H), OUT_POISON, dtype=torch.int16, device=dev)

    def calls(self):
        c, g, p = self.c, self.g, self
        T, k, H, V = c.T, c.k, c.H, c.T * c.k
        return [
            lambda: uep.ultraep_count(p.tk_d, T, k, c.E, c.R, p.load, p.st),
            lambda: uep.ultraep_plan(p.load, g, p.plan),
            lambda: uep.ultraep_dispatch(p.x, p.tk_r, T, k, H, p.rank, g, p.plan, p.send, p.ros,
                                         p.boff, p.ws, p.st),
            lambda: uep.ultraep_pack_replicas(p.w, p.W, p.rank, g, p.plan, p.stg, p.cap, p.doff,
                                              p.st),
            lambda: uep.ultraep_relay_plan(g, p.plan, 4, p.src, p.vol, p.rst, p.st),
            lambda: uep.ultraep_combine(p.send, V, p.gate, p.ros, T, k, H, p.out, p.st),
        ]

    def check(self):
        c, name = self.c, f"workload {self.c.cid} microbatch {self.m} rank {self.rank}"
        assert int(self.st.item()) == 0, name
        ocnt, _ = oracle.count(self.tk_all, c.E, c.R)
        gp.assert_same(f"{name} counts", self.load.cpu().numpy(), ocnt)
        gp.assert_plan_equal(self.plan, self.op)
        osend, oros, oboff, _ = oracle.dispatch(self.x_h, self.tk_all[self.rank], self.rank,
                                                self.og, self.op)
        gp.assert_same(f"{name} row_of_slot", self.ros.cpu().numpy(), oros)
        gp.assert_same(f"{name} block_off", self.boff.cpu().numpy(), oboff)
        gp.assert_same(f"{name} send", gp.host_u16(self.send), osend)
        ostg, odoff, n_out, _ = oracle.pack(self.w_h, self.rank, self.og, self.op, self.cap)
        gp.assert_same(f"{name} dest_off", self.doff.cpu().numpy(), odoff)
        gp.assert_same(f"{name} staging", gp.host_u16(self.stg)[:n_out], ostg[:n_out])
        rel = oracle.relay(self.og, self.op, 4)
        gp.assert_same(f"{name} slot_src",
                       self.src.cpu().numpy()[: c.R * c.n_slot].reshape(c.R, c.n_slot),
                       rel.slot_src.reshape(c.R, c.n_slot))
        gp.assert_same(f"{name} send_vol", self.vol.cpu().numpy(), rel.send_vol)
        oout, _ = oracle.combine(osend, self.gate_h, oros)
        out = gp.host_u16(self.out)
        if not np.array_equal(out, oout):
            # facts that tell a kernel fault from a visibility fault, gathered
            # once: elements never written (still the poison), a second read
            # of the same buffer, and the combine run again alone on the
            # default stream over the same inputs
            bad = out != oout
            poison = int((out[bad] == OUT_POISON).sum())
            again = gp.host_u16(self.out)
            fresh = torch.full_like(self.out, OUT_POISON)
            st = gp.zero_status()
            T, k, H = c.T, c.k, c.H
            uep.ultraep_combine(self.send, T * k, self.gate, self.ros, T, k, H, fresh, st)
            torch.cuda.synchronize()
            rerun = gp.host_u16(fresh)
            print(f"{name}: {int(bad.sum())} combine outputs differ, {poison} of them still "
                  f"hold the poison; a second read differs from the first in "
                  f"{int((again != out).sum())}; the combine run again alone differs from "
                  f"the oracle in {int((rerun != oout).sum())} (status {int(st.item())})",
                  flush=True)
            gp.assert_same(f"{name} combine out", out, oout)


def test_two_pipelines_on_two_streams():
    print("two pipelines: workload 2 microbatch 0, workload 3 microbatch 4", flush=True)
    pipes = [Pipe(2, 0, 8 * 4096), Pipe(3, 4, 8 * 4096)]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    for s in streams:
        s.wait_stream(torch.cuda.current_stream())  # inputs were written on the default stream
    calls = [p.calls() for p in pipes]
    for rep in range(3):
        for pair in zip(*calls):
            for s, f in zip(streams, pair):
                with torch.cuda.stream(s):
                    f()
    torch.cuda.synchronize()
    errors = []
    for p in pipes:  # both pipelines are checked before any failure is raised
        try:
            p.check()
        except AssertionError as e:
            errors.append(str(e))
    assert not errors, "\n".join(errors)
