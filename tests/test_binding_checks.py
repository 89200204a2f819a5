"""The Python binding refuses tensors too small (or of the wrong element size)
for the shapes it is given, before the library is called, so that no kernel
runs past a caller's buffer.  No GPU needed: the check comes first."""
import pytest
import torch

import paper_2606_04101_amd as uep


def t(n, dtype=torch.int32):
    return torch.zeros(n, dtype=dtype)


G = uep.Group(4, 16, 2, 8)  # n_main = 4, S = 6, R * n_slot = 8


def test_count_buffers():
    with pytest.raises(ValueError, match="topk"):
        uep.ultraep_count(t(2 * 10 * 2 - 1), 10, 2, 16, 2, t(32), t(1))
    with pytest.raises(ValueError, match="counts"):
        uep.ultraep_count(t(40), 10, 2, 16, 2, t(31), t(1))
    with pytest.raises(ValueError, match="status"):
        uep.ultraep_count(t(40), 10, 2, 16, 2, t(32), None)


def test_plan_load():
    plan = type("P", (), {})()  # never reached
    for f in (uep.ultraep_plan, uep.ultraep_plan_replicate):
        with pytest.raises(ValueError, match="load"):
            f(t(4 * 16 - 1), G, plan, ws=t(1, torch.uint8))
    with pytest.raises(ValueError, match="load"):
        uep.ultraep_plan_reroute(t(63), G, plan)


def test_dispatch_buffers():
    T, k, H = 10, 2, 16
    ok = dict(x=t(T * H, torch.int16), topk=t(T * k), send=t(T * k * H, torch.int16),
              row_of_slot=t(T * k), block_off=t(4 * 6 + 1, torch.int64), status=t(1))
    for name, bad in [("x", t(T * H - 1, torch.int16)), ("send", t(T * k * H - 8, torch.int16)),
                      ("topk", t(T * k - 1)), ("row_of_slot", t(T * k - 1)),
                      ("block_off", t(4 * 6, torch.int64)), ("block_off", t(25, torch.int32))]:
        a = dict(ok, **{name: bad})
        with pytest.raises(ValueError, match=name):
            uep.ultraep_dispatch(a["x"], a["topk"], T, k, H, 0, G, None, a["send"],
                                 a["row_of_slot"], a["block_off"], t(1, torch.uint8), a["status"])
    with pytest.raises(ValueError, match="n_routed"):
        uep.ultraep_dispatch_scatter(ok["x"], T, k, H, ok["row_of_slot"], None, ok["send"])


def test_pack_and_relay_buffers():
    W, cap = 64, 3
    w = t(4 * W, torch.int16)
    with pytest.raises(ValueError, match="w_main"):
        uep.ultraep_pack_replicas(t(4 * W - 1, torch.int16), W, 0, G, None,
                                  t(cap * W, torch.int16), cap, t(5, torch.int64), t(1))
    with pytest.raises(ValueError, match="staging"):
        uep.ultraep_pack_replicas(w, W, 0, G, None, t(cap * W - 1, torch.int16), cap,
                                  t(5, torch.int64), t(1))
    with pytest.raises(ValueError, match="dest_off"):
        uep.ultraep_reroute_and_pack(t(64), G, None, w, W, 0, t(cap * W, torch.int16), cap,
                                     t(4, torch.int64), t(1))
    with pytest.raises(ValueError, match="relay_src"):
        uep.ultraep_pack_relay(w, t(2 * W - 1, torch.int16), W, 0, G, None, t(8),
                               t(cap * W, torch.int16), cap, t(5, torch.int64), t(1))
    with pytest.raises(ValueError, match="send_vol"):
        uep.ultraep_relay_plan(G, None, 4, t(8), t(3), t(4, torch.int64), t(1))
    with pytest.raises(ValueError, match="relay_stats"):
        uep.ultraep_relay_plan(G, None, 4, t(8), t(4), t(4), t(1))


def test_combine_and_reduce_buffers():
    T, k, H = 5, 3, 8
    args = dict(y=t(15 * H, torch.int16), gate=t(T * k, torch.float32), ros=t(T * k),
                out=t(T * H, torch.int16))
    for name, key, bad in [("y", "y", t(15 * H - 1, torch.int16)),
                           ("gate", "gate", t(T * k, torch.float16)),
                           ("row_of_slot", "ros", t(T * k - 1)),
                           ("out", "out", t(T * H, torch.float32))]:
        a = dict(args, **{key: bad})
        with pytest.raises(ValueError, match=name):
            uep.ultraep_combine(a["y"], 15, a["gate"], a["ros"], T, k, H, a["out"], t(1))
    with pytest.raises(ValueError, match="main_grad"):
        uep.ultraep_grad_reduce(t(4 * 8 - 1, torch.float32), t(8, torch.float32), 8, 0, G, None,
                                1, t(1))
    with pytest.raises(ValueError, match="rgrad"):
        uep.ultraep_grad_reduce(t(32, torch.float32), t(2 * 8, torch.int16), 8, 0, G, None, 2,
                                t(1))
